"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer, on the
CPU (no GPU is needed or used):

* the C ABI's host argument checks: every library source built with
  host-side instrumentation (the device code is compiled as usual and never
  runs) and linked with tests/sanitize/abi_checks.cpp, which makes only calls
  that are rejected before anything is enqueued, or size queries;
* the oracle and the input generator: oracle.c and gen.c built with the same
  sanitizers and loaded, in a subprocess with the sanitizer runtimes
  preloaded, by the pin tests that exercise them without torch (the CSR,
  aggregation, typed-graph and stacked-aggregation pins)."""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2507_16991_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all"]
SOURCES = ["scan.hip", "sort.hip", "spmm.hip", "backward.hip", "gmm.hip", "messages.hip",
           "layout.hip", "probe.hip", "api.cpp"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd[:3])} ... failed:\n{r.stdout[-3000:]}\n{r.stderr[-3000:]}"
    return r


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_abi_host_checks_sanitized(tmp_path):
    inc = ["-I" + os.path.join(ROOT, "include"), "-I" + CSRC]

    def compile_one(src):
        obj = str(tmp_path / (src + ".o"))
        _run([HIPCC, "-x", "hip", "--offload-arch=gfx950", "-O1", "-std=c++17", *HOST_SAN, *inc,
              "-c", os.path.join(CSRC, src), "-o", obj])
        return obj

    with ThreadPoolExecutor(max_workers=4) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    drv = str(tmp_path / "abi_checks.o")
    _run([HIPCC, "-x", "hip", "--offload-host-only", "-O1", "-std=c++17", *HOST_SAN, *inc, "-c",
          os.path.join(ROOT, "tests", "sanitize", "abi_checks.cpp"), "-o", drv])
    exe = str(tmp_path / "abi_checks")
    _run([HIPCC, "--offload-arch=gfx950", *HOST_SAN, *objs, drv, "-o", exe])
    r = _run([exe], env=ENV)
    assert "abi checks ok" in r.stdout


def test_oracle_and_generator_sanitized(tmp_path):
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
    libs = {}
    for mod, src in (("oracle", "oracle/oracle.c"), ("graphgen", "graphgen/gen.c")):
        out = str(tmp_path / f"lib{mod}_san.so")
        _run(["gcc", "-O1", "-g", *san, "-fopenmp", "-fPIC", "-shared", "-std=c11",
              os.path.join(ROOT, src), "-o", out, "-lm"])
        libs[mod] = out
    rt = [_run(["gcc", f"-print-file-name={n}"]).stdout.strip() for n in ("libasan.so",
                                                                          "libubsan.so")]
    script = (
        "import sys; sys.path.insert(0, {root!r}); sys.path.insert(0, {tests!r})\n"
        "import oracle, graphgen\n"
        "oracle._LIB_PATH = {o!r}; graphgen._LIB_PATH = {g!r}\n"
        "import pytest\n"
        "sys.exit(pytest.main(['-q', '-x', '-p', 'no:cacheprovider', '-m', 'not gpu', {files}]))\n"
    ).format(root=ROOT, tests=os.path.join(ROOT, "tests"), o=libs["oracle"], g=libs["graphgen"],
             files=", ".join(repr(os.path.join(ROOT, "tests", f)) for f in
                             ("test_oracle_csr.py", "test_oracle_spmm.py", "test_oracle_hetero.py",
                              "test_oracle_multi.py")))
    env = dict(ENV, LD_PRELOAD=":".join(rt), OMP_NUM_THREADS="4")
    r = _run([sys.executable, "-c", script], env=env, cwd=str(tmp_path))
    assert " passed" in r.stdout
