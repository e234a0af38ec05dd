"""Build libmp.so (HIP, gfx950) in-tree with hipcc.

Every source under csrc/ is compiled for gfx950 only, with packed-fp32
instruction selection disabled, and linked into paper_2507_16991_amd/libmp.so.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OBJ = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libmp.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = ["scan.hip", "sort.hip", "spmm.hip", "backward.hip", "gmm.hip", "messages.hip",
           "layout.hip", "probe.hip", "api.cpp"]
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-command-line-argument",
    "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
]


def _compile(src: str, obj_dir: str = OBJ, extra=()) -> str:
    out = os.path.join(obj_dir, src + ".o")
    cmd = [HIPCC, *FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", out]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed on {src}")
    warn = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l
                     and "not a recognized feature" not in l)
    if warn.strip():
        sys.stderr.write(warn + "\n")
    return out


def build(lib: str = LIB, defines=()) -> str:
    """Compile and link; `defines` (e.g. ["-DMP_SORT_ITEMS=8"]) override the
    compile-time tuning constants, `lib` the output path."""
    obj_dir = OBJ if lib == LIB else lib + ".objs"
    os.makedirs(obj_dir, exist_ok=True)
    with ThreadPoolExecutor(max_workers=4) as ex:
        objs = list(ex.map(lambda s: _compile(s, obj_dir, defines), SOURCES))
    tmp = lib + ".tmp"
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, lib)
    return lib


def resource_usage(out: str, pattern: str = "") -> str:
    """Registers, spills, LDS and occupancy of every kernel, as the compiler
    reports them (-Rpass-analysis=kernel-resource-usage), one line per kernel
    whose demangled name matches `pattern`; written to `out`."""
    import re
    rows = []
    for src in SOURCES:
        if not src.endswith(".hip"):
            continue
        cmd = [HIPCC, *FLAGS, "--offload-device-only", "-c", os.path.join(CSRC, src),
               "-o", os.devnull, "-Rpass-analysis=kernel-resource-usage"]
        err = subprocess.run(cmd, capture_output=True, text=True).stderr
        cur = None
        for line in err.splitlines():
            m = re.search(r"remark: (.*?) \[-Rpass", line)
            if not m:
                continue
            key, _, val = m.group(1).strip().partition(":")
            if key == "Function Name":
                cur = {"src": src, "name": val.strip()}
                rows.append(cur)
            elif cur is not None:
                cur[key.strip()] = val.strip()
    names = subprocess.run(["c++filt"], input="\n".join(r["name"] for r in rows),
                           capture_output=True, text=True).stdout.splitlines()
    lines = ["# kernel resource usage (hipcc -Rpass-analysis=kernel-resource-usage, gfx950)",
             f"command: python paper_2507_16991_amd/build.py --resource-usage {out}"
             + (f" '{pattern}'" if pattern else ""), "",
             f"{'vgpr':>4} {'agpr':>4} {'sgpr':>4} {'spill':>5} {'lds_B':>6} {'waves/SIMD':>10}  kernel"]
    for r, n in zip(rows, names):
        n = n.replace("mp::(anonymous namespace)::", "").replace("void ", "")
        depth = 0  # drop the parameter list
        for i, ch in enumerate(n):
            depth += (ch == "<") - (ch == ">")
            if ch == "(" and depth == 0:
                n = n[:i]
                break
        if pattern and not re.search(pattern, n):
            continue
        lines.append(f"{r.get('VGPRs', '?'):>4} {r.get('AGPRs', '?'):>4} {r.get('TotalSGPRs', '?'):>4} "
                     f"{r.get('VGPRs Spill', '?'):>5} {r.get('LDS Size [bytes/block]', '?'):>6} "
                     f"{r.get('Occupancy [waves/SIMD]', '?'):>10}  {r['src']}: {n}")
    open(out, "w").write("\n".join(lines) + "\n")
    return out


if __name__ == "__main__":
    if len(sys.argv) > 2 and sys.argv[1] == "--resource-usage":
        print(resource_usage(sys.argv[2], sys.argv[3] if len(sys.argv) > 3 else ""))
    else:
        print(build())
