"""CPU checks of the C ABI: the library loads, exports every function that
include/mp.h declares, and rejects bad arguments on the host (before any
device work) with the documented status codes."""
import ctypes
import os
import re

import pytest

import paper_2507_16991_amd as mp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("mp.h", "mp_probe.h")]

FAKE = 0x10000  # a non-NULL, aligned pointer value; never dereferenced by these cases


def declared_functions():
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mp_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_function():
    L = mp.lib()
    names = declared_functions()
    assert "mp_spmm" in names and "mp_coo_to_csr" in names and "mp_hetero_spmm" in names
    for n in names:
        assert hasattr(L, n), f"{n} declared in mp.h but not exported"


def test_probe_argument_errors():
    L = mp.lib()
    assert L.mp_probe_read(None, 64, FAKE, None) == -1
    assert L.mp_probe_read(FAKE, 60, FAKE, None) == -2
    assert L.mp_probe_read(FAKE + 4, 64, FAKE, None) == -8
    assert L.mp_probe_copy(FAKE, FAKE, 0, None) == -2
    assert L.mp_probe_copy(FAKE, FAKE + 8, 64, None) == -8
    assert L.mp_probe_gather(FAKE, 10, FAKE, 400, 400, None, None) == -1
    assert L.mp_probe_gather(FAKE, 10, FAKE, 400, 392, FAKE, None) == -2   # not whole chunks
    assert L.mp_probe_gather(FAKE, 10, FAKE, 256, 400, FAKE, None) == -2   # row > stride
    assert L.mp_probe_gather(FAKE, 10, FAKE, 2048, 2048, FAKE, None) == -2  # over 1024 bytes
    assert L.mp_probe_gather(FAKE, 10, FAKE + 8, 400, 400, FAKE, None) == -8
    assert L.mp_probe_gather(None, 0, None, 400, 400, FAKE, None) == 0     # nothing to read
    assert L.mp_probe_scatter(FAKE, None, 10, 8, FAKE, None) == -1
    assert L.mp_probe_scatter(FAKE, FAKE, 10, 2, FAKE, None) == -2          # 4 or 8 bytes
    assert L.mp_probe_scatter(FAKE, FAKE, -1, 8, FAKE, None) == -2
    assert L.mp_probe_scatter(FAKE + 4, FAKE, 10, 8, FAKE, None) == -8
    assert L.mp_probe_scatter(FAKE, FAKE + 2, 10, 4, FAKE, None) == -8
    assert L.mp_probe_scatter(None, None, 0, 8, None, None) == 0            # nothing to move


def test_noalloc_argument_errors():
    L = mp.lib()
    # arguments of a valid plan-free sum; each case breaks one (never a valid call: the
    # pointers are fake)
    a = [None, FAKE, 0, FAKE, None, FAKE, 0, 10, 10, 8, 8, 1, FAKE, 0, None, 0, None, None]
    b = list(a); b[11] = 3  # SUM|MEAN
    assert L.mp_spmm_noalloc(*b) == -4
    b = list(a); b[3] = None
    assert L.mp_spmm_noalloc(*b) == -1
    b = list(a); b[5] = FAKE + 2
    assert L.mp_spmm_noalloc(*b) == -8


def test_version_and_status_strings():
    assert mp.mp_version() == 5
    for st in range(-10, 1):
        assert mp.mp_status_str(st) != "unknown status"
    assert mp.mp_status_str(-99) == "unknown status"


def test_coo_to_csr_workspace_sizes():
    assert mp.mp_coo_to_csr_workspace(0, 5, mp.MP_I32, 0) == 0
    a = mp.mp_coo_to_csr_workspace(1000, 5, mp.MP_I32, 0)
    b = mp.mp_coo_to_csr_workspace(1000, 5, mp.MP_I32, 1)
    assert 0 < a < b
    # more key bits -> more passes -> ping-pong buffers
    assert mp.mp_coo_to_csr_workspace(10**6, 2**20, mp.MP_I32, 0) > \
        mp.mp_coo_to_csr_workspace(10**6, 200, mp.MP_I32, 0)


@pytest.mark.parametrize("E,N", [(-1, 5), (5, 0), (2**31, 5), (5, 2**31)])
def test_coo_to_csr_size_errors(E, N):
    with pytest.raises(mp.MPError) as e:
        mp.mp_coo_to_csr_workspace(E, N, mp.MP_I32, 0)
    assert e.value.status == -2


def test_coo_to_csr_argument_errors():
    L = mp.lib()
    # bad index type
    assert L.mp_coo_to_csr(FAKE, FAKE, 10, 5, FAKE, 7, FAKE, None, None, None, FAKE, 1 << 20,
                           None, None) == -3
    # NULL rowptr / src
    assert L.mp_coo_to_csr(FAKE, FAKE, 10, 5, None, 0, FAKE, None, None, None, FAKE, 1 << 20,
                           None, None) == -1
    assert L.mp_coo_to_csr(None, FAKE, 10, 5, FAKE, 0, FAKE, None, None, None, FAKE, 1 << 20,
                           None, None) == -1
    # val_in without val_out
    assert L.mp_coo_to_csr(FAKE, FAKE, 10, 5, FAKE, 0, FAKE, None, FAKE, None, FAKE, 1 << 20,
                           None, None) == -1
    # misaligned int64 rowptr; misaligned status word
    assert L.mp_coo_to_csr(FAKE, FAKE, 10, 5, FAKE + 4, 1, FAKE, None, None, None, FAKE, 1 << 20,
                           None, None) == -8
    assert L.mp_coo_to_csr(FAKE, FAKE, 10, 5, FAKE, 0, FAKE, None, None, None, FAKE, 1 << 20,
                           FAKE + 2, None) == -8
    # workspace too small
    assert L.mp_coo_to_csr(FAKE, FAKE, 10, 5, FAKE, 0, FAKE, None, None, None, FAKE, 16,
                           None, None) == -5


def test_plan_errors():
    L = mp.lib()
    h = ctypes.c_void_p(0)
    assert mp.mp_spmm_plan_size(100, 1000) > 0
    assert L.mp_spmm_plan_build(FAKE, 0, 100, 1000, 64, 0, FAKE, 16, None, ctypes.byref(h)) == -5
    assert L.mp_spmm_plan_build(FAKE, 0, 100, 1000, 0, 0, FAKE, 1 << 30, None,
                                ctypes.byref(h)) == -2
    assert L.mp_spmm_plan_build(FAKE, 0, 100, 1000, 64, 9, FAKE, 1 << 30, None,
                                ctypes.byref(h)) == -3
    assert L.mp_spmm_plan_build(None, 0, 100, 1000, 64, 0, FAKE, 1 << 30, None,
                                ctypes.byref(h)) == -1
    assert mp.mp_spmm_workspace(None, mp.MP_SUM) == 0
    with pytest.raises(mp.MPError):
        mp.mp_spmm_workspace(None, 3)  # SUM|MEAN is not a valid combination
    # explicit thresholds: negative fields and chunks over INT32_MAX are rejected
    for bad in ((-1, 0, 0), (0, -1, 0), (0, 0, -1), (0, 0, 1 << 31)):
        o = mp.mp_plan_opts(*bad)
        assert L.mp_spmm_plan_build_opts(FAKE, 0, 100, 1000, 64, 0, FAKE, 1 << 30,
                                         ctypes.byref(o), None, ctypes.byref(h)) == -2
    o = mp.mp_plan_opts(8, 64, 16)
    assert L.mp_spmm_plan_build_opts(FAKE, 0, 100, 1000, 64, 0, FAKE, 16, ctypes.byref(o), None,
                                     ctypes.byref(h)) == -5


def _spmm(**kw):
    a = dict(plan=None, rowptr=FAKE, itype=0, col=FAKE, w=None, x=FAKE, x_dtype=0, N_src=10,
             N_dst=10, F=8, ldx=8, reduce=1, out=FAKE, out_dtype=0, out_max=None, max_dtype=0,
             argout=None, ws=None, ws_bytes=0, stream=None)
    a.update(kw)
    return mp.lib().mp_spmm(*a.values())


def test_spmm_argument_errors():
    assert _spmm(reduce=0) == -4
    assert _spmm(reduce=1 | 2) == -4
    assert _spmm(reduce=8) == -4
    assert _spmm(x_dtype=5) == -3
    assert _spmm(itype=3) == -3
    assert _spmm(reduce=4, max_dtype=1, out_max=FAKE, argout=FAKE) == -3   # bf16 max of f32 x
    assert _spmm(reduce=4, x_dtype=1, w=FAKE, max_dtype=1, out_max=FAKE, argout=FAKE) == -3
    assert _spmm(F=0) == -2
    assert _spmm(N_src=-1) == -2
    assert _spmm(N_dst=2**31) == -2
    assert _spmm(out=None) == -1
    assert _spmm(reduce=4, out_max=FAKE, argout=None) == -1
    assert _spmm(col=None) == -1
    assert _spmm(x=FAKE + 2) == -8
    assert _spmm(ldx=7) == -2  # rows may not overlap


def test_copy_rows_argument_errors():
    L = mp.lib()
    assert L.mp_copy_rows(FAKE, 8, FAKE, 8, 10, 8, 7, None) == -3
    assert L.mp_copy_rows(FAKE, 7, FAKE, 8, 10, 8, 0, None) == -2
    assert L.mp_copy_rows(FAKE, 8, FAKE, 7, 10, 8, 0, None) == -2
    assert L.mp_copy_rows(FAKE, 8, FAKE, 8, -1, 8, 0, None) == -2
    assert L.mp_copy_rows(None, 8, FAKE, 8, 10, 8, 0, None) == -1
    assert L.mp_copy_rows(FAKE + 2, 8, FAKE, 8, 10, 8, 0, None) == -8
    assert L.mp_copy_rows(None, 8, None, 8, 0, 8, 0, None) == 0


def test_aligned_row_strides():
    import torch
    assert mp.aligned_ld(100, torch.bfloat16) == 128   # 200-byte rows: 2.5 -> 2 lines
    assert mp.aligned_ld(50, torch.float32) == 64
    assert mp.aligned_ld(100, torch.float32) == 100    # 400-byte rows touch 4 lines anyway
    assert mp.aligned_ld(64, torch.bfloat16) == 64     # already whole lines
    assert mp.aligned_ld(24, torch.bfloat16) == 24     # below one line: never padded
    assert mp.aligned_ld(300, torch.bfloat16) == 320


def test_hetero_errors():
    L = mp.lib()
    npt = (ctypes.c_int64 * 2)(10, 5)
    b = ctypes.c_size_t(0)
    rel = (mp.mp_relation * 1)(mp.mp_relation(0, 1, FAKE, FAKE, 20))
    assert L.mp_hetero_build_workspace(2, npt, 1, rel, 1, 0, ctypes.byref(b)) == 0 and b.value > 0
    assert L.mp_hetero_build_workspace(2, npt, 1, rel, 2, 0, ctypes.byref(b)) == -2
    assert L.mp_hetero_build_workspace(2, npt, 1, rel, -2, 0, ctypes.byref(b)) == -2
    # every destination type at once: rows are all 15 nodes
    assert L.mp_hetero_build_workspace(2, npt, 1, rel, mp.MP_ALL_TYPES, 0,
                                       ctypes.byref(b)) == 0 and b.value > 0
    assert L.mp_hetero_build_workspace(0, npt, 1, rel, 0, 0, ctypes.byref(b)) == -2
    bad = (mp.mp_relation * 1)(mp.mp_relation(0, 3, FAKE, FAKE, 20))
    assert L.mp_hetero_build_workspace(2, npt, 1, bad, 1, 0, ctypes.byref(b)) == -2
    # build: NULL col, small workspace, misaligned status word
    assert L.mp_hetero_build(2, npt, 1, rel, 1, FAKE, 0, None, FAKE, 1 << 20, None, None) == -1
    assert L.mp_hetero_build(2, npt, 1, rel, 1, FAKE, 0, FAKE, FAKE, 16, None, None) == -5
    assert L.mp_hetero_build(2, npt, 1, rel, 1, FAKE, 0, FAKE, FAKE, 1 << 20, FAKE + 2,
                             None) == -8
    xs = (ctypes.c_void_p * 2)(FAKE, FAKE)
    assert L.mp_hetero_spmm(2, npt, xs, 0, 8, 1, None, FAKE, 0, FAKE, mp.MP_MEAN, FAKE, 0, None,
                            0, None) == -4


def test_sorted_coo_to_csr_errors():
    L = mp.lib()
    assert L.mp_sorted_coo_to_csr(FAKE, FAKE, 10, 5, FAKE, 7, FAKE, None, None, None, None) == -3
    assert L.mp_sorted_coo_to_csr(FAKE, FAKE, 10, 5, None, 0, FAKE, None, None, None, None) == -1
    assert L.mp_sorted_coo_to_csr(None, FAKE, 10, 5, FAKE, 0, FAKE, None, None, None, None) == -1
    assert L.mp_sorted_coo_to_csr(FAKE, FAKE, 10, 5, FAKE, 0, FAKE, None, FAKE, None, None) == -1
    assert L.mp_sorted_coo_to_csr(FAKE, FAKE, 10, 5, FAKE + 4, 1, FAKE, None, None, None,
                                  None) == -8
    assert L.mp_sorted_coo_to_csr(FAKE, FAKE, -1, 5, FAKE, 0, FAKE, None, None, None, None) < 0


def test_transpose_errors_and_sizes():
    L = mp.lib()
    nb = ctypes.c_size_t(0)
    assert L.mp_csr_transpose_workspace(1000, 50, 0, 1, ctypes.byref(nb)) == 0
    assert nb.value >= 4 * 1000
    assert L.mp_csr_transpose_workspace(1000, 0, 0, 1, ctypes.byref(nb)) == -2
    args = [FAKE, 0, FAKE, 10, 20, 100, FAKE, 0, FAKE, FAKE, None, None, FAKE, 1 << 20, None,
            None]
    def call(**kw):
        a = list(args)
        names = ["rowptr", "it", "col", "N_dst", "N_src", "E", "rowptrT", "itT", "colT", "posT",
                 "val_in", "val_out", "ws", "ws_bytes", "status", "stream"]
        for k, v in kw.items():
            a[names.index(k)] = v
        return L.mp_csr_transpose(*a)
    assert call(it=5) == -3
    assert call(itT=5) == -3
    assert call(N_dst=0) == -2
    assert call(rowptrT=None) == -1
    assert call(val_in=FAKE) == -1
    assert call(rowptrT=FAKE + 4, itT=1) == -8
    assert call(status=FAKE + 1) == -8
    assert call(ws_bytes=16) == -5


def test_backward_errors_and_sizes():
    L = mp.lib()
    nb = ctypes.c_size_t(0)
    assert L.mp_spmm_backward_w_workspace(1000, ctypes.byref(nb)) == 0 and nb.value == 4096
    assert L.mp_spmm_backward_x_workspace(None, 10, 100, 8, mp.MP_MEAN, ctypes.byref(nb)) == 0
    assert nb.value == 512
    assert L.mp_spmm_backward_x_workspace(None, 10, 100, 8, mp.MP_SUM, ctypes.byref(nb)) == 0
    assert nb.value == 0
    # max: one 32-bit win-mask word per edge for F <= 32, ceil(F / 32) beyond
    assert L.mp_spmm_backward_x_workspace(None, 10, 100, 8, mp.MP_MAX, ctypes.byref(nb)) == 0
    assert nb.value == 512
    assert L.mp_spmm_backward_x_workspace(None, 10, 1000, 100, mp.MP_MAX,
                                          ctypes.byref(nb)) == 0
    assert nb.value == 16128  # 1000 * 4 words * 4 bytes, rounded up to 256
    assert L.mp_spmm_backward_x_workspace(None, 10, 100, 8, mp.MP_SUM | mp.MP_MAX,
                                          ctypes.byref(nb)) == -4
    assert L.mp_spmm_backward_x_workspace(None, 10, -1, 8, mp.MP_MAX, ctypes.byref(nb)) == -2
    assert L.mp_spmm_backward_x_workspace(None, 10, 1 << 31, 8, mp.MP_MAX,
                                          ctypes.byref(nb)) == -2
    bx = dict(planT=None, rowptrT=FAKE, itT=0, colT=FAKE, posT=FAKE, wT=None, rowptr=FAKE, it=0,
              argout=FAKE, g=FAKE, g_dtype=0, N_dst=10, N_src=10, E=100, F=8, reduce=mp.MP_SUM,
              out=FAKE, out_dtype=0, ws=None, ws_bytes=0, stream=None)
    def bwx(**kw):
        a = dict(bx, **kw)
        return L.mp_spmm_backward_x(*a.values())
    assert bwx(reduce=mp.MP_SUM | mp.MP_MAX) == -4
    assert bwx(reduce=mp.MP_MAX, argout=None) == -1
    assert bwx(reduce=mp.MP_MAX, posT=None) == -1
    assert bwx(reduce=mp.MP_MAX, rowptr=None) == -1  # rows of the forward positions
    assert bwx(reduce=mp.MP_MEAN, rowptr=None) == -1
    assert bwx(reduce=mp.MP_MEAN) == -5  # needs a workspace for the scaled gradient
    assert bwx(reduce=mp.MP_MAX) == -5  # needs a workspace for the win masks
    assert bwx(reduce=mp.MP_MAX, ws=FAKE, ws_bytes=511) == -5
    assert bwx(reduce=mp.MP_MAX, it=5) == -3
    assert bwx(reduce=mp.MP_MAX, rowptr=FAKE + 2) == -8
    assert bwx(E=-1) == -2
    assert bwx(g_dtype=3) == -3
    assert bwx(g=FAKE + 2) == -8
    assert bwx(F=0) == -2
    bw = dict(rowptr=FAKE, it=0, col=FAKE, x=FAKE, x_dtype=0, g=FAKE, g_dtype=0, argout=None,
              N_src=10, N_dst=10, E=100, F=8, reduce=mp.MP_SUM, out=FAKE, ws=FAKE,
              ws_bytes=1 << 20, stream=None)
    def bww(**kw):
        a = dict(bw, **kw)
        return L.mp_spmm_backward_w(*a.values())
    assert bww(reduce=mp.MP_MEAN | mp.MP_MAX) == -4
    assert bww(reduce=mp.MP_MAX) == -1
    assert bww(ws_bytes=16) == -5
    assert bww(N_dst=0) == -2
    assert bww(x=FAKE + 2) == -8
    assert bww(x_dtype=7) == -3


def test_multi_errors():
    L = mp.lib()
    nb = ctypes.c_size_t(7)
    assert L.mp_spmm_multi_workspace(None, ctypes.byref(nb)) == 0 and nb.value == 0

    def outs(*specs):
        arr = (mp.mp_aggr_out * max(len(specs), 1))()
        for k, (a, o, g) in enumerate(specs):
            arr[k].aggr, arr[k].out, arr[k].arg = a, o, g
        return arr

    def multi(specs, n=None, col=FAKE):
        arr = outs(*specs)
        return L.mp_spmm_multi(None, FAKE, 0, col, None, FAKE, 0, 10, 10, 8, 8,
                               len(specs) if n is None else n, arr, None, 0, None)

    assert multi([(mp.MP_SUM, FAKE, None), (mp.MP_SUM, FAKE, None)]) == -4  # duplicate
    assert multi([(mp.MP_SUM | mp.MP_MAX, FAKE, FAKE)]) == -4  # two aggregators in one
    assert multi([(64, FAKE, None)]) == -4
    assert multi([(mp.MP_SUM, FAKE, None)], n=0) == -2
    assert multi([(mp.MP_SUM, FAKE, None)], n=7) == -2
    assert multi([(mp.MP_MAX, FAKE, None)]) == -1  # max needs its positions
    assert multi([(mp.MP_MIN, FAKE, None)]) == -1
    assert multi([(mp.MP_VAR, None, None)]) == -1
    assert multi([(mp.MP_STD, FAKE + 2, None)]) == -8
    assert multi([(mp.MP_SUM, FAKE, None)], col=None) == -1
    arr = outs((mp.MP_MEAN, FAKE, None))
    assert L.mp_spmm_multi(None, FAKE, 0, FAKE, None, FAKE, 5, 10, 10, 8, 8, 1, arr, None, 0,
                           None) == -3
    assert L.mp_spmm_multi(None, FAKE, 0, FAKE, None, FAKE, 0, 10, 10, 8, 4, 1, arr, None, 0,
                           None) == -2
    assert L.mp_readout_multi(None, FAKE, 0, FAKE, 0, 100, 10, 0, 0, 1, arr, None, 0, None) == -2
    assert L.mp_readout_multi(None, None, 0, FAKE, 0, 100, 10, 8, 8, 1, arr, None, 0, None) == -1


def test_segment_matmul_errors_and_sizes():
    L = mp.lib()
    nb = ctypes.c_size_t(0)
    assert L.mp_segment_matmul_workspace(3, 128, 64, ctypes.byref(nb)) == 0
    assert nb.value == 3 * 128 * 64 * 2
    seg = (ctypes.c_int64 * 4)(0, 5000, 5000, 7000)
    assert L.mp_segment_matmul_backward_workspace(seg, 3, 64, 32, ctypes.byref(nb)) == 0
    assert nb.value == 4 * 64 * 32 * 4  # chunks of 2048 rows: 3 + 0 + 1
    assert L.mp_segment_matmul_workspace(0, 128, 64, ctypes.byref(nb)) == -2
    assert L.mp_segment_matmul_workspace(2, 12, 64, ctypes.byref(nb)) == -2

    def fwd(seg_vals, T=None, F=16, Fo=16, x=FAKE, ws_bytes=1 << 20, out_dtype=0):
        sg = (ctypes.c_int64 * len(seg_vals))(*seg_vals)
        T = len(seg_vals) - 1 if T is None else T
        return L.mp_segment_matmul(sg, T, x, FAKE, F, Fo, FAKE, out_dtype, FAKE, ws_bytes, None)

    assert fwd([1, 10]) == -2          # seg[0] != 0
    assert fwd([0, 10, 5]) == -2       # decreasing
    assert fwd([0, 10], T=17) == -2
    assert fwd([0, 10], F=20) == -2    # F not a multiple of 8
    assert fwd([0, 10], x=FAKE + 8) == -8
    assert fwd([0, 10], ws_bytes=16) == -5
    assert fwd([0, 10], out_dtype=4) == -3
    sg = (ctypes.c_int64 * 2)(0, 10)
    assert L.mp_segment_matmul(None, 1, FAKE, FAKE, 16, 16, FAKE, 0, FAKE, 1 << 20, None) == -1
    assert L.mp_segment_matmul_backward(sg, 1, FAKE, FAKE, FAKE, 16, 16, None, 0, None, FAKE,
                                        1 << 20, None) == -1  # nothing requested
    assert L.mp_segment_matmul_backward(sg, 1, FAKE, None, FAKE, 16, 16, FAKE, 0, None, FAKE,
                                        1 << 20, None) == -1  # dx needs W
    assert L.mp_segment_matmul_backward(sg, 1, FAKE, FAKE, FAKE, 16, 16, None, 0, FAKE, FAKE,
                                        16, None) == -5


def test_validate_errors():
    L = mp.lib()
    assert L.mp_validate_sorted(FAKE, 10, None, None) == -1
    assert L.mp_validate_sorted(FAKE, -1, FAKE, None) == -2
    assert L.mp_validate_coo(FAKE, FAKE, 10, 5, 5, None, None) == -1
    assert L.mp_validate_csr(FAKE, 4, FAKE, 5, 5, 10, FAKE, None) == -3


# ---- edge-materialized messages -------------------------------------------------------

def test_message_gather_argument_errors():
    L = mp.lib()
    F32, BF16 = mp.MP_F32, mp.MP_BF16
    assert L.mp_message_gather(FAKE, None, FAKE, 5, 10, 10, 4, FAKE, F32, None) == -3
    assert L.mp_message_gather(FAKE, None, FAKE, F32, 10, 10, 4, FAKE, BF16, None) == -3
    assert L.mp_message_gather(FAKE, FAKE, FAKE, BF16, 10, 10, 4, FAKE, BF16, None) == -3
    assert L.mp_message_gather(FAKE, None, FAKE, F32, 10, -1, 4, FAKE, F32, None) == -2
    assert L.mp_message_gather(FAKE, None, FAKE, F32, 10, 10, 0, FAKE, F32, None) == -2
    assert L.mp_message_gather(FAKE, None, FAKE, F32, 10, 2**31, 4, FAKE, F32, None) == -2
    assert L.mp_message_gather(None, None, FAKE, F32, 10, 10, 4, FAKE, F32, None) == -1
    assert L.mp_message_gather(FAKE, None, FAKE, F32, 10, 10, 4, None, F32, None) == -1
    assert L.mp_message_gather(FAKE, None, FAKE, F32, 10, 10, 4, FAKE + 2, F32, None) == -8
    assert L.mp_message_gather(None, None, None, F32, 0, 0, 4, None, F32, None) == 0


def test_message_scale_argument_errors():
    L = mp.lib()
    assert L.mp_message_scale(FAKE, FAKE, 10, 4, None, None, 10, None) == -1
    assert L.mp_message_scale(FAKE, FAKE, 10, 4, FAKE, None, 9, None) == -2
    assert L.mp_message_scale(FAKE, FAKE, 10, 0, FAKE, None, 10, None) == -2
    assert L.mp_message_scale(FAKE + 2, FAKE, 10, 4, FAKE, None, 10, None) == -8
    assert L.mp_message_scale(None, None, 0, 4, None, None, 0, None) == 0


def test_message_aggregate_argument_errors():
    L = mp.lib()
    F32, BF16 = mp.MP_F32, mp.MP_BF16
    args = lambda **k: [k.get("plan"), k.get("rowptr", FAKE), mp.MP_I32, FAKE,
                        k.get("mdt", F32), k.get("E", 100), 10, 4, k.get("reduce", mp.MP_SUM),
                        FAKE, F32, FAKE, k.get("xdt", F32), FAKE, None, 0, None]
    assert L.mp_message_aggregate(*args(reduce=3)) == -4
    assert L.mp_message_aggregate(*args(rowptr=None)) == -1
    assert L.mp_message_aggregate(*args(E=2**31)) == -2
    assert L.mp_message_aggregate(*args(reduce=mp.MP_MAX, xdt=BF16)) == -3


def test_materialized_checks_everything_before_the_callback():
    L = mp.lib()
    calls = []
    cb = mp.MESSAGE_FN(lambda *a: calls.append(a) or 0)
    F32 = mp.MP_F32

    def call(reduce=mp.MP_SUM, msg=FAKE, col=FAKE, E=100, msg_dtype=F32):
        return L.mp_spmm_materialized(None, FAKE, mp.MP_I32, col, None, FAKE, F32, 50, 10, E, 4,
                                      msg, msg_dtype, ctypes.cast(cb, ctypes.c_void_p), None,
                                      reduce, FAKE, F32, FAKE, F32, FAKE, None, 0, None)

    assert call(reduce=3) == -4
    assert call(msg=None) == -1
    assert call(col=None) == -1
    assert call(E=-1) == -2
    assert call(msg_dtype=mp.MP_BF16) == -3
    assert calls == []


def test_message_backward_argument_errors():
    L = mp.lib()
    F32 = mp.MP_F32
    assert mp.mp_message_backward_workspace(0) == 0
    assert mp.mp_message_backward_workspace(1000) == 0  # no workspace needed
    assert L.mp_message_backward(FAKE, mp.MP_I32, None, FAKE, F32, 10, 100, 4, 3, FAKE, FAKE,
                                 1 << 20, None) == -4
    assert L.mp_message_backward(FAKE, mp.MP_I32, None, FAKE, F32, 10, 100, 4, mp.MP_MAX, FAKE,
                                 FAKE, 1 << 20, None) == -1
    assert L.mp_message_backward(FAKE, mp.MP_I32, None, None, F32, 10, 100, 4, mp.MP_SUM, FAKE,
                                 None, 0, None) == -1
    assert L.mp_message_backward(FAKE + 2, mp.MP_I32, None, FAKE, F32, 10, 100, 4, mp.MP_SUM,
                                 FAKE, None, 0, None) == -8
    assert L.mp_message_backward(FAKE, mp.MP_I32, None, FAKE, F32, 0, 100, 4, mp.MP_SUM, FAKE,
                                 FAKE, 1 << 20, None) == -2
    assert L.mp_message_backward(FAKE, mp.MP_I32, None, None, F32, 10, 0, 4, mp.MP_SUM, None,
                                 None, 0, None) == 0


def test_edge_dot_and_csr_rows_argument_errors():
    L = mp.lib()
    F32 = mp.MP_F32
    assert L.mp_edge_dot(FAKE, F32, FAKE, F32, None, 5, None, 10, 4, FAKE, None) == -2
    assert L.mp_edge_dot(FAKE, 3, FAKE, F32, FAKE, 5, None, 10, 4, FAKE, None) == -3
    assert L.mp_edge_dot(None, F32, FAKE, F32, FAKE, 5, None, 10, 4, FAKE, None) == -1
    assert L.mp_edge_dot(FAKE + 2, F32, FAKE, F32, FAKE, 5, None, 10, 4, FAKE, None) == -8
    assert L.mp_edge_dot(None, F32, None, F32, None, 0, None, 0, 4, None, None) == 0
    assert L.mp_csr_rows(FAKE, mp.MP_I32, 0, 10, FAKE, None) == -2
    assert L.mp_csr_rows(FAKE, mp.MP_I32, 5, 10, None, None) == -1
    assert L.mp_csr_rows(FAKE + 4, mp.MP_I64, 5, 10, FAKE, None) == -8
