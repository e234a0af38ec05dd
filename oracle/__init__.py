"""CPU oracle for the message-passing aggregation path (fp64, plain loops).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``, never by the device library or its
Python binding.  It shares no code with the device path; both are fed from
``graphgen``.

The arithmetic lives in ``oracle.c`` (see its header for the paper passages it
follows: Eq. (1), the sorted-CSR aggregation of Sec. 2.2, and the nested
heterogeneous sum).  This module only marshals numpy arrays.

Every function here is pinned by ``tests/test_oracle_*.py`` against library
routines (numpy stable argsort, scipy.sparse, dense matmul), closed forms and
brute force; none is "parity unpinned".
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "_liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c with gcc -O2 (no fast-math) + OpenMP."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                               _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _L():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        i64, i32, p = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p
        lib.oracle_coo_to_csr.argtypes = [i64, i64, i64, p, p, p, p, p, p, p]
        lib.oracle_coo_to_csr.restype = i32
        lib.oracle_spmm.argtypes = [i64, p, i64, i64, p, p, p, p, i32, i64,
                                    p, p, p, p, p, i32]
        lib.oracle_spmm.restype = i32
        lib.oracle_spmm_coo_rows.argtypes = [i64, i64, i64, p, p, p, p, i32, i64, i64, p,
                                             p, p, p, p, p, p]
        lib.oracle_spmm_coo_rows.restype = i32
        lib.oracle_hetero_sum.argtypes = [i32, p, p, i32, i64, i32, p, p, p, p, p, p, p]
        lib.oracle_hetero_sum.restype = i32
        lib.oracle_csr_rows.argtypes = [i64, i64, p, p, i64, p, p, p]
        lib.oracle_csr_rows.restype = i32
        lib.oracle_spmm_multi.argtypes = [i64, p, i64, i64, p, p, p, p, i32, i64, p, p, p, p,
                                          i32]
        lib.oracle_spmm_multi.restype = i32
        lib.oracle_segment_matmul.argtypes = [i32, p, p, p, i64, i64, p, p]
        lib.oracle_segment_matmul.restype = i32
        lib.oracle_segment_matmul_backward.argtypes = [i32, p, p, p, p, i64, i64, p, p, p, p]
        lib.oracle_segment_matmul_backward.restype = i32
        lib.oracle_csr_transpose.argtypes = [i64, i64, p, p, p, p, p]
        lib.oracle_csr_transpose.restype = i32
        lib.oracle_spmm_backward_x.argtypes = [i64, p, i64, i64, p, p, p, p, i32, i64, i32, p,
                                               p, p]
        lib.oracle_spmm_backward_x.restype = i32
        lib.oracle_spmm_backward_w.argtypes = [i64, p, i64, i64, p, p, p, i32, p, i32, i64, i32,
                                               p, p, p, i32]
        lib.oracle_spmm_backward_w.restype = i32
        lib.oracle_message_gather.argtypes = [i64, i64, p, p, p, i32, i64, p]
        lib.oracle_message_gather.restype = i32
        lib.oracle_message_scale.argtypes = [i64, i64, p, p, p, i64, p]
        lib.oracle_message_scale.restype = i32
        lib.oracle_message_backward.argtypes = [i64, p, p, i32, i64, i32, p, p]
        lib.oracle_message_backward.restype = i32
        lib.oracle_edge_dot.argtypes = [i64, i64, p, i32, p, i32, p, i64, p, p, p]
        lib.oracle_edge_dot.restype = i32
        lib.oracle_message_backward_x.argtypes = [i64, i64, p, p, p, i64, p, p]
        lib.oracle_message_backward_x.restype = i32
        _lib = lib
    return _lib


def default_threads() -> int:
    """Threads of the multithreaded oracle loops: OMP_NUM_THREADS when set,
    else the CPUs this process may run on."""
    n = int(os.environ.get("OMP_NUM_THREADS", "0") or 0)
    if n > 0:
        return n
    try:
        return len(os.sched_getaffinity(0)) or 1
    except AttributeError:
        return os.cpu_count() or 1


def _p(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _c(a, dt):
    return None if a is None else np.ascontiguousarray(a, dtype=dt)


def coo_to_csr(src, dst, n_dst, n_src=None, val=None):
    """Stable counting sort of the COO edges by destination.

    Returns (rowptr int64[N+1], col int32[E], perm int64[E], val_out or None)."""
    src, dst = _c(src, np.int32), _c(dst, np.int32)
    E = src.shape[0]
    n_src = n_dst if n_src is None else n_src
    rowptr = np.empty(n_dst + 1, np.int64)
    col = np.empty(E, np.int32)
    perm = np.empty(E, np.int64)
    val = _c(val, np.float32)
    vout = None if val is None else np.empty(E, np.float32)
    rc = _L().oracle_coo_to_csr(E, n_dst, n_src, _p(src), _p(dst), _p(val), _p(rowptr),
                                _p(col), _p(perm), _p(vout))
    if rc != 0:
        raise ValueError(f"oracle_coo_to_csr failed ({rc})")
    return rowptr, col, perm, vout


def _x_args(x, x_bf16):
    if x_bf16 is not None:
        xb = _c(x_bf16, np.uint16)
        return xb, 1, xb.shape[0], xb.shape[1]
    xf = _c(x, np.float32)
    return xf, 0, xf.shape[0], xf.shape[1]


def spmm(rowptr, col, x=None, x_bf16=None, w=None, rows=None, nthreads=None,
         want=("sum", "mean", "max", "scale")):
    """Aggregate every row (or the listed rows) of a destination-major CSR.

    x is fp32 [N_src, F] or x_bf16 is uint16 bit patterns.  w (fp32, CSR
    order) optional.  Returns a dict with the requested fp64 'sum', 'mean',
    'scale' and fp32 'max' + int64 'argmax' arrays of shape [rows, F]."""
    rowptr, col = _c(rowptr, np.int64), _c(col, np.int32)
    xa, isb, n_src, F = _x_args(x, x_bf16)
    n_dst = rowptr.shape[0] - 1
    rows = _c(rows, np.int64)
    n = n_dst if rows is None else rows.shape[0]
    w = _c(w, np.float32)
    out = {}
    s = np.empty((n, F), np.float64) if "sum" in want else None
    m = np.empty((n, F), np.float64) if "mean" in want else None
    mx = np.empty((n, F), np.float32) if "max" in want else None
    am = np.empty((n, F), np.int64) if "max" in want else None
    sc = np.empty((n, F), np.float64) if "scale" in want else None
    if nthreads is None:
        nthreads = default_threads()
    rc = _L().oracle_spmm(n, _p(rows), n_dst, n_src, _p(rowptr), _p(col), _p(w), _p(xa), isb,
                          F, _p(s), _p(m), _p(mx), _p(am), _p(sc), int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_spmm failed ({rc})")
    for k, v in (("sum", s), ("mean", m), ("max", mx), ("argmax", am), ("scale", sc)):
        if v is not None:
            out[k] = v
    return out


def spmm_multi(rowptr, col, x=None, x_bf16=None, w=None, rows=None, nthreads=None):
    """Min (+ first argmin), population variance, standard deviation and the
    variance error scale of every row (or the listed rows).  Returns a dict of
    'min' fp32, 'argmin' int64, 'var', 'std' fp64, shape [rows, F]."""
    rowptr, col = _c(rowptr, np.int64), _c(col, np.int32)
    xa, isb, n_src, F = _x_args(x, x_bf16)
    n_dst = rowptr.shape[0] - 1
    rows = _c(rows, np.int64)
    n = n_dst if rows is None else rows.shape[0]
    w = _c(w, np.float32)
    out = {"min": np.empty((n, F), np.float32), "argmin": np.empty((n, F), np.int64),
           "var": np.empty((n, F), np.float64), "std": np.empty((n, F), np.float64)}
    if nthreads is None:
        nthreads = default_threads()
    rc = _L().oracle_spmm_multi(n, _p(rows), n_dst, n_src, _p(rowptr), _p(col), _p(w), _p(xa),
                                isb, F, _p(out["min"]), _p(out["argmin"]), _p(out["var"]),
                                _p(out["std"]), int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_spmm_multi failed ({rc})")
    return out


def spmm_coo_rows(src, dst, n_dst, rows, x=None, x_bf16=None, w_coo=None, n_src=None,
                  row_start=None):
    """Outputs of the listed distinct rows, straight from COO (no CSR built).

    argmax is reported as a position in the stable destination-major CSR;
    row_start (optional, int64 per listed row) gives the number of edges
    whose destination is below each row, else it is counted here."""
    src, dst = _c(src, np.int32), _c(dst, np.int32)
    xa, isb, nx, F = _x_args(x, x_bf16)
    n_src = nx if n_src is None else n_src
    rows = _c(rows, np.int64)
    n = rows.shape[0]
    s = np.empty((n, F), np.float64)
    m = np.empty((n, F), np.float64)
    mx = np.empty((n, F), np.float32)
    am = np.empty((n, F), np.int64)
    sc = np.empty((n, F), np.float64)
    w_coo = _c(w_coo, np.float32)
    row_start = _c(row_start, np.int64)
    rc = _L().oracle_spmm_coo_rows(src.shape[0], n_dst, n_src, _p(src), _p(dst), _p(w_coo),
                                   _p(xa), isb, F, n, _p(rows), _p(row_start), _p(s), _p(m),
                                   _p(mx), _p(am), _p(sc))
    if rc != 0:
        raise ValueError(f"oracle_spmm_coo_rows failed ({rc})")
    return {"sum": s, "mean": m, "max": mx, "argmax": am, "scale": sc}


def csr_rows(src, dst, n_dst, rows):
    """Column segments of the listed distinct rows of the stable CSR, from COO.

    Returns (seg int64[len(rows)+1], cols int32[seg[-1]])."""
    src, dst = _c(src, np.int32), _c(dst, np.int32)
    rows = _c(rows, np.int64)
    n = rows.shape[0]
    seg = np.empty(n + 1, np.int64)
    rc = _L().oracle_csr_rows(src.shape[0], n_dst, _p(src), _p(dst), n, _p(rows), _p(seg), None)
    if rc != 0:
        raise ValueError(f"oracle_csr_rows failed ({rc})")
    cols = np.empty(int(seg[-1]), np.int32)
    rc = _L().oracle_csr_rows(src.shape[0], n_dst, _p(src), _p(dst), n, _p(rows), _p(seg),
                              _p(cols))
    if rc != 0:
        raise ValueError(f"oracle_csr_rows failed ({rc})")
    return seg, cols


def hetero_sum(n_per_type, x_bf16_per_type, rel_src_type, rel_dst_type, rel_src, rel_dst):
    """Nested sum: per destination type, the sum over its incoming relations of
    the per-relation sums.  Returns (out list fp64 [N_t, F], scale list)."""
    T = len(n_per_type)
    xs = [_c(x, np.uint16) for x in x_bf16_per_type]
    F = xs[0].shape[1]
    npt = np.asarray(n_per_type, np.int64)
    outs = [np.empty((n, F), np.float64) for n in n_per_type]
    scs = [np.empty((n, F), np.float64) for n in n_per_type]
    rs = [_c(a, np.int32) for a in rel_src]
    rd = [_c(a, np.int32) for a in rel_dst]
    R = len(rs)
    arr = lambda lst: (ctypes.c_void_p * len(lst))(*[a.ctypes.data for a in lst])
    # keep every temporary alive across the call
    rst = np.asarray(rel_src_type, np.int32)
    rdt = np.asarray(rel_dst_type, np.int32)
    re_ = np.asarray([a.shape[0] for a in rs], np.int64)
    rc = _L().oracle_hetero_sum(T, _p(npt), arr(xs), 1, F, R, _p(rst), _p(rdt), _p(re_),
                                arr(rs) if R else None, arr(rd) if R else None,
                                arr(outs), arr(scs))
    if rc != 0:
        raise ValueError(f"oracle_hetero_sum failed ({rc})")
    return outs, scs



REDUCE_CODES = {"sum": 1, "mean": 2, "max": 4}


def csr_transpose(rowptr, col, n_src):
    """Source-major CSR of the same edges, stable in forward CSR order.

    Returns (rowptrT int64[N_src+1], colT int32[E] = destination,
    posT int64[E] = forward CSR position)."""
    rowptr, col = _c(rowptr, np.int64), _c(col, np.int32)
    n_dst = rowptr.shape[0] - 1
    E = col.shape[0]
    rpt = np.empty(n_src + 1, np.int64)
    colt = np.empty(E, np.int32)
    post = np.empty(E, np.int64)
    rc = _L().oracle_csr_transpose(n_dst, n_src, _p(rowptr), _p(col), _p(rpt), _p(colt),
                                   _p(post))
    if rc != 0:
        raise ValueError(f"oracle_csr_transpose failed ({rc})")
    return rpt, colt, post


def _g_args(g, g_bf16):
    if g_bf16 is not None:
        gb = _c(g_bf16, np.uint16)
        return gb, 1, gb.shape[1]
    gf = _c(g, np.float32)
    return gf, 0, gf.shape[1]


def spmm_backward_x(rowptr, col, n_src, reduce, g=None, g_bf16=None, w=None, argout=None,
                    rows=None):
    """Gradient of the aggregation with respect to x (sum, mean or max).

    g (fp32 [N_dst, F], or g_bf16 bits) is the gradient of the output; w the
    CSR-order edge weights (optional); argout [N_dst, F] the forward argmax
    (max only).  Returns (gx fp64 [rows, F], scale fp64 [rows, F]) for the
    listed source rows (all when rows is None)."""
    rowptr, col = _c(rowptr, np.int64), _c(col, np.int32)
    ga, gisb, F = _g_args(g, g_bf16)
    n_dst = rowptr.shape[0] - 1
    rows = _c(rows, np.int64)
    n = n_src if rows is None else rows.shape[0]
    w = _c(w, np.float32)
    am = _c(argout, np.int64)
    gx = np.empty((n, F), np.float64)
    sc = np.empty((n, F), np.float64)
    rc = _L().oracle_spmm_backward_x(n, _p(rows), n_dst, n_src, _p(rowptr), _p(col), _p(w),
                                     _p(ga), gisb, F, REDUCE_CODES[reduce], _p(am), _p(gx),
                                     _p(sc))
    if rc != 0:
        raise ValueError(f"oracle_spmm_backward_x failed ({rc})")
    return gx, sc


def spmm_backward_w(rowptr, col, reduce, x=None, x_bf16=None, g=None, g_bf16=None,
                    argout=None, rows=None, nthreads=None):
    """Gradient of the aggregation with respect to the CSR-order edge weights.

    Returns (gw fp64 [E], scale fp64 [E]); with rows given, only the edges of
    those destination rows are filled (the rest are NaN)."""
    rowptr, col = _c(rowptr, np.int64), _c(col, np.int32)
    xa, xisb, n_src, F = _x_args(x, x_bf16)
    ga, gisb, Fg = _g_args(g, g_bf16)
    if Fg != F:
        raise ValueError("x and g widths differ")
    n_dst = rowptr.shape[0] - 1
    rows = _c(rows, np.int64)
    n = n_dst if rows is None else rows.shape[0]
    am = _c(argout, np.int64)
    E = col.shape[0]
    gw = np.full(E, np.nan, np.float64)
    sc = np.full(E, np.nan, np.float64)
    if nthreads is None:
        nthreads = default_threads()
    rc = _L().oracle_spmm_backward_w(n, _p(rows), n_dst, n_src, _p(rowptr), _p(col), _p(xa), xisb,
                                     _p(ga), gisb, F, REDUCE_CODES[reduce], _p(am), _p(gw),
                                     _p(sc), int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_spmm_backward_w failed ({rc})")
    return gw, sc


def segment_matmul(seg, x_bf16, w_bf16):
    """out[r] = x[r] @ W[t] for rows r of segment t (bf16 bits in, fp64 out).
    seg: [T+1] row offsets; x_bf16 [N, F]; w_bf16 [T, F, Fo].  Returns (out,
    scale) fp64 [N, Fo]."""
    seg = _c(seg, np.int64)
    x = _c(x_bf16, np.uint16)
    w = _c(w_bf16, np.uint16)
    T, F, Fo = w.shape
    N = x.shape[0]
    out = np.empty((N, Fo), np.float64)
    sc = np.empty((N, Fo), np.float64)
    rc = _L().oracle_segment_matmul(T, _p(seg), _p(x), _p(w), F, Fo, _p(out), _p(sc))
    if rc != 0:
        raise ValueError(f"oracle_segment_matmul failed ({rc})")
    return out, sc


def segment_matmul_backward(seg, x_bf16, w_bf16, dout_bf16):
    """Gradients of segment_matmul given dL/d out (bf16 bits [N, Fo]).
    Returns (dx, dx_scale [N, F], dw, dw_scale [T, F, Fo]) in fp64."""
    seg = _c(seg, np.int64)
    x = _c(x_bf16, np.uint16)
    w = _c(w_bf16, np.uint16)
    d = _c(dout_bf16, np.uint16)
    T, F, Fo = w.shape
    N = x.shape[0]
    dx, dxs = np.empty((N, F), np.float64), np.empty((N, F), np.float64)
    dw, dws = np.empty((T, F, Fo), np.float64), np.empty((T, F, Fo), np.float64)
    rc = _L().oracle_segment_matmul_backward(T, _p(seg), _p(x), _p(w), _p(d), F, Fo, _p(dx),
                                             _p(dxs), _p(dw), _p(dws))
    if rc != 0:
        raise ValueError(f"oracle_segment_matmul_backward failed ({rc})")
    return dx, dxs, dw, dws


# ---- edge-materialized messages (explanation mode) ------------------------------------

def message_gather(idx, x=None, x_bf16=None, w=None):
    """Materialized messages msg[p] = x[idx[p]] (or fl32(w[p] * x[idx[p]])),
    fp32 [E, F]; with idx = the CSR columns, row p is the message of CSR edge p."""
    idx = _c(idx, np.int32)
    xa, isb, n_src, F = _x_args(x, x_bf16)
    E = idx.shape[0]
    w = _c(w, np.float32)
    msg = np.empty((E, F), np.float32)
    rc = _L().oracle_message_gather(E, n_src, _p(idx), _p(w), _p(xa), isb, F, _p(msg))
    if rc != 0:
        raise ValueError(f"oracle_message_gather failed ({rc})")
    return msg


def message_scale(msg, mask, idx=None):
    """The edge-mask callback: out[p] = fl32(msg[p] * mask[idx[p]]) (idx None:
    mask[p]).  Returns a new fp32 [E, F] array."""
    msg = _c(msg, np.float32)
    mask = _c(mask, np.float32)
    idx = _c(idx, np.int32)
    E, F = msg.shape
    out = np.empty_like(msg)
    rc = _L().oracle_message_scale(E, F, _p(msg), _p(mask), _p(idx), mask.shape[0], _p(out))
    if rc != 0:
        raise ValueError(f"oracle_message_scale failed ({rc})")
    return out


def aggregate_messages(rowptr, msg=None, msg_bf16=None, rows=None, nthreads=None,
                       want=("sum", "mean", "max", "scale")):
    """Aggregation of materialized messages: row v reduces the message rows
    rowptr[v] .. rowptr[v+1] - 1 (the aggregation of ``spmm`` with column p at
    position p, so argmax is a message row)."""
    rowptr = _c(rowptr, np.int64)
    E = int(rowptr[-1])
    ident = np.arange(E, dtype=np.int32)
    return spmm(rowptr, ident, x=msg, x_bf16=msg_bf16, rows=rows, nthreads=nthreads, want=want)


def spmm_materialized(rowptr, col, x=None, x_bf16=None, w=None, callback=None,
                      want=("sum", "mean", "max", "scale")):
    """Explanation-mode aggregation: materialize the messages, apply the
    callback c (a function of the fp32 [E, F] message table returning one of
    the same shape; None: identity), aggregate.  Returns (aggregates, msg)."""
    msg = message_gather(col, x=x, x_bf16=x_bf16, w=w)
    if callback is not None:
        msg = np.ascontiguousarray(callback(msg), dtype=np.float32)
    return aggregate_messages(rowptr, msg, want=want), msg


def message_backward(rowptr, reduce, g=None, g_bf16=None, argout=None):
    """dL/dmsg [E, F] fp32 of the aggregation of materialized messages, given
    g = dL/d out (fp32, or g_bf16 bits) and, for max, the forward argout."""
    rowptr = _c(rowptr, np.int64)
    ga, gisb, F = _g_args(g, g_bf16)
    n_dst = rowptr.shape[0] - 1
    E = int(rowptr[-1])
    am = _c(argout, np.int64)
    dmsg = np.empty((E, F), np.float32)
    rc = _L().oracle_message_backward(n_dst, _p(rowptr), _p(ga), gisb, F, REDUCE_CODES[reduce],
                                      _p(am), _p(dmsg))
    if rc != 0:
        raise ValueError(f"oracle_message_backward failed ({rc})")
    return dmsg


def edge_dot(a=None, a_bf16=None, b=None, b_bf16=None, bidx=None, oidx=None):
    """out[oidx[p]] = sum_f a[p, f] * b[bidx[p], f] (fp64; None indices are
    the identity).  Returns (out [E], scale [E])."""
    aa, aisb, E, F = _x_args(a, a_bf16)
    ba, bisb, n_b, Fb = _x_args(b, b_bf16)
    if Fb != F:
        raise ValueError("a and b widths differ")
    bidx, oidx = _c(bidx, np.int32), _c(oidx, np.int32)
    out = np.empty(E, np.float64)
    sc = np.empty(E, np.float64)
    rc = _L().oracle_edge_dot(E, F, _p(aa), aisb, _p(ba), bisb, _p(bidx), n_b, _p(oidx),
                              _p(out), _p(sc))
    if rc != 0:
        raise ValueError(f"oracle_edge_dot failed ({rc})")
    return out, sc


def message_backward_x(col, n_src, dmsg, w=None):
    """dL/dx [N_src, F] fp64 of the messages w[p] * x[col[p]] given dL/dmsg,
    summed per source in CSR order.  Returns (gx, scale)."""
    col = _c(col, np.int32)
    dmsg = _c(dmsg, np.float32)
    w = _c(w, np.float32)
    E, F = dmsg.shape
    gx = np.empty((n_src, F), np.float64)
    sc = np.empty((n_src, F), np.float64)
    rc = _L().oracle_message_backward_x(E, n_src, _p(col), _p(w), _p(dmsg), F, _p(gx), _p(sc))
    if rc != 0:
        raise ValueError(f"oracle_message_backward_x failed ({rc})")
    return gx, sc
