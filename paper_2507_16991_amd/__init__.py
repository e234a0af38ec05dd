"""Python binding of libmp, the MI355X message-passing aggregation library.

Argument marshalling only: every step of the path runs in the HIP kernels of
``libmp.so`` (built from ``csrc/`` by ``build.py``).  Tensors are torch
tensors on the GPU; torch supplies device memory and the current stream.
There is no fallback: if the library is missing, importing the binding's
entry points raises.

Two layers:
  * ``mp_*`` functions with the names of the C ABI (``include/mp.h``), taking
    tensors or None for pointers and raising ``MPError`` on a non-zero status;
  * convenience wrappers (``coo_to_csr``, ``Plan``, ``spmm``, ``hetero_build``,
    ``hetero_spmm``) that size and allocate outputs and workspaces with torch.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "MPError", "lib", "MP_F32", "MP_BF16", "MP_I32", "MP_I64", "MP_SUM", "MP_MEAN", "MP_MAX",
    "mp_version", "mp_status_str", "mp_coo_to_csr_workspace", "mp_coo_to_csr",
    "mp_sorted_coo_to_csr", "mp_validate_sorted", "sorted_coo_to_csr",
    "mp_csr_transpose_workspace", "mp_csr_transpose", "mp_spmm_backward_x_workspace",
    "mp_spmm_backward_x", "mp_spmm_backward_w_workspace", "mp_spmm_backward_w",
    "csr_transpose", "spmm_backward_x", "spmm_backward_w", "MP_MIN", "MP_VAR", "MP_STD", "AGGR",
    "mp_aggr_out", "mp_spmm_multi_workspace", "mp_spmm_multi", "mp_readout_multi", "spmm_multi",
    "readout", "mp_segment_matmul_workspace", "mp_segment_matmul",
    "mp_segment_matmul_backward_workspace", "mp_segment_matmul_backward", "segment_matmul",
    "segment_matmul_backward",
    "mp_spmm_plan_size", "mp_spmm_plan_build", "mp_spmm_plan_free", "mp_spmm_workspace",
    "mp_spmm", "mp_hetero_build_workspace", "mp_hetero_build", "mp_hetero_spmm",
    "mp_validate_coo", "mp_validate_csr", "coo_to_csr", "Plan", "spmm", "hetero_build",
    "hetero_spmm", "LIB_PATH", "MESSAGE_FN", "mp_csr_rows", "mp_message_gather",
    "mp_message_scale", "mp_message_aggregate", "mp_spmm_materialized",
    "mp_message_backward_workspace", "mp_message_backward", "mp_edge_dot", "csr_rows",
    "message_gather", "message_scale", "message_aggregate", "spmm_materialized",
    "message_backward", "edge_dot", "mp_copy_rows", "aligned_ld", "pad_rows", "MP_MAX_TYPES",
    "MP_ALL_TYPES", "MP_ERR_SORT", "mp_plan_opts", "mp_spmm_plan_build_opts", "new_status",
    "check_status", "mp_spmm_noalloc", "MP_NOALLOC_SCRATCH_BYTES", "mp_probe_read",
    "mp_probe_copy", "mp_probe_gather", "mp_probe_scatter", "MP_PROBE_SINK_WORDS",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmp.so")

MP_OK = 0
MP_F32, MP_BF16 = 0, 1
MP_I32, MP_I64 = 0, 1
MP_SUM, MP_MEAN, MP_MAX = 1, 2, 4
MP_MIN, MP_VAR, MP_STD = 8, 16, 32
AGGR = {"sum": MP_SUM, "mean": MP_MEAN, "max": MP_MAX, "min": MP_MIN, "var": MP_VAR,
        "std": MP_STD}
MP_MAX_TYPES = 16
MP_ALL_TYPES = -1  # dst_type selecting every destination type at once
MP_ERR_CALLBACK = -9
MP_ERR_SORT = -10
MP_NOALLOC_SCRATCH_BYTES = 64 << 20  # the static scratch of mp_spmm_noalloc, per GPU
MP_PROBE_SINK_WORDS = 65536  # uint32 words of a bandwidth probe's sink

# int c(void* msg, int msg_dtype, int64_t E, int64_t F, void* user, void* stream)
MESSAGE_FN = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_void_p, ctypes.c_int, ctypes.c_int64,
                              ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p)

_lib = None


class MPError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {status} ({mp_status_str(status)})")
        self.status = status


class mp_relation(ctypes.Structure):
    _fields_ = [("src_type", ctypes.c_int32), ("dst_type", ctypes.c_int32),
                ("src", ctypes.c_void_p), ("dst", ctypes.c_void_p), ("E", ctypes.c_int64)]


class mp_plan_opts(ctypes.Structure):
    _fields_ = [("small_max", ctypes.c_int64), ("hub_min", ctypes.c_int64),
                ("chunk_min", ctypes.c_int64)]


class mp_aggr_out(ctypes.Structure):
    _fields_ = [("aggr", ctypes.c_int), ("out", ctypes.c_void_p), ("arg", ctypes.c_void_p)]


def lib():
    """The loaded libmp.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2507_16991_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        i32, i64, p, sz = ctypes.c_int, ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t
        psz = ctypes.POINTER(ctypes.c_size_t)
        L.mp_version.restype = i32
        L.mp_status_str.argtypes = [i32]
        L.mp_status_str.restype = ctypes.c_char_p
        L.mp_coo_to_csr_workspace.argtypes = [i64, i64, i32, i32, psz]
        L.mp_coo_to_csr.argtypes = [p, p, i64, i64, p, i32, p, p, p, p, p, sz, p, p]
        L.mp_sorted_coo_to_csr.argtypes = [p, p, i64, i64, p, i32, p, p, p, p, p]
        L.mp_spmm_plan_size.argtypes = [i64, i64, psz]
        L.mp_spmm_plan_build.argtypes = [p, i32, i64, i64, i64, i32, p, sz, p,
                                         ctypes.POINTER(ctypes.c_void_p)]
        L.mp_spmm_plan_build_opts.argtypes = [p, i32, i64, i64, i64, i32, p, sz, p, p,
                                              ctypes.POINTER(ctypes.c_void_p)]
        L.mp_spmm_plan_free.argtypes = [p]
        L.mp_spmm_plan_free.restype = None
        L.mp_spmm_workspace.argtypes = [p, i32, psz]
        L.mp_spmm.argtypes = [p, p, i32, p, p, p, i32, i64, i64, i64, i64, i32, p, i32, p, i32, p,
                              p, sz, p]
        L.mp_spmm_noalloc.argtypes = [p, p, i32, p, p, p, i32, i64, i64, i64, i64, i32, p, i32,
                                      p, i32, p, p]
        L.mp_copy_rows.argtypes = [p, i64, p, i64, i64, i64, i32, p]
        L.mp_probe_read.argtypes = [p, i64, p, p]
        L.mp_probe_copy.argtypes = [p, p, i64, p]
        L.mp_probe_gather.argtypes = [p, i64, p, i64, i64, p, p]
        L.mp_probe_scatter.argtypes = [p, p, i64, i64, p, p]
        L.mp_hetero_build_workspace.argtypes = [i32, p, i32, p, i32, i32, psz]
        L.mp_hetero_build.argtypes = [i32, p, i32, p, i32, p, i32, p, p, sz, p, p]
        L.mp_hetero_spmm.argtypes = [i32, p, p, i32, i64, i32, p, p, i32, p, i32, p, i32, p, sz,
                                     p]
        L.mp_validate_coo.argtypes = [p, p, i64, i64, i64, p, p]
        L.mp_validate_csr.argtypes = [p, i32, p, i64, i64, i64, p, p]
        L.mp_validate_sorted.argtypes = [p, i64, p, p]
        L.mp_segment_matmul_workspace.argtypes = [i32, i64, i64, psz]
        L.mp_segment_matmul.argtypes = [p, i32, p, p, i64, i64, p, i32, p, sz, p]
        L.mp_segment_matmul_backward_workspace.argtypes = [p, i32, i64, i64, psz]
        L.mp_segment_matmul_backward.argtypes = [p, i32, p, p, p, i64, i64, p, i32, p, p, sz, p]
        L.mp_spmm_multi_workspace.argtypes = [p, psz]
        L.mp_spmm_multi.argtypes = [p, p, i32, p, p, p, i32, i64, i64, i64, i64, i32, p, p, sz,
                                    p]
        L.mp_readout_multi.argtypes = [p, p, i32, p, i32, i64, i64, i64, i64, i32, p, p, sz, p]
        L.mp_csr_transpose_workspace.argtypes = [i64, i64, i32, i32, psz]
        L.mp_csr_transpose.argtypes = [p, i32, p, i64, i64, i64, p, i32, p, p, p, p, p, sz, p,
                                       p]
        L.mp_spmm_backward_x_workspace.argtypes = [p, i64, i64, i64, i32, psz]
        L.mp_spmm_backward_x.argtypes = [p, p, i32, p, p, p, p, i32, p, p, i32, i64, i64, i64,
                                         i64, i32, p, i32, p, sz, p]
        L.mp_spmm_backward_w_workspace.argtypes = [i64, psz]
        L.mp_spmm_backward_w.argtypes = [p, i32, p, p, i32, p, i32, p, i64, i64, i64, i64, i32, p,
                                         p, sz, p]
        L.mp_csr_rows.argtypes = [p, i32, i64, i64, p, p]
        L.mp_message_gather.argtypes = [p, p, p, i32, i64, i64, i64, p, i32, p]
        L.mp_message_scale.argtypes = [p, p, i64, i64, p, p, i64, p]
        L.mp_message_aggregate.argtypes = [p, p, i32, p, i32, i64, i64, i64, i32, p, i32, p, i32,
                                           p, p, sz, p]
        L.mp_spmm_materialized.argtypes = [p, p, i32, p, p, p, i32, i64, i64, i64, i64, p, i32,
                                           p, p, i32, p, i32, p, i32, p, p, sz, p]
        L.mp_message_backward_workspace.argtypes = [i64, psz]
        L.mp_message_backward.argtypes = [p, i32, p, p, i32, i64, i64, i64, i32, p, p, sz, p]
        L.mp_edge_dot.argtypes = [p, i32, p, i32, p, i64, p, i64, i64, p, p]
        for name in ("mp_copy_rows", "mp_csr_rows", "mp_message_gather", "mp_message_scale",
                     "mp_message_aggregate", "mp_spmm_materialized",
                     "mp_message_backward_workspace", "mp_message_backward", "mp_edge_dot",
                     "mp_coo_to_csr_workspace", "mp_coo_to_csr", "mp_sorted_coo_to_csr",
                     "mp_validate_sorted", "mp_csr_transpose_workspace", "mp_csr_transpose",
                     "mp_spmm_multi_workspace", "mp_spmm_multi", "mp_readout_multi",
                     "mp_segment_matmul_workspace", "mp_segment_matmul",
                     "mp_segment_matmul_backward_workspace", "mp_segment_matmul_backward",
                     "mp_spmm_backward_x_workspace", "mp_spmm_backward_x",
                     "mp_spmm_backward_w_workspace", "mp_spmm_backward_w", "mp_spmm_plan_size",
                     "mp_spmm_plan_build", "mp_spmm_plan_build_opts", "mp_spmm_workspace",
                     "mp_spmm", "mp_spmm_noalloc", "mp_probe_read", "mp_probe_copy",
                     "mp_probe_gather", "mp_probe_scatter",
                     "mp_hetero_build_workspace", "mp_hetero_build", "mp_hetero_spmm",
                     "mp_validate_coo", "mp_validate_csr"):
            getattr(L, name).restype = i32
        _lib = L
    return _lib


# ---- marshalling helpers ------------------------------------------------------

def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_contiguous():
        raise ValueError("tensors passed to libmp must be contiguous")
    if t.numel() == 0:
        # torch reports 0 for an empty tensor; pass its storage address (NULL
        # only when nothing was ever allocated, see _edge_array)
        return t.untyped_storage().data_ptr() + t.storage_offset() * t.element_size() or None
    return t.data_ptr()


def _rows_ptr(t):
    """Address of a 2-D table whose rows may be strided (stride(1) == 1,
    stride(0) >= shape[1]), and that stride in elements."""
    if t.dim() != 2 or (t.shape[0] > 1 and t.stride(1) != 1) or t.stride(0) < t.shape[1]:
        raise ValueError("feature tables passed to libmp must have unit column stride")
    if t.numel() == 0:
        return _ptr(t.contiguous()), int(t.shape[1])
    return t.data_ptr(), int(t.stride(0)) if t.shape[0] > 1 else int(t.shape[1])


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def _dtype_code(dt):
    if dt == torch.float32:
        return MP_F32
    if dt == torch.bfloat16:
        return MP_BF16
    raise ValueError(f"unsupported feature dtype {dt}")


def _itype_code(dt):
    if dt == torch.int32:
        return MP_I32
    if dt == torch.int64:
        return MP_I64
    raise ValueError(f"unsupported rowptr dtype {dt}")


def _check(fn, st):
    if st != MP_OK:
        raise MPError(fn, st)


def _bytes(fn, *args):
    b = ctypes.c_size_t(0)
    _check(fn, getattr(lib(), fn)(*args, ctypes.byref(b)))
    return b.value


def _edge_array(E, dtype, device):
    """[E] tensor whose storage holds at least one element, so that its data
    pointer is never NULL (an empty graph still passes valid pointers)."""
    return torch.empty(max(E, 1), dtype=dtype, device=device)[:E]


def _workspace(nbytes, device):
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


# ---- C ABI names ---------------------------------------------------------------

def mp_version() -> int:
    return lib().mp_version()


def mp_status_str(status: int) -> str:
    return lib().mp_status_str(status).decode()


def mp_coo_to_csr_workspace(E, N, rowptr_itype, with_payload) -> int:
    return _bytes("mp_coo_to_csr_workspace", E, N, rowptr_itype, int(with_payload))


def mp_coo_to_csr(src, dst, E, N, rowptr, rowptr_itype, col, perm, val_in, val_out, ws,
                  ws_bytes, status=None, stream=None):
    _check("mp_coo_to_csr", lib().mp_coo_to_csr(
        _ptr(src), _ptr(dst), E, N, _ptr(rowptr), rowptr_itype, _ptr(col), _ptr(perm),
        _ptr(val_in), _ptr(val_out), _ptr(ws), ws_bytes, _ptr(status), _stream(stream)))


def mp_sorted_coo_to_csr(src, dst, E, N, rowptr, rowptr_itype, col, perm, val_in, val_out,
                         stream=None):
    _check("mp_sorted_coo_to_csr", lib().mp_sorted_coo_to_csr(
        _ptr(src), _ptr(dst), E, N, _ptr(rowptr), rowptr_itype, _ptr(col), _ptr(perm),
        _ptr(val_in), _ptr(val_out), _stream(stream)))


def mp_spmm_plan_size(N_dst, E) -> int:
    return _bytes("mp_spmm_plan_size", N_dst, E)


def mp_spmm_plan_build(rowptr, rowptr_itype, N_dst, E, F, x_dtype, plan_buf, plan_bytes,
                       stream=None) -> int:
    h = ctypes.c_void_p(0)
    _check("mp_spmm_plan_build", lib().mp_spmm_plan_build(
        _ptr(rowptr), rowptr_itype, N_dst, E, F, x_dtype, _ptr(plan_buf), plan_bytes,
        _stream(stream), ctypes.byref(h)))
    return h.value


def mp_spmm_plan_build_opts(rowptr, rowptr_itype, N_dst, E, F, x_dtype, plan_buf, plan_bytes,
                            opts=None, stream=None) -> int:
    """opts: None, or (small_max, hub_min, chunk_min) with 0 for a default."""
    h = ctypes.c_void_p(0)
    o = ctypes.byref(mp_plan_opts(*[int(v) for v in opts])) if opts is not None else None
    _check("mp_spmm_plan_build_opts", lib().mp_spmm_plan_build_opts(
        _ptr(rowptr), rowptr_itype, N_dst, E, F, x_dtype, _ptr(plan_buf), plan_bytes, o,
        _stream(stream), ctypes.byref(h)))
    return h.value


def mp_spmm_plan_free(handle) -> None:
    lib().mp_spmm_plan_free(handle)


def mp_spmm_workspace(plan_handle, reduce) -> int:
    return _bytes("mp_spmm_workspace", plan_handle, reduce)


def mp_spmm(plan_handle, rowptr, rowptr_itype, col, w, x, x_dtype, N_src, N_dst, F, ldx, reduce,
            out, out_dtype, out_max, max_dtype, argout, ws, ws_bytes, stream=None):
    """x: a tensor (its row stride is used when strided) or a raw address."""
    xp = _rows_ptr(x)[0] if isinstance(x, torch.Tensor) else x
    _check("mp_spmm", lib().mp_spmm(
        plan_handle, _ptr(rowptr), rowptr_itype, _ptr(col), _ptr(w), xp, x_dtype, N_src,
        N_dst, F, ldx, reduce, _ptr(out), out_dtype, _ptr(out_max), max_dtype, _ptr(argout),
        _ptr(ws), ws_bytes, _stream(stream)))


def mp_spmm_noalloc(plan_handle, rowptr, rowptr_itype, col, w, x, x_dtype, N_src, N_dst, F,
                    ldx, reduce, out, out_dtype, out_max, max_dtype, argout, stream=None):
    """mp_spmm for callers that cannot allocate: no workspace argument (the
    library's static per-GPU scratch array holds the hub partials)."""
    xp = _rows_ptr(x)[0] if isinstance(x, torch.Tensor) else x
    _check("mp_spmm_noalloc", lib().mp_spmm_noalloc(
        plan_handle, _ptr(rowptr), rowptr_itype, _ptr(col), _ptr(w), xp, x_dtype, N_src, N_dst,
        F, ldx, reduce, _ptr(out), out_dtype, _ptr(out_max), max_dtype, _ptr(argout),
        _stream(stream)))


def mp_probe_read(p, nbytes, sink, stream=None):
    _check("mp_probe_read", lib().mp_probe_read(_ptr(p), nbytes, _ptr(sink), _stream(stream)))


def mp_probe_copy(src, dst, nbytes, stream=None):
    _check("mp_probe_copy", lib().mp_probe_copy(_ptr(src), _ptr(dst), nbytes, _stream(stream)))


def mp_probe_gather(idx, n, table, stride_bytes, row_bytes, sink, stream=None):
    """table: a tensor (its data address) or a raw address."""
    tp = table.data_ptr() if isinstance(table, torch.Tensor) else table
    _check("mp_probe_gather", lib().mp_probe_gather(_ptr(idx), n, tp, stride_bytes, row_bytes,
                                                    _ptr(sink), _stream(stream)))


def mp_probe_scatter(src, dest, n, elem_bytes, out, stream=None):
    _check("mp_probe_scatter", lib().mp_probe_scatter(_ptr(src), _ptr(dest), n, elem_bytes,
                                                      _ptr(out), _stream(stream)))


def mp_copy_rows(x_in, ld_in, x_out, ld_out, N, F, dtype, stream=None):
    pi = _rows_ptr(x_in)[0] if isinstance(x_in, torch.Tensor) else x_in
    po = _rows_ptr(x_out)[0] if isinstance(x_out, torch.Tensor) else x_out
    _check("mp_copy_rows", lib().mp_copy_rows(pi, ld_in, po, ld_out, N, F, dtype,
                                              _stream(stream)))


def _rel_array(rels):
    arr = (mp_relation * max(len(rels), 1))()
    for k, (st, dt, s, d) in enumerate(rels):
        arr[k] = mp_relation(st, dt, _ptr(s), _ptr(d), int(s.numel()))
    return arr


def mp_hetero_build_workspace(N_per_type, rels, dst_type, rowptr_itype) -> int:
    npt = (ctypes.c_int64 * len(N_per_type))(*N_per_type)
    return _bytes("mp_hetero_build_workspace", len(N_per_type), npt, len(rels), _rel_array(rels),
                  dst_type, rowptr_itype)


def mp_hetero_build(N_per_type, rels, dst_type, rowptr, rowptr_itype, col, ws, ws_bytes,
                    status=None, stream=None):
    npt = (ctypes.c_int64 * len(N_per_type))(*N_per_type)
    _check("mp_hetero_build", lib().mp_hetero_build(
        len(N_per_type), npt, len(rels), _rel_array(rels), dst_type, _ptr(rowptr), rowptr_itype,
        _ptr(col), _ptr(ws), ws_bytes, _ptr(status), _stream(stream)))


def mp_hetero_spmm(N_per_type, x_per_type, x_dtype, F, dst_type, plan_handle, rowptr,
                   rowptr_itype, col, reduce, out, out_dtype, ws, ws_bytes, stream=None):
    T = len(N_per_type)
    npt = (ctypes.c_int64 * T)(*N_per_type)
    xs = (ctypes.c_void_p * T)(*[_ptr(x) for x in x_per_type])
    _check("mp_hetero_spmm", lib().mp_hetero_spmm(
        T, npt, xs, x_dtype, F, dst_type, plan_handle, _ptr(rowptr), rowptr_itype, _ptr(col),
        reduce, _ptr(out), out_dtype, _ptr(ws), ws_bytes, _stream(stream)))


def mp_validate_coo(src, dst, E, N_src, N_dst, d_count, stream=None):
    _check("mp_validate_coo", lib().mp_validate_coo(_ptr(src), _ptr(dst), E, N_src, N_dst,
                                                    _ptr(d_count), _stream(stream)))


def mp_csr_transpose_workspace(E, N_src, rowptrT_itype, with_payload) -> int:
    return _bytes("mp_csr_transpose_workspace", E, N_src, rowptrT_itype, int(with_payload))


def mp_csr_transpose(rowptr, rowptr_itype, col, N_dst, N_src, E, rowptrT, rowptrT_itype, colT,
                     posT, val_in, val_out, ws, ws_bytes, status=None, stream=None):
    _check("mp_csr_transpose", lib().mp_csr_transpose(
        _ptr(rowptr), rowptr_itype, _ptr(col), N_dst, N_src, E, _ptr(rowptrT), rowptrT_itype,
        _ptr(colT), _ptr(posT), _ptr(val_in), _ptr(val_out), _ptr(ws), ws_bytes, _ptr(status),
        _stream(stream)))


def mp_spmm_backward_x_workspace(planT_handle, N_dst, E, F, reduce) -> int:
    return _bytes("mp_spmm_backward_x_workspace", planT_handle, N_dst, E, F, reduce)


def mp_spmm_backward_x(planT_handle, rowptrT, rowptrT_itype, colT, posT, wT, rowptr,
                       rowptr_itype, argout, grad_out, g_dtype, N_dst, N_src, E, F, reduce,
                       grad_x, out_dtype, ws, ws_bytes, stream=None):
    _check("mp_spmm_backward_x", lib().mp_spmm_backward_x(
        planT_handle, _ptr(rowptrT), rowptrT_itype, _ptr(colT), _ptr(posT), _ptr(wT),
        _ptr(rowptr), rowptr_itype, _ptr(argout), _ptr(grad_out), g_dtype, N_dst, N_src, E, F,
        reduce, _ptr(grad_x), out_dtype, _ptr(ws), ws_bytes, _stream(stream)))


def mp_spmm_backward_w_workspace(E) -> int:
    return _bytes("mp_spmm_backward_w_workspace", E)


def mp_spmm_backward_w(rowptr, rowptr_itype, col, x, x_dtype, grad_out, g_dtype, argout, N_src,
                       N_dst, E, F, reduce, grad_w, ws, ws_bytes, stream=None):
    _check("mp_spmm_backward_w", lib().mp_spmm_backward_w(
        _ptr(rowptr), rowptr_itype, _ptr(col), _ptr(x), x_dtype, _ptr(grad_out), g_dtype,
        _ptr(argout), N_src, N_dst, E, F, reduce, _ptr(grad_w), _ptr(ws), ws_bytes,
        _stream(stream)))


def mp_spmm_multi_workspace(plan_handle) -> int:
    return _bytes("mp_spmm_multi_workspace", plan_handle)


def _aggr_array(outs):
    """outs: list of (aggr code, out tensor, arg tensor or None)."""
    arr = (mp_aggr_out * len(outs))()
    for k, (a, o, g) in enumerate(outs):
        arr[k].aggr, arr[k].out, arr[k].arg = a, _ptr(o), _ptr(g)
    return arr


def mp_spmm_multi(plan_handle, rowptr, rowptr_itype, col, w, x, x_dtype, N_src, N_dst, F, ldx,
                  outs, ws, ws_bytes, stream=None):
    arr = _aggr_array(outs)
    xp = _rows_ptr(x)[0] if isinstance(x, torch.Tensor) else x
    _check("mp_spmm_multi", lib().mp_spmm_multi(
        plan_handle, _ptr(rowptr), rowptr_itype, _ptr(col), _ptr(w), xp, x_dtype, N_src,
        N_dst, F, ldx, len(outs), arr, _ptr(ws), ws_bytes, _stream(stream)))


def mp_readout_multi(plan_handle, ptr, ptr_itype, x, x_dtype, N_nodes, N_seg, F, ldx, outs, ws,
                     ws_bytes, stream=None):
    arr = _aggr_array(outs)
    xp = _rows_ptr(x)[0] if isinstance(x, torch.Tensor) else x
    _check("mp_readout_multi", lib().mp_readout_multi(
        plan_handle, _ptr(ptr), ptr_itype, xp, x_dtype, N_nodes, N_seg, F, ldx, len(outs), arr,
        _ptr(ws), ws_bytes, _stream(stream)))


def _seg_array(seg):
    a = (ctypes.c_int64 * len(seg))(*[int(v) for v in seg])
    return a


def mp_segment_matmul_workspace(T, F, Fo) -> int:
    return _bytes("mp_segment_matmul_workspace", T, F, Fo)


def mp_segment_matmul(seg, T, x, W, F, Fo, out, out_dtype, ws, ws_bytes, stream=None):
    _check("mp_segment_matmul", lib().mp_segment_matmul(
        _seg_array(seg), T, _ptr(x), _ptr(W), F, Fo, _ptr(out), out_dtype, _ptr(ws), ws_bytes,
        _stream(stream)))


def mp_segment_matmul_backward_workspace(seg, T, F, Fo) -> int:
    return _bytes("mp_segment_matmul_backward_workspace", _seg_array(seg), T, F, Fo)


def mp_segment_matmul_backward(seg, T, x, W, dout, F, Fo, dx, dx_dtype, dW, ws, ws_bytes,
                               stream=None):
    _check("mp_segment_matmul_backward", lib().mp_segment_matmul_backward(
        _seg_array(seg), T, _ptr(x), _ptr(W), _ptr(dout), F, Fo, _ptr(dx), dx_dtype, _ptr(dW),
        _ptr(ws), ws_bytes, _stream(stream)))


def mp_validate_sorted(dst, E, d_count, stream=None):
    _check("mp_validate_sorted", lib().mp_validate_sorted(_ptr(dst), E, _ptr(d_count),
                                                          _stream(stream)))


def mp_validate_csr(rowptr, rowptr_itype, col, N_dst, N_src, E, d_count, stream=None):
    _check("mp_validate_csr", lib().mp_validate_csr(_ptr(rowptr), rowptr_itype, _ptr(col), N_dst,
                                                    N_src, E, _ptr(d_count), _stream(stream)))


def mp_csr_rows(rowptr, rowptr_itype, N_dst, E, row, stream=None):
    _check("mp_csr_rows", lib().mp_csr_rows(_ptr(rowptr), rowptr_itype, N_dst, E, _ptr(row),
                                            _stream(stream)))


def mp_message_gather(idx, w, x, x_dtype, N_src, E, F, msg, msg_dtype, stream=None):
    _check("mp_message_gather", lib().mp_message_gather(
        _ptr(idx), _ptr(w), _ptr(x), x_dtype, N_src, E, F, _ptr(msg), msg_dtype, _stream(stream)))


def mp_message_scale(msg_in, msg_out, E, F, mask, idx, n_mask, stream=None):
    _check("mp_message_scale", lib().mp_message_scale(
        _ptr(msg_in), _ptr(msg_out), E, F, _ptr(mask), _ptr(idx), n_mask, _stream(stream)))


def mp_message_aggregate(plan_handle, rowptr, rowptr_itype, msg, msg_dtype, E, N_dst, F, reduce,
                         out, out_dtype, out_max, max_dtype, argout, ws, ws_bytes, stream=None):
    _check("mp_message_aggregate", lib().mp_message_aggregate(
        plan_handle, _ptr(rowptr), rowptr_itype, _ptr(msg), msg_dtype, E, N_dst, F, reduce,
        _ptr(out), out_dtype, _ptr(out_max), max_dtype, _ptr(argout), _ptr(ws), ws_bytes,
        _stream(stream)))


def mp_spmm_materialized(plan_handle, rowptr, rowptr_itype, col, w, x, x_dtype, N_src, N_dst, E,
                         F, msg, msg_dtype, c, user, reduce, out, out_dtype, out_max, max_dtype,
                         argout, ws, ws_bytes, stream=None):
    """c: a MESSAGE_FN (keep a reference to it for the call), a function
    address, or None."""
    if isinstance(c, int):
        c = ctypes.cast(c, MESSAGE_FN)
    _check("mp_spmm_materialized", lib().mp_spmm_materialized(
        plan_handle, _ptr(rowptr), rowptr_itype, _ptr(col), _ptr(w), _ptr(x), x_dtype, N_src,
        N_dst, E, F, _ptr(msg), msg_dtype, ctypes.cast(c, ctypes.c_void_p) if c else None, user,
        reduce, _ptr(out), out_dtype, _ptr(out_max), max_dtype, _ptr(argout), _ptr(ws), ws_bytes,
        _stream(stream)))


def mp_message_backward_workspace(E) -> int:
    return _bytes("mp_message_backward_workspace", E)


def mp_message_backward(rowptr, rowptr_itype, argout, grad_out, g_dtype, N_dst, E, F, reduce,
                        dmsg, ws, ws_bytes, stream=None):
    _check("mp_message_backward", lib().mp_message_backward(
        _ptr(rowptr), rowptr_itype, _ptr(argout), _ptr(grad_out), g_dtype, N_dst, E, F, reduce,
        _ptr(dmsg), _ptr(ws), ws_bytes, _stream(stream)))


def mp_edge_dot(a, a_dtype, b, b_dtype, bidx, N_b, oidx, E, F, out, stream=None):
    _check("mp_edge_dot", lib().mp_edge_dot(
        _ptr(a), a_dtype, _ptr(b), b_dtype, _ptr(bidx), N_b, _ptr(oidx), E, F, _ptr(out),
        _stream(stream)))


# ---- convenience wrappers ---------------------------------------------------------

def new_status(device) -> torch.Tensor:
    """A device status word for the sorting calls (int32 [1])."""
    return torch.empty(1, dtype=torch.int32, device=device)


def check_status(status: torch.Tensor, fn: str = "device sort", stream=None) -> None:
    """Wait for the stream and raise MPError if a sort reported failure."""
    if hasattr(stream, "synchronize"):
        stream.synchronize()
    elif stream is None:
        torch.cuda.current_stream(status.device).synchronize()
    else:  # a raw stream handle
        torch.cuda.synchronize(status.device)
    _check(fn, int(status.item()))


def _sort_status(status, check, device):
    """(status tensor to pass, whether to check it after the call)."""
    if status is not None:
        return status, False
    return (new_status(device), True) if check else (None, False)


def coo_to_csr(src: torch.Tensor, dst: torch.Tensor, N: int, *, rowptr_dtype=torch.int32,
               want_perm=False, val=None, stream=None, ws=None, status=None, check=True):
    """Stable destination-major CSR of the COO edges (src, dst int32 on GPU).

    The sort's device status is written into `status` (an int32 [1] tensor)
    when one is given; otherwise, with check=True, the call waits for the
    stream and raises MPError(MP_ERR_SORT) if the sort failed.
    Returns (rowptr, col, perm or None, val_csr or None)."""
    E = int(src.numel())
    dev = src.device
    it = _itype_code(rowptr_dtype)
    rowptr = torch.empty(N + 1, dtype=rowptr_dtype, device=dev)
    col = _edge_array(E, torch.int32, dev)
    perm = _edge_array(E, torch.int32, dev) if want_perm else None
    vout = _edge_array(E, torch.float32, dev) if val is not None else None
    nb = mp_coo_to_csr_workspace(E, N, it, want_perm or val is not None)
    if ws is None or ws.numel() < nb:
        ws = _workspace(nb, dev)
    st, chk = _sort_status(status, check, dev)
    mp_coo_to_csr(src, dst, E, N, rowptr, it, col, perm, val, vout, ws, ws.numel(), st, stream)
    if chk:
        check_status(st, "mp_coo_to_csr", stream)
    return rowptr, col, perm, vout


def sorted_coo_to_csr(src: torch.Tensor, dst: torch.Tensor, N: int, *, rowptr_dtype=torch.int32,
                      want_perm=False, val=None, stream=None):
    """CSR of COO edges already sorted by destination (no sort is run).

    Returns (rowptr, col, perm or None, val_csr or None) like coo_to_csr."""
    E = int(src.numel())
    dev = src.device
    it = _itype_code(rowptr_dtype)
    rowptr = torch.empty(N + 1, dtype=rowptr_dtype, device=dev)
    col = _edge_array(E, torch.int32, dev)
    perm = _edge_array(E, torch.int32, dev) if want_perm else None
    vout = _edge_array(E, torch.float32, dev) if val is not None else None
    mp_sorted_coo_to_csr(src, dst, E, N, rowptr, it, col, perm, val, vout, stream)
    return rowptr, col, perm, vout


class Plan:
    """Degree-binned aggregation plan for one CSR and one (F, dtype).

    Building it synchronizes the stream once (bin sizes go to the host).
    opts: None for the default thresholds, or (small_max, hub_min, chunk_min)
    with 0 for a default (mp_plan_opts)."""

    def __init__(self, rowptr: torch.Tensor, E: int, F: int, x_dtype=torch.float32, stream=None,
                 opts=None):
        self.rowptr = rowptr
        self.itype = _itype_code(rowptr.dtype)
        self.N_dst = int(rowptr.numel()) - 1
        self.E, self.F = int(E), int(F)
        self.x_dtype = _dtype_code(x_dtype)
        nb = mp_spmm_plan_size(self.N_dst, self.E)
        self.buf = _workspace(nb, rowptr.device)
        if opts is None:
            self.handle = mp_spmm_plan_build(rowptr, self.itype, self.N_dst, self.E, self.F,
                                             self.x_dtype, self.buf, self.buf.numel(), stream)
        else:
            self.handle = mp_spmm_plan_build_opts(rowptr, self.itype, self.N_dst, self.E,
                                                  self.F, self.x_dtype, self.buf,
                                                  self.buf.numel(), opts, stream)
        self._ws = {}

    def workspace(self, reduce: int) -> torch.Tensor | None:
        nb = mp_spmm_workspace(self.handle, reduce)
        if nb == 0:
            return None
        t = self._ws.get(reduce)
        if t is None or t.numel() < nb:
            t = self._ws[reduce] = _workspace(nb, self.rowptr.device)
        return t

    def __del__(self):
        h = getattr(self, "handle", None)
        if h:
            try:
                mp_spmm_plan_free(h)
            except Exception:  # interpreter shutdown: module globals already gone
                pass
            self.handle = None


def spmm(rowptr, col, x, reduce, *, w=None, plan: Plan | None = None, out_dtype=torch.float32,
         max_dtype=None, out=None, out_max=None, argout=None, stream=None):
    """Aggregate x over the destination-major CSR.

    reduce: MP_SUM, MP_MEAN, MP_MAX or MP_SUM|MP_MAX / MP_MEAN|MP_MAX.
    Returns (out or None, out_max or None, argout or None)."""
    N_dst = int(rowptr.numel()) - 1
    N_src, F = int(x.shape[0]), int(x.shape[1])
    dev = x.device
    hs = bool(reduce & (MP_SUM | MP_MEAN))
    hm = bool(reduce & MP_MAX)
    if max_dtype is None:
        max_dtype = torch.float32
    if hs and out is None:
        out = torch.empty(N_dst, F, dtype=out_dtype, device=dev)
    if hm and out_max is None:
        out_max = torch.empty(N_dst, F, dtype=max_dtype, device=dev)
    if hm and argout is None:
        argout = torch.empty(N_dst, F, dtype=torch.int32, device=dev)
    ws = plan.workspace(reduce) if plan is not None else None
    ldx = _rows_ptr(x)[1]
    mp_spmm(plan.handle if plan is not None else None, rowptr, _itype_code(rowptr.dtype), col, w,
            x, _dtype_code(x.dtype), N_src, N_dst, F, ldx, reduce, out if hs else None,
            _dtype_code(out.dtype) if hs else MP_F32, out_max if hm else None,
            _dtype_code(out_max.dtype) if hm else MP_F32, argout if hm else None, ws,
            0 if ws is None else ws.numel(), stream)
    return (out if hs else None, out_max if hm else None, argout if hm else None)


def csr_transpose(rowptr, col, N_src, *, rowptrT_dtype=torch.int32, want_pos=True, val=None,
                  stream=None, status=None, check=True):
    """Source-major CSR of a destination-major CSR's edges (status and check
    as in coo_to_csr).

    Returns (rowptrT, colT = destinations, posT = forward CSR positions or
    None, val in transposed order or None)."""
    N_dst = int(rowptr.numel()) - 1
    E = int(col.numel())
    dev = col.device
    itT = _itype_code(rowptrT_dtype)
    rowptrT = torch.empty(N_src + 1, dtype=rowptrT_dtype, device=dev)
    colT = _edge_array(E, torch.int32, dev)
    posT = _edge_array(E, torch.int32, dev) if want_pos else None
    vout = _edge_array(E, torch.float32, dev) if val is not None else None
    nb = mp_csr_transpose_workspace(E, N_src, itT, want_pos or val is not None)
    ws = _workspace(nb, dev) if nb else None
    st, chk = _sort_status(status, check, dev)
    mp_csr_transpose(rowptr, _itype_code(rowptr.dtype), col, N_dst, N_src, E, rowptrT, itT, colT,
                     posT, val, vout, ws, 0 if ws is None else ws.numel(), st, stream)
    if chk:
        check_status(st, "mp_csr_transpose", stream)
    return rowptrT, colT, posT, vout


def spmm_backward_x(rowptrT, colT, grad_out, reduce, *, posT=None, wT=None, rowptr=None,
                    argout=None, planT: Plan | None = None, out_dtype=torch.float32, out=None,
                    stream=None):
    """dL/dx of spmm for one reduction, over the transposed CSR (rowptr, the
    forward one, is needed for mean and max)."""
    N_src = int(rowptrT.numel()) - 1
    N_dst, F = int(grad_out.shape[0]), int(grad_out.shape[1])
    E = int(colT.numel())
    dev = grad_out.device
    if out is None:
        out = torch.empty(N_src, F, dtype=out_dtype, device=dev)
    h = planT.handle if planT is not None else None
    nb = mp_spmm_backward_x_workspace(h, N_dst, E, F, reduce)
    ws = _workspace(nb, dev) if nb else None
    mp_spmm_backward_x(h, rowptrT, _itype_code(rowptrT.dtype), colT, posT, wT, rowptr,
                       _itype_code(rowptr.dtype) if rowptr is not None else MP_I32, argout,
                       grad_out, _dtype_code(grad_out.dtype), N_dst, N_src, E, F, reduce, out,
                       _dtype_code(out.dtype), ws, 0 if ws is None else ws.numel(), stream)
    return out


def spmm_backward_w(rowptr, col, x, grad_out, reduce, *, argout=None, out=None, stream=None):
    """dL/dw (forward CSR order, fp32) of a weighted spmm for one reduction."""
    N_dst = int(rowptr.numel()) - 1
    N_src, F = int(x.shape[0]), int(x.shape[1])
    E = int(col.numel())
    dev = x.device
    if out is None:
        out = _edge_array(E, torch.float32, dev)
    nb = mp_spmm_backward_w_workspace(E)
    ws = _workspace(nb, dev) if nb else None
    mp_spmm_backward_w(rowptr, _itype_code(rowptr.dtype), col, x, _dtype_code(x.dtype), grad_out,
                       _dtype_code(grad_out.dtype), argout, N_src, N_dst, E, F, reduce, out, ws,
                       0 if ws is None else ws.numel(), stream)
    return out


def _multi_outputs(names, N, F, dev):
    res, outs = {}, []
    for n in names:
        o = torch.empty(N, F, dtype=torch.float32, device=dev)
        g = torch.empty(N, F, dtype=torch.int32, device=dev) if n in ("max", "min") else None
        res[n] = o
        if g is not None:
            res["arg" + n] = g
        outs.append((AGGR[n], o, g))
    return res, outs


def spmm_multi(rowptr, col, x, aggrs, *, w=None, plan: Plan | None = None, stream=None):
    """Several aggregations from one gather.  aggrs: names among sum, mean,
    max, min, var, std.  Returns {name: [N_dst, F] fp32, 'argmax'/'argmin':
    int32 positions}."""
    N_dst = int(rowptr.numel()) - 1
    N_src, F = int(x.shape[0]), int(x.shape[1])
    res, outs = _multi_outputs(aggrs, N_dst, F, x.device)
    h = plan.handle if plan is not None else None
    nb = mp_spmm_multi_workspace(h)
    ws = _workspace(nb, x.device) if nb else None
    mp_spmm_multi(h, rowptr, _itype_code(rowptr.dtype), col, w, x, _dtype_code(x.dtype), N_src,
                  N_dst, F, _rows_ptr(x)[1], outs, ws, 0 if ws is None else ws.numel(), stream)
    return res


def readout(ptr, x, aggrs, *, plan: Plan | None = None, stream=None):
    """Global readout over segments of consecutive rows of x (ptr: [S+1], the
    CSR of a sorted batch vector).  Same outputs as spmm_multi, arg = row."""
    N_seg = int(ptr.numel()) - 1
    N_nodes, F = int(x.shape[0]), int(x.shape[1])
    res, outs = _multi_outputs(aggrs, N_seg, F, x.device)
    h = plan.handle if plan is not None else None
    nb = mp_spmm_multi_workspace(h)
    ws = _workspace(nb, x.device) if nb else None
    mp_readout_multi(h, ptr, _itype_code(ptr.dtype), x, _dtype_code(x.dtype), N_nodes, N_seg, F,
                     _rows_ptr(x)[1], outs, ws, 0 if ws is None else ws.numel(), stream)
    return res


def segment_matmul(seg, x, W, *, out_dtype=torch.float32, stream=None):
    """out[r] = x[r] @ W[t] for the rows of segment t (seg: host list of T+1
    offsets; x [N, F] and W [T, F, Fo] bf16)."""
    T, F, Fo = (int(v) for v in W.shape)
    N = int(x.shape[0])
    out = torch.empty(N, Fo, dtype=out_dtype, device=x.device)
    ws = _workspace(mp_segment_matmul_workspace(T, F, Fo), x.device)
    mp_segment_matmul(seg, T, x, W, F, Fo, out, _dtype_code(out_dtype), ws, ws.numel(), stream)
    return out


def segment_matmul_backward(seg, x, W, dout, *, dx_dtype=torch.float32, want_dx=True,
                            want_dw=True, stream=None):
    """Gradients of segment_matmul: (dx [N, F] or None, dW [T, F, Fo] fp32 or None)."""
    T, F, Fo = (int(v) for v in W.shape)
    N = int(dout.shape[0])
    dx = torch.empty(N, F, dtype=dx_dtype, device=dout.device) if want_dx else None
    dW = torch.empty(T, F, Fo, dtype=torch.float32, device=dout.device) if want_dw else None
    ws = _workspace(mp_segment_matmul_backward_workspace(seg, T, F, Fo), dout.device) \
        if want_dw else None
    mp_segment_matmul_backward(seg, T, x, W, dout, F, Fo, dx, _dtype_code(dx_dtype), dW, ws,
                               0 if ws is None else ws.numel(), stream)
    return dx, dW


def hetero_build(N_per_type, rels, dst_type, *, rowptr_dtype=torch.int32, stream=None,
                 status=None, check=True):
    """Combined destination-major CSR of one destination type, or of all of
    them (dst_type = MP_ALL_TYPES: rows are all nodes as global ids); status
    and check as in coo_to_csr.

    rels: list of (src_type, dst_type, src int32 tensor, dst int32 tensor).
    Returns (rowptr, col with global source ids)."""
    it = _itype_code(rowptr_dtype)
    dev = next(r[2].device for r in rels)
    everything = dst_type == MP_ALL_TYPES
    E_T = sum(int(r[2].numel()) for r in rels if everything or r[1] == dst_type)
    n_rows = sum(N_per_type) if everything else N_per_type[dst_type]
    rowptr = torch.empty(n_rows + 1, dtype=rowptr_dtype, device=dev)
    col = _edge_array(E_T, torch.int32, dev)
    nb = mp_hetero_build_workspace(N_per_type, rels, dst_type, it)
    ws = _workspace(nb, dev)
    st, chk = _sort_status(status, check, dev)
    mp_hetero_build(N_per_type, rels, dst_type, rowptr, it, col, ws, ws.numel(), st, stream)
    if chk:
        check_status(st, "mp_hetero_build", stream)
    return rowptr, col


def hetero_spmm(N_per_type, x_per_type, dst_type, rowptr, col, *, plan: Plan | None = None,
                out_dtype=torch.float32, out=None, stream=None):
    """Sum over the combined CSR of dst_type (or of all types), gathering
    from per-type tables."""
    F = int(x_per_type[0].shape[1])
    dev = x_per_type[0].device
    if out is None:
        n_rows = sum(N_per_type) if dst_type == MP_ALL_TYPES else N_per_type[dst_type]
        out = torch.empty(n_rows, F, dtype=out_dtype, device=dev)
    ws = plan.workspace(MP_SUM) if plan is not None else None
    mp_hetero_spmm(N_per_type, x_per_type, _dtype_code(x_per_type[0].dtype), F, dst_type,
                   plan.handle if plan is not None else None, rowptr, _itype_code(rowptr.dtype),
                   col, MP_SUM, out, _dtype_code(out.dtype), ws, 0 if ws is None else ws.numel(),
                   stream)
    return out


# ---- feature-table layout --------------------------------------------------------------

CACHE_LINE = 128


def aligned_ld(F: int, dtype) -> int:
    """Row stride (elements) for a table of F-element rows: F itself, or the
    next stride whose row bytes are a multiple of the 128-byte cache line when
    that makes a randomly gathered row touch fewer lines on average (rows of
    at least one line, padded by at most half their size)."""
    b = torch.tensor([], dtype=dtype).element_size()
    rb = F * b
    if rb % CACHE_LINE == 0 or rb < CACHE_LINE:
        return F
    step = __import__("math").gcd(rb, CACHE_LINE)
    offs = range(0, CACHE_LINE, step)
    lines = sum(-(-(o + rb) // CACHE_LINE) for o in offs) / len(offs)
    padded = -(-rb // CACHE_LINE)
    if padded < lines and 2 * padded * CACHE_LINE <= 3 * rb:
        return padded * CACHE_LINE // b
    return F


def pad_rows(x, ld=None, *, out=None, stream=None):
    """x [N, F] copied into rows ld elements apart (default aligned_ld);
    returns the [N, F] view of the padded [N, ld] buffer."""
    N, F = int(x.shape[0]), int(x.shape[1])
    ld = aligned_ld(F, x.dtype) if ld is None else int(ld)
    if out is None:
        out = torch.empty(max(N, 1), ld, dtype=x.dtype, device=x.device)[:N, :F]
    mp_copy_rows(x, _rows_ptr(x)[1], out, _rows_ptr(out)[1], N, F, _dtype_code(x.dtype), stream)
    return out


# ---- edge-materialized messages (explanation mode) ------------------------------------

def csr_rows(rowptr, E, *, stream=None):
    """The destination row of every CSR position (int32 [E])."""
    N_dst = int(rowptr.numel()) - 1
    row = _edge_array(int(E), torch.int32, rowptr.device)
    mp_csr_rows(rowptr, _itype_code(rowptr.dtype), N_dst, int(E), row, stream)
    return row


def message_gather(idx, x, *, w=None, msg_dtype=torch.float32, out=None, stream=None):
    """msg[p] = w[p] * x[idx[p]] (or x[idx[p]]): the materialized messages,
    [E, F] of msg_dtype (bf16 only for unweighted bf16 x)."""
    E = int(idx.numel())
    N_src, F = int(x.shape[0]), int(x.shape[1])
    if out is None:
        out = torch.empty(max(E, 1), F, dtype=msg_dtype, device=x.device)[:E]
    mp_message_gather(idx, w, x, _dtype_code(x.dtype), N_src, E, F, out, _dtype_code(out.dtype),
                      stream)
    return out


def message_scale(msg, mask, *, idx=None, out=None, stream=None):
    """out[p] = msg[p] * mask[idx[p]] (idx None: mask[p]); out may be msg."""
    E, F = int(msg.shape[0]), int(msg.shape[1])
    if out is None:
        out = torch.empty_like(msg)
    mp_message_scale(msg, out, E, F, mask, idx, int(mask.numel()), stream)
    return out


def message_aggregate(rowptr, msg, reduce, *, plan: Plan | None = None, out_dtype=torch.float32,
                      max_dtype=None, stream=None):
    """Aggregate the message rows of each CSR row: (out, out_max, argout)
    like spmm, argout = the message row."""
    N_dst = int(rowptr.numel()) - 1
    E, F = int(msg.shape[0]), int(msg.shape[1])
    dev = msg.device
    hs = bool(reduce & (MP_SUM | MP_MEAN))
    hm = bool(reduce & MP_MAX)
    out = torch.empty(N_dst, F, dtype=out_dtype, device=dev) if hs else None
    out_max = torch.empty(N_dst, F, dtype=max_dtype or torch.float32, device=dev) if hm else None
    argout = torch.empty(N_dst, F, dtype=torch.int32, device=dev) if hm else None
    ws = plan.workspace(reduce) if plan is not None else None
    mp_message_aggregate(plan.handle if plan is not None else None, rowptr,
                         _itype_code(rowptr.dtype), msg, _dtype_code(msg.dtype), E, N_dst, F,
                         reduce, out, _dtype_code(out.dtype) if hs else MP_F32, out_max,
                         _dtype_code(out_max.dtype) if hm else MP_F32, argout, ws,
                         0 if ws is None else ws.numel(), stream)
    return out, out_max, argout


def spmm_materialized(rowptr, col, x, reduce, *, callback=None, w=None, plan: Plan | None = None,
                      msg=None, msg_dtype=torch.float32, out_dtype=torch.float32, max_dtype=None,
                      stream=None):
    """Explanation-mode aggregation: gather the messages into msg ([E, F],
    allocated unless given), call callback(msg) (a Python function that edits
    the tensor in place, enqueuing its work on the current stream), then
    aggregate.  Returns (out, out_max, argout, msg)."""
    N_dst = int(rowptr.numel()) - 1
    N_src, F = int(x.shape[0]), int(x.shape[1])
    E = int(col.numel())
    dev = x.device
    if msg is None:
        msg = torch.empty(max(E, 1), F, dtype=msg_dtype, device=dev)[:E]
    hs = bool(reduce & (MP_SUM | MP_MEAN))
    hm = bool(reduce & MP_MAX)
    out = torch.empty(N_dst, F, dtype=out_dtype, device=dev) if hs else None
    out_max = torch.empty(N_dst, F, dtype=max_dtype or torch.float32, device=dev) if hm else None
    argout = torch.empty(N_dst, F, dtype=torch.int32, device=dev) if hm else None
    ws = plan.workspace(reduce) if plan is not None else None
    failure = []

    def trampoline(ptr, dtype, e, f, user, strm):
        try:
            callback(msg)
            return 0
        except Exception as exc:  # reported after the C call returns
            failure.append(exc)
            return 1

    c = MESSAGE_FN(trampoline) if callback is not None else None
    try:
        mp_spmm_materialized(plan.handle if plan is not None else None, rowptr,
                             _itype_code(rowptr.dtype), col, w, x, _dtype_code(x.dtype), N_src,
                             N_dst, E, F, msg, _dtype_code(msg.dtype), c, None, reduce, out,
                             _dtype_code(out.dtype) if hs else MP_F32, out_max,
                             _dtype_code(out_max.dtype) if hm else MP_F32, argout, ws,
                             0 if ws is None else ws.numel(), stream)
    except MPError as err:
        if failure:
            raise err from failure[0]
        raise
    return out, out_max, argout, msg


def message_backward(rowptr, grad_out, reduce, *, E=None, argout=None, out=None, stream=None):
    """dL/dmsg [E, F] fp32 of message_aggregate for one reduction."""
    N_dst = int(rowptr.numel()) - 1
    F = int(grad_out.shape[1])
    if E is None:
        E = int(rowptr[-1].item())
    dev = grad_out.device
    if out is None:
        out = torch.empty(max(E, 1), F, dtype=torch.float32, device=dev)[:E]
    nb = mp_message_backward_workspace(E)
    ws = _workspace(nb, dev) if nb else None
    mp_message_backward(rowptr, _itype_code(rowptr.dtype), argout, grad_out,
                        _dtype_code(grad_out.dtype), N_dst, E, F, reduce, out, ws,
                        0 if ws is None else ws.numel(), stream)
    return out


def edge_dot(a, b, *, bidx=None, oidx=None, out=None, stream=None):
    """out[oidx[p]] = sum_f a[p, f] * b[bidx[p], f] (fp32 [E])."""
    E, F = int(a.shape[0]), int(a.shape[1])
    if out is None:
        out = _edge_array(E, torch.float32, a.device)
    mp_edge_dot(a, _dtype_code(a.dtype), b, _dtype_code(b.dtype), bidx, int(b.shape[0]), oidx, E,
                F, out, stream)
    return out
