"""Seeded synthetic graph workloads (inputs only).

Every array here is a pure function of (seed, stream, index) through the
counter-based SplitMix64 generator in ``gen.c``; nothing in this module
computes any part of the aggregation.  Both the CPU oracle and the device
library are fed from these arrays, so the two never share method code.

The workloads stand in for public graphs of the same shape (a small citation
graph, an arxiv-scale and a products-scale power-law graph, a three-type
academic graph, a web-scale shard); none of those datasets is used.

Feature arrays in bfloat16 are returned as ``uint16`` bit patterns.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
_LIB_PATH = os.path.join(_HERE, "_libgraphgen.so")
_lib = None

# Stream ids: one per independent array so that no two arrays share draws.
S_SRC, S_DST, S_X, S_PERM = 1, 2, 3, 4


def build(force: bool = True) -> str:
    """Compile ``gen.c`` into ``_libgraphgen.so`` with gcc + OpenMP."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", _SRC, "-o", tmp, "-lm"]
        )
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _L():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        u64, i64, p = ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p
        lib.gg_key.argtypes = [u64, u64]
        lib.gg_key.restype = u64
        lib.gg_draw.argtypes = [u64, u64]
        lib.gg_draw.restype = u64
        lib.gg_uniform_ints.argtypes = [u64, u64, i64, i64, p]
        lib.gg_permutation.argtypes = [u64, u64, i64, p]
        lib.gg_alias_powerlaw.argtypes = [i64, ctypes.c_double, p, p]
        lib.gg_alias_powerlaw.restype = ctypes.c_int
        lib.gg_sample_alias.argtypes = [u64, u64, i64, i64, p, p, p, p]
        lib.gg_zeta_partial.argtypes = [i64, ctypes.c_double]
        lib.gg_zeta_partial.restype = ctypes.c_double
        lib.gg_fit_beta.argtypes = [i64, i64, ctypes.c_double, ctypes.c_double,
                                    ctypes.c_double, ctypes.c_int]
        lib.gg_fit_beta.restype = ctypes.c_double
        lib.gg_uniform_f32.argtypes = [u64, u64, i64, p]
        lib.gg_normal_f32.argtypes = [u64, u64, i64, p]
        lib.gg_f32_to_bf16.argtypes = [i64, p, p]
        lib.gg_uniform_bf16.argtypes = [u64, u64, i64, p]
        lib.gg_gcn_weights.argtypes = [i64, p, p, i64, i64, p]
        lib.gg_gcn_weights.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


# ---- primitives -------------------------------------------------------------

def draws(seed: int, stream: int, n: int) -> np.ndarray:
    """Raw 64-bit draws (for tests of the generator itself)."""
    L = _L()
    k = L.gg_key(seed, stream)
    return np.array([L.gg_draw(k, i) for i in range(n)], dtype=np.uint64)


def uniform_ints(seed: int, stream: int, n: int, upper: int) -> np.ndarray:
    out = np.empty(n, dtype=np.int32)
    if n:
        _L().gg_uniform_ints(seed, stream, n, upper, _ptr(out))
    return out


def permutation(seed: int, stream: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.int32)
    if n:
        _L().gg_permutation(seed, stream, n, _ptr(out))
    return out


def powerlaw_endpoints(seed: int, stream: int, n: int, e: int, beta: float,
                       perm: np.ndarray) -> np.ndarray:
    """E i.i.d. endpoints with P(rank r) proportional to r^-beta, ids = perm[rank]."""
    prob = np.empty(n, dtype=np.float64)
    alias = np.empty(n, dtype=np.int32)
    if _L().gg_alias_powerlaw(n, beta, _ptr(prob), _ptr(alias)) != 0:
        raise MemoryError("alias table allocation failed")
    out = np.empty(e, dtype=np.int32)
    if e:
        _L().gg_sample_alias(seed, stream, e, n, _ptr(prob), _ptr(alias), _ptr(perm), _ptr(out))
    return out


def fit_beta(n: int, e: int, dmax: float) -> float:
    """Exponent beta such that Chung-Lu weights r^-beta give rank 1 degree dmax."""
    return _L().gg_fit_beta(n, e, dmax, 0.0, 1.5, 60)


def zeta_partial(n: int, beta: float) -> float:
    return _L().gg_zeta_partial(n, beta)


def uniform_f32(seed: int, stream: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.float32)
    if n:
        _L().gg_uniform_f32(seed, stream, n, _ptr(out))
    return out


def normal_f32(seed: int, stream: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.float32)
    if n:
        _L().gg_normal_f32(seed, stream, n, _ptr(out))
    return out


def uniform_bf16(seed: int, stream: int, n: int) -> np.ndarray:
    """The bf16 rounding of uniform_f32(seed, stream, n), drawn directly."""
    out = np.empty(n, dtype=np.uint16)
    if n:
        _L().gg_uniform_bf16(seed, stream, n, _ptr(out))
    return out


def f32_to_bf16(a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    out = np.empty(a.shape, dtype=np.uint16)
    if a.size:
        _L().gg_f32_to_bf16(a.size, _ptr(a), _ptr(out))
    return out


def bf16_to_f32(a: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to fp32."""
    return (np.ascontiguousarray(a, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def gcn_weights(src: np.ndarray, dst: np.ndarray, n_src: int, n_dst: int) -> np.ndarray:
    w = np.empty(src.shape[0], dtype=np.float32)
    if src.shape[0] and _L().gg_gcn_weights(src.shape[0], _ptr(src), _ptr(dst), n_src,
                                            n_dst, _ptr(w)) != 0:
        raise ValueError("bad edge index for gcn_weights")
    return w


# ---- workloads --------------------------------------------------------------

@dataclass
class Graph:
    """One homogeneous workload: COO edges, features, optional edge weights."""
    name: str
    n_src: int
    n_dst: int
    src: np.ndarray           # int32 [E]
    dst: np.ndarray           # int32 [E]
    F: int
    x: np.ndarray | None = None        # fp32 [n_src, F]
    x_bf16: np.ndarray | None = None   # uint16 [n_src, F]
    w: np.ndarray | None = None        # fp32 [E], COO order
    meta: dict = field(default_factory=dict)

    @property
    def E(self) -> int:
        return int(self.src.shape[0])


@dataclass
class HeteroGraph:
    """Typed nodes and relations; relation r goes from rel_src[r] to rel_dst[r]."""
    name: str
    n_per_type: list
    rel_src_type: list
    rel_dst_type: list
    rel_src: list             # int32 [E_r], local ids in the source type
    rel_dst: list             # int32 [E_r], local ids in the destination type
    F: int
    x_bf16: list              # uint16 [N_t, F] per type
    meta: dict = field(default_factory=dict)


def uniform_graph(seed: int, n: int, e: int, f: int, feat: str = "uniform",
                  bf16: bool = False) -> Graph:
    """src, dst ~ U{0..n-1} i.i.d.; self-loops and duplicates kept."""
    src = uniform_ints(seed, S_SRC, e, n)
    dst = uniform_ints(seed, S_DST, e, n)
    x = (uniform_f32 if feat == "uniform" else normal_f32)(seed, S_X, n * f).reshape(n, f)
    g = Graph(f"uniform-n{n}-e{e}-f{f}", n, n, src, dst, f, x=x)
    if bf16:
        g.x_bf16 = f32_to_bf16(x)
    return g


def powerlaw_dst_graph(seed: int, n: int, e: int, f: int, alpha: float,
                       feat: str = "normal", weights: bool = False, bf16: bool = False,
                       fp32: bool = True) -> Graph:
    """Destinations with P(rank r) ~ r^-beta, beta = 1/(alpha-1) (a Zipf-like
    in-degree law with exponent alpha), sources uniform."""
    beta = 1.0 / (alpha - 1.0)
    perm = permutation(seed, S_PERM, n)
    dst = powerlaw_endpoints(seed, S_DST, n, e, beta, perm)
    src = uniform_ints(seed, S_SRC, e, n)
    g = Graph(f"powerlaw-n{n}-e{e}-f{f}-a{alpha}", n, n, src, dst, f,
              meta={"alpha": alpha, "beta": beta})
    if feat == "uniform" and bf16 and not fp32:
        g.x_bf16 = uniform_bf16(seed, S_X, n * f).reshape(n, f)
        return g
    xf = (uniform_f32 if feat == "uniform" else normal_f32)(seed, S_X, n * f).reshape(n, f)
    if bf16:
        g.x_bf16 = f32_to_bf16(xf)
    if fp32:
        g.x = xf
    if weights:
        g.w = gcn_weights(src, dst, n, n)
    return g


def chung_lu_graph(seed: int, n: int, e: int, f: int, dmax: float, beta: float | None = None,
                   bf16: bool = True, fp32: bool = True) -> Graph:
    """Chung-Lu: both endpoints drawn with P(rank r) ~ r^-beta (same id
    permutation for both), beta fitted so the expected top degree is dmax."""
    if beta is None:
        beta = fit_beta(n, e, dmax)
    perm = permutation(seed, S_PERM, n)
    src = powerlaw_endpoints(seed, S_SRC, n, e, beta, perm)
    dst = powerlaw_endpoints(seed, S_DST, n, e, beta, perm)
    xf = normal_f32(seed, S_X, n * f).reshape(n, f)
    g = Graph(f"chunglu-n{n}-e{e}-f{f}", n, n, src, dst, f, meta={"beta": beta, "dmax": dmax})
    if bf16:
        g.x_bf16 = f32_to_bf16(xf)
    if fp32:
        g.x = xf
    return g


def hetero_graph(seed: int, n_per_type, rels, f: int) -> HeteroGraph:
    """rels: list of (src_type, dst_type, E); endpoints uniform within types;
    features N(0,1) rounded to bfloat16."""
    rs, rd, es, ed = [], [], [], []
    for r, (st, dt, e) in enumerate(rels):
        rs.append(st)
        rd.append(dt)
        es.append(uniform_ints(seed, 16 * r + 1, e, n_per_type[st]))
        ed.append(uniform_ints(seed, 16 * r + 2, e, n_per_type[dt]))
    xs = [f32_to_bf16(normal_f32(seed, 16 * (8 + t) + 3, n * f)).reshape(n, f)
          for t, n in enumerate(n_per_type)]
    return HeteroGraph(f"hetero-{len(n_per_type)}t-{len(rels)}r", list(n_per_type), rs, rd,
                       es, ed, f, xs)


# Full-size workloads, named by what they are.  The sizes are those of the
# public graphs they stand in for; all content is synthetic.
CHUNGLU_124M = dict(n=2_449_029, e=123_718_280, f=100, dmax=17_000.0)
POWERLAW_1_2M = dict(n=169_343, e=1_166_243, f=128, alpha=2.1)
UNIFORM_10K = dict(n=2_708, e=10_556, f=64)
HETERO_20M = dict(n_per_type=[1_900_000, 736_000, 8_700],
                  rels=[(0, 0, 5_400_000), (0, 1, 7_100_000), (1, 0, 7_100_000),
                        (1, 2, 1_000_000)], f=128)
WEB_1_6B = dict(n=100_000_000, e=1_600_000_000, f=64, alpha=2.0)

# The Chung-Lu exponent for CHUNGLU_124M, fitted once by bisection
# (fit_beta(2449029, 123718280, 17000)); a test re-fits it.
CHUNGLU_124M_BETA = 0.43423


def workload(name: str, seed: int = 0, scale: float = 1.0, **kw):
    """Build a named workload; `scale` shrinks N and E together (same shape)."""
    def s(v):
        return max(1, int(round(v * scale)))
    if name == "uniform-10k":
        c = UNIFORM_10K
        return uniform_graph(seed, s(c["n"]), s(c["e"]), c["f"], **kw)
    if name == "powerlaw-1.2M":
        c = POWERLAW_1_2M
        return powerlaw_dst_graph(seed, s(c["n"]), s(c["e"]), c["f"], c["alpha"],
                                  weights=True, **kw)
    if name == "chunglu-124M":
        c = CHUNGLU_124M
        beta = CHUNGLU_124M_BETA if scale == 1.0 else None
        dmax = c["dmax"] * scale if scale != 1.0 else c["dmax"]
        return chung_lu_graph(seed, s(c["n"]), s(c["e"]), c["f"], dmax, beta=beta, **kw)
    if name == "hetero-20M":
        c = HETERO_20M
        return hetero_graph(seed, [s(n) for n in c["n_per_type"]],
                            [(a, b, s(e)) for a, b, e in c["rels"]], c["f"])
    if name == "web-1.6B":
        c = WEB_1_6B
        return powerlaw_dst_graph(seed, s(c["n"]), s(c["e"]), c["f"], c["alpha"],
                                  feat="uniform", bf16=True, fp32=False, **kw)
    raise KeyError(name)


def mixed_graph(seed: int, n: int = 3000, e: int = 40_000, f: int = 64, alpha: float = 2.1,
                signed_weights: bool = False, bf16: bool = True) -> Graph:
    """Small power-law graph with every degree regime at once: ~18% empty
    rows, many small rows, mid rows and a few hubs of ~1-2k edges.  Weights
    are GCN-style (positive) or U(-1,1) (signed)."""
    g = powerlaw_dst_graph(seed, n, e, f, alpha, feat="normal", weights=not signed_weights,
                           bf16=bf16, fp32=True)
    if signed_weights:
        g.w = uniform_f32(seed, 7, e)
    g.name = f"mixed-n{n}-e{e}-f{f}"
    return g
