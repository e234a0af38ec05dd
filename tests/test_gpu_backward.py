"""Parity of the HIP backward pass (through the C ABI) with the CPU oracle.

The transposed CSR (rowptrT, colT, posT, weights in transposed order) must be
bit-exact.  Gradients are sums, held to the same summand-scaled bound as the
forward sums: max |y - y_ref| / sum |terms| <= 1e-5 for an fp32 gradient
input and <= 1e-2 for a bf16 one (fp32 accumulation in both cases).

The device receives the oracle's forward CSR and argmax as inputs, so every
check here depends only on the backward kernels.
"""
import sys

import numpy as np
import pytest
import torch

import graphgen
import oracle
import paper_2507_16991_amd as mp
from checks import scaled_error

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
TOL = {torch.float32: 1e-5, torch.bfloat16: 1e-2}
RED = {"sum": mp.MP_SUM, "mean": mp.MP_MEAN, "max": mp.MP_MAX}


@pytest.fixture(autouse=True)
def _announce(request):
    sys.stderr.write(f"\n[gpu-case] {request.node.nodeid}\n")
    sys.stderr.flush()
    yield
    torch.cuda.synchronize()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def grad_input(seed, n, f, dtype):
    """Seeded N(0,1) gradient of the aggregation output: (device tensor,
    oracle keyword arguments)."""
    gf = graphgen.normal_f32(seed, 11, n * f).reshape(n, f)
    if dtype == torch.float32:
        return dev(gf), {"g": gf}
    gb = graphgen.f32_to_bf16(gf)
    return dev(gb.view(np.int16)).view(torch.bfloat16), {"g_bf16": gb}


def x_input(g, dtype):
    if dtype == torch.float32:
        return dev(g.x), {"x": g.x}
    return dev(g.x_bf16.view(np.int16)).view(torch.bfloat16), {"x_bf16": g.x_bf16}


# ---- transposed CSR ----------------------------------------------------------------

def check_transpose(rp_o, col_o, n_src, val=None, itype=torch.int32, itypeT=torch.int32):
    rp = dev(rp_o.astype(np.int32 if itype == torch.int32 else np.int64))
    col = dev(col_o)
    v = None if val is None else dev(val)
    rpt, colt, post, vt = mp.csr_transpose(rp, col, n_src, rowptrT_dtype=itypeT, val=v)
    rpt_o, colt_o, post_o = oracle.csr_transpose(rp_o, col_o, n_src)
    assert np.array_equal(rpt.cpu().numpy().astype(np.int64), rpt_o), "rowptrT"
    assert np.array_equal(colt.cpu().numpy(), colt_o), "colT"
    assert np.array_equal(post.cpu().numpy().astype(np.int64), post_o), "posT"
    if val is not None:
        assert np.array_equal(vt.cpu().numpy().view(np.uint32), val[post_o].view(np.uint32))
    return rpt, colt, post, vt, (rpt_o, colt_o, post_o)


@pytest.mark.parametrize("n_dst,n_src,e", [(1, 1, 0), (1, 5, 9), (7, 1, 300), (300, 2000, 4097),
                                           (2000, 300, 70_001), ((1 << 20) + 3, 5000, 50_000),
                                           (5000, (1 << 18) + 1, 50_000)])
@pytest.mark.parametrize("itypes", [(torch.int32, torch.int32), (torch.int64, torch.int64),
                                    (torch.int32, torch.int64)])
def test_transpose_shapes(n_dst, n_src, e, itypes):
    src = graphgen.uniform_ints(n_dst + e, 1, e, n_src)
    dst = graphgen.uniform_ints(n_dst + e, 2, e, n_dst)
    val = graphgen.uniform_f32(n_dst + e, 3, e)
    rp_o, col_o, _, v_o = oracle.coo_to_csr(src, dst, n_dst, n_src=n_src, val=val)
    check_transpose(rp_o, col_o, n_src, v_o, *itypes)


def test_transpose_without_positions():
    g = graphgen.mixed_graph(1, n=2000, e=30_000, f=4)
    rp_o, col_o, _, _ = oracle.coo_to_csr(g.src, g.dst, g.n_dst)
    rpt, colt, post, _ = mp.csr_transpose(dev(rp_o.astype(np.int32)), dev(col_o), g.n_src,
                                          want_pos=False)
    rpt_o, colt_o, _ = oracle.csr_transpose(rp_o, col_o, g.n_src)
    assert post is None
    assert np.array_equal(rpt.cpu().numpy(), rpt_o) and np.array_equal(colt.cpu().numpy(), colt_o)


# ---- gradients ----------------------------------------------------------------------

def backward_case(g, reduce, gdtype, xdtype, weighted, use_plan, seed=0, out_dtype=torch.float32,
                  opts=None):
    """Run both gradients on device and compare with the oracle; returns the
    worst scaled errors."""
    rp_o, col_o, _, w_o = oracle.coo_to_csr(g.src, g.dst, g.n_dst, n_src=g.n_src, val=g.w)
    w_use = w_o if weighted else None
    F = g.F
    am_o = None
    if reduce == "max":
        am_o = oracle.spmm(rp_o, col_o, x=g.x if xdtype == torch.float32 else None,
                           x_bf16=g.x_bf16 if xdtype == torch.bfloat16 else None,
                           w=w_use, want=("max",))["argmax"]
    G, gkw = grad_input(seed, g.n_dst, F, gdtype)
    rp = dev(rp_o.astype(np.int32))
    col = dev(col_o)
    w = dev(w_o) if weighted else None
    argout = dev(am_o.astype(np.int32)) if am_o is not None else None
    rpt, colt, post, wt, _ = check_transpose(rp_o, col_o, g.n_src, w_o)
    planT = mp.Plan(rpt, g.E, F, gdtype, opts=opts) if use_plan else None
    gx = mp.spmm_backward_x(rpt, colt, G, RED[reduce], posT=post, wT=wt if weighted else None,
                            rowptr=rp, argout=argout, planT=planT, out_dtype=out_dtype)
    torch.cuda.synchronize()
    ref, scale = oracle.spmm_backward_x(rp_o, col_o, g.n_src, reduce, w=w_use, argout=am_o, **gkw)
    tol = TOL[gdtype] + (2.0 ** -8 if out_dtype == torch.bfloat16 else 0.0)
    ex = scaled_error(gx.float().cpu().numpy(), ref, scale)
    assert ex <= tol, f"grad_x error {ex}"
    errs = {"x": ex}
    if weighted:
        X, xkw = x_input(g, xdtype)
        gw = mp.spmm_backward_w(rp, col, X, G, RED[reduce], argout=argout)
        torch.cuda.synchronize()
        refw, scw = oracle.spmm_backward_w(rp_o, col_o, reduce, argout=am_o, **xkw, **gkw)
        ew = scaled_error(gw.cpu().numpy()[:, None], refw[:, None], scw[:, None])
        assert ew <= max(TOL[gdtype], TOL[xdtype]), f"grad_w error {ew}"
        errs["w"] = ew
    return errs


@pytest.fixture(scope="module")
def mixed():
    return graphgen.mixed_graph(0, f=64)


@pytest.mark.parametrize("F,gdtype", [(24, torch.float32), (24, torch.bfloat16), (7, torch.float32),
                                      (64, torch.float32), (100, torch.bfloat16),
                                      (130, torch.float32)])
@pytest.mark.parametrize("rp_dtype", [np.int32, np.int64])
def test_backward_max_long_rows(F, gdtype, rp_dtype):
    """Destination rows of up to 70,000 edges (positions beyond 16 bits
    within a row, win masks built over many 64-edge chunks of one row), empty
    and single-edge rows; feature counts that fill one win-mask word, two,
    four and five (a last tile with one word)."""
    degs = [1, 100, 65535, 65536, 65537, 0, 300, 70000, 3]
    n_dst = len(degs)
    n_src = 5000
    dst = np.repeat(np.arange(n_dst, dtype=np.int32), degs)
    src = graphgen.uniform_ints(5, 1, dst.size, n_src)
    shuffle = graphgen.permutation(5, 4, dst.size)
    src, dst = src[shuffle], dst[shuffle]
    x = graphgen.normal_f32(5, 3, n_src * F).reshape(n_src, F)
    rp_o, col_o, _, _ = oracle.coo_to_csr(src, dst, n_dst, n_src=n_src)
    am_o = oracle.spmm(rp_o, col_o, x=x, want=("max",))["argmax"]
    G, gkw = grad_input(2, n_dst, F, gdtype)
    rpt, colt, post, _, _ = check_transpose(rp_o, col_o, n_src)
    gx = mp.spmm_backward_x(rpt, colt, G, mp.MP_MAX, posT=post,
                            rowptr=dev(rp_o.astype(rp_dtype)),
                            argout=dev(am_o.astype(np.int32)))
    torch.cuda.synchronize()
    ref, scale = oracle.spmm_backward_x(rp_o, col_o, n_src, "max", argout=am_o, **gkw)
    assert scaled_error(gx.cpu().numpy(), ref, scale) <= TOL[gdtype]


def test_backward_max_dense_wins():
    """Rows of 1 to 70 edges over 2 sources with many duplicate edges, so a
    source row collects several wins of one destination and one feature tile
    can hold more winners than a 64-edge chunk has positions (both ways of
    building the win masks).  Every routed element of G is a small integer,
    so the gradient is exact and compared bit for bit."""
    F = 100
    degs = np.arange(1, 71)
    n_dst = degs.size
    dst = np.repeat(np.arange(n_dst, dtype=np.int32), degs)
    src = graphgen.uniform_ints(9, 1, dst.size, 2)
    x = graphgen.normal_f32(9, 3, 2 * F).reshape(2, F)
    rp_o, col_o, _, _ = oracle.coo_to_csr(src, dst, n_dst, n_src=2)
    # distinct message values per edge: x varies by source only, so ties
    # between duplicates go to the first CSR position
    am_o = oracle.spmm(rp_o, col_o, x=x, want=("max",))["argmax"]
    g = (graphgen.uniform_ints(9, 5, n_dst * F, 64) - 32).astype(np.float32).reshape(n_dst, F)
    rpt, colt, post, _, _ = check_transpose(rp_o, col_o, 2)
    gx = mp.spmm_backward_x(rpt, colt, dev(g), mp.MP_MAX, posT=post,
                            rowptr=dev(rp_o.astype(np.int32)),
                            argout=dev(am_o.astype(np.int32)), planT=mp.Plan(rpt, dst.size, F))
    torch.cuda.synchronize()
    ref, _ = oracle.spmm_backward_x(rp_o, col_o, 2, "max", argout=am_o, g=g)
    assert np.array_equal(gx.cpu().numpy(), ref.astype(np.float32))


def test_backward_plan_edge_count_mismatch():
    rp_o = np.array([0, 2, 3], np.int64)
    col_o = np.array([0, 1, 1], np.int32)
    rpt, colt, post, _, _ = check_transpose(rp_o, col_o, 2)
    planT = mp.Plan(rpt, 3, 4)
    G = torch.ones(2, 4, device=DEV)
    argout = dev(np.array([[0] * 4, [2] * 4], np.int32))
    L = mp.lib()
    nb = mp.mp_spmm_backward_x_workspace(planT.handle, 2, 3, 4, mp.MP_MAX)
    ws = torch.empty(max(nb, 1), dtype=torch.uint8, device=DEV)
    out = torch.empty(2, 4, device=DEV)
    rp = dev(rp_o.astype(np.int32))
    args = [planT.handle, rpt.data_ptr(), mp.MP_I32, colt.data_ptr(), post.data_ptr(), None,
            rp.data_ptr(), mp.MP_I32, argout.data_ptr(), G.data_ptr(), mp.MP_F32, 2, 2, 4, 4,
            mp.MP_MAX, out.data_ptr(), mp.MP_F32, ws.data_ptr(), nb, None]
    assert L.mp_spmm_backward_x(*args) == -6  # E = 4, the plan has 3 edges
    args[13] = 3
    assert L.mp_spmm_backward_x(*args) == 0
    torch.cuda.synchronize()
    assert out.cpu().tolist() == [[1.0] * 4, [1.0] * 4]


@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
@pytest.mark.parametrize("gdtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("weighted", [False, True])
@pytest.mark.parametrize("use_plan", [False, True])
def test_backward_mixed(mixed, reduce, gdtype, weighted, use_plan):
    backward_case(mixed, reduce, gdtype, gdtype, weighted, use_plan)


@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
@pytest.mark.parametrize("xdtype,gdtype", [(torch.bfloat16, torch.float32),
                                           (torch.float32, torch.bfloat16)])
def test_backward_w_mixed_dtypes(mixed, reduce, xdtype, gdtype):
    backward_case(mixed, reduce, gdtype, xdtype, True, True)


@pytest.mark.parametrize("thresholds", [(8, 64, 16), (1, 2, 1)])
@pytest.mark.parametrize("reduce", ["sum", "max"])
def test_backward_plan_regimes(thresholds, reduce):
    """Power-law sources, so the transposed CSR has hub rows; tiny thresholds
    push them through every code path, including the chunk fix-up."""
    g = graphgen.chung_lu_graph(2, 4000, 60_000, 32, dmax=3000.0)
    g.w = graphgen.uniform_f32(2, 7, g.E)
    backward_case(g, reduce, torch.float32, torch.float32, True, True, opts=thresholds)


@pytest.mark.parametrize("F", [1, 3, 8, 24, 64, 100, 128, 256, 300, 520, 1024])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_backward_feature_widths(F, dtype):
    """Every lane-chunk width (1 to 8 elements), one to several 64-chunk
    feature tiles, and win masks of 1 to 32 words per edge (so that the
    masked gather caps its edges per step at 4 when a step's mask words
    would not fit the wavefront)."""
    g = graphgen.mixed_graph(F, n=700, e=9000, f=F, signed_weights=True)
    for reduce in ("mean", "max"):
        backward_case(g, reduce, dtype, dtype, True, True, seed=F)


def test_backward_bf16_output(mixed):
    backward_case(mixed, "sum", torch.float32, torch.float32, True, True,
                  out_dtype=torch.bfloat16)


def test_backward_empty_graph():
    rp = torch.zeros(5, dtype=torch.int32, device=DEV)  # 4 destinations, no edges
    col = torch.empty(0, dtype=torch.int32, device=DEV)
    rpt, colt, post, _ = mp.csr_transpose(rp, col, 3)
    assert rpt.cpu().tolist() == [0, 0, 0, 0]
    G = torch.ones(4, 8, device=DEV)
    for r in ("sum", "mean", "max"):
        argout = torch.full((4, 8), -1, dtype=torch.int32, device=DEV)
        gx = mp.spmm_backward_x(rpt, colt, G, RED[r], posT=post, rowptr=rp, argout=argout,
                                planT=mp.Plan(rpt, 0, 8))
        assert torch.count_nonzero(gx).item() == 0
        gw = mp.spmm_backward_w(rp, col, torch.ones(3, 8, device=DEV), G, RED[r], argout=argout)
        assert gw.numel() == 0


def test_backward_deterministic(mixed):
    rp_o, col_o, _, w_o = oracle.coo_to_csr(mixed.src, mixed.dst, mixed.n_dst, val=mixed.w)
    rp, col = dev(rp_o.astype(np.int32)), dev(col_o)
    rpt, colt, post, wt = mp.csr_transpose(rp, col, mixed.n_src, val=dev(w_o))
    G, _ = grad_input(5, mixed.n_dst, mixed.F, torch.float32)
    planT = mp.Plan(rpt, mixed.E, mixed.F)
    a = mp.spmm_backward_x(rpt, colt, G, mp.MP_SUM, wT=wt, planT=planT)
    b = mp.spmm_backward_x(rpt, colt, G, mp.MP_SUM, wT=wt, planT=planT)
    x = dev(mixed.x)
    c = mp.spmm_backward_w(rp, col, x, G, mp.MP_SUM)
    d = mp.spmm_backward_w(rp, col, x, G, mp.MP_SUM)
    assert torch.equal(a, b) and torch.equal(c, d)
    # the max gradient (win masks, then the masked gather), twice
    am = dev(oracle.spmm(rp_o, col_o, x=mixed.x, want=("max",))["argmax"].astype(np.int32))
    e = mp.spmm_backward_x(rpt, colt, G, mp.MP_MAX, posT=post, rowptr=rp, argout=am,
                           planT=planT)
    f = mp.spmm_backward_x(rpt, colt, G, mp.MP_MAX, posT=post, rowptr=rp, argout=am,
                           planT=planT)
    h = mp.spmm_backward_w(rp, col, x, G, mp.MP_MEAN)
    k = mp.spmm_backward_w(rp, col, x, G, mp.MP_MEAN)
    torch.cuda.synchronize()
    assert torch.equal(e, f) and torch.equal(h, k)


@pytest.mark.parametrize("name", ["powerlaw-1.2M", "uniform-10k"])
def test_backward_workloads(name):
    g = graphgen.workload(name, seed=1)
    for reduce in ("sum", "mean", "max"):
        backward_case(g, reduce, torch.float32, torch.float32, g.w is not None, True)


def test_backward_chunglu_full_sampled():
    """Full-size power-law graph (both endpoints power-law, 124M edges, F=100):
    the whole transposed CSR bit-exact, gradients on sampled rows (all source
    hubs plus random rows)."""
    g = graphgen.workload("chunglu-124M", seed=0, bf16=False)
    print(f"[note] generated E={g.E}", file=sys.stderr, flush=True)
    rp_o, col_o, _, _ = oracle.coo_to_csr(g.src, g.dst, g.n_dst)
    rp, col = dev(rp_o.astype(np.int32)), dev(col_o)
    rpt, colt, post, _ = mp.csr_transpose(rp, col, g.n_src)
    rpt_o, colt_o, post_o = oracle.csr_transpose(rp_o, col_o, g.n_src)
    assert np.array_equal(rpt.cpu().numpy(), rpt_o)
    assert np.array_equal(colt.cpu().numpy(), colt_o)
    assert np.array_equal(post.cpu().numpy(), post_o)
    print("[note] transpose exact", file=sys.stderr, flush=True)
    F = g.F
    rng = np.random.default_rng(0)
    degT = np.diff(rpt_o)
    rows = np.unique(np.concatenate([np.argsort(degT)[-64:], rng.integers(0, g.n_src, 2000)]))
    G, gkw = grad_input(3, g.n_dst, F, torch.float32)
    planT = mp.Plan(rpt, g.E, F)
    am_o = oracle.spmm(rp_o, col_o, x=g.x, want=("max",))["argmax"]
    argout = dev(am_o.astype(np.int32))
    for reduce in ("sum", "mean", "max"):
        gx = mp.spmm_backward_x(rpt, colt, G, RED[reduce], posT=post, rowptr=rp, argout=argout,
                                planT=planT)
        torch.cuda.synchronize()
        ref, scale = oracle.spmm_backward_x(rp_o, col_o, g.n_src, reduce, argout=am_o,
                                            rows=rows, **gkw)
        e = scaled_error(gx.cpu().numpy()[rows], ref, scale)
        print(f"[note] grad_x {reduce} error {e:.3g}", file=sys.stderr, flush=True)
        assert e <= TOL[torch.float32]
        del gx
    drows = np.unique(np.concatenate([np.argsort(np.diff(rp_o))[-16:],
                                      rng.integers(0, g.n_dst, 2000)]))
    X = dev(g.x)
    for reduce in ("sum", "max"):
        gw = mp.spmm_backward_w(rp, col, X, G, RED[reduce], argout=argout)
        torch.cuda.synchronize()
        refw, scw = oracle.spmm_backward_w(rp_o, col_o, reduce, x=g.x, argout=am_o, rows=drows,
                                           **gkw)
        sel = np.concatenate([np.arange(rp_o[r], rp_o[r + 1]) for r in drows])
        e = scaled_error(gw.cpu().numpy()[sel][:, None], refw[sel][:, None], scw[sel][:, None])
        print(f"[note] grad_w {reduce} error {e:.3g}", file=sys.stderr, flush=True)
        assert e <= TOL[torch.float32]
        del gw


@pytest.mark.parametrize("reduce", ["sum", "mean"])
@pytest.mark.parametrize("weighted", [False, True])
@pytest.mark.parametrize("use_plan", [False, True])
def test_undirected_forward_csr_as_transpose(reduce, weighted, use_plan):
    """An undirected graph (every edge in both directions) with symmetric
    weights: the forward CSR lists, for each node, the same neighbours and
    weights as its transpose, so dL/dx of sum and mean may be taken over the
    forward CSR itself (posT NULL), skipping the second CSR, as include/mp.h
    documents.  Checked against the oracle's gradient (which transposes) and
    against the gradient over the real transposed CSR."""
    n, e_half, F = 3000, 25_000, 48
    a = graphgen.uniform_ints(21, 1, e_half, n)
    b = graphgen.uniform_ints(21, 2, e_half, n)
    wh = graphgen.uniform_f32(21, 7, e_half)
    src = np.concatenate([a, b]).astype(np.int32)
    dst = np.concatenate([b, a]).astype(np.int32)
    w = np.concatenate([wh, wh]).astype(np.float32)  # w(u, v) = w(v, u)
    rp_o, col_o, _, w_o = oracle.coo_to_csr(src, dst, n, n_src=n, val=w)
    w_use = w_o if weighted else None
    G, gkw = grad_input(22, n, F, torch.float32)
    rp, col = dev(rp_o.astype(np.int32)), dev(col_o)
    wd = dev(w_o) if weighted else None
    plan = mp.Plan(rp, src.size, F) if use_plan else None
    gx = mp.spmm_backward_x(rp, col, G, RED[reduce], posT=None, wT=wd, rowptr=rp, planT=plan)
    rpt, colt, post, wt, _ = check_transpose(rp_o, col_o, n, w_o)
    gx2 = mp.spmm_backward_x(rpt, colt, G, RED[reduce], posT=post, wT=wt if weighted else None,
                             rowptr=rp)
    torch.cuda.synchronize()
    ref, scale = oracle.spmm_backward_x(rp_o, col_o, n, reduce, w=w_use, **gkw)
    for y in (gx, gx2):
        err = scaled_error(y.cpu().numpy(), ref, scale)
        assert err <= TOL[torch.float32], f"{reduce} undirected grad_x error {err}"
