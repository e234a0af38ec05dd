"""Parity of the edge-materialized path (explanation mode) on the GPU, through
the C ABI, with the CPU oracle.

Gathered messages, the edge-mask callback, the gradient with respect to the
messages and the destination rows are bit-exact (copies, one correctly
rounded fp32 product or quotient per element).  Aggregations follow the
fused path's bar: argmax and max bit-exact; sums and means within the
summand-scaled 1e-5 (fp32 messages) or 1e-2 (bf16 messages); per-edge dot
products and the gradient with respect to x within 1e-5 of their summand
scale.
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
REDUCES = {"sum": mp.MP_SUM, "mean": mp.MP_MEAN, "max": mp.MP_MAX,
           "sum+max": mp.MP_SUM | mp.MP_MAX, "mean+max": mp.MP_MEAN | mp.MP_MAX}


@pytest.fixture(autouse=True)
def _announce(request):
    sys.stderr.write(f"\n[gpu-case] {request.node.nodeid}\n")
    sys.stderr.flush()
    yield
    torch.cuda.synchronize()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def bf16_dev(bits):
    return dev(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)


def host_f32(t):
    return t.float().cpu().numpy()


@pytest.fixture(scope="module")
def mixed():
    g = graphgen.mixed_graph(0, f=64)
    rp_o, col_o, perm_o, w_o = oracle.coo_to_csr(g.src, g.dst, g.n_dst, val=g.w)
    return g, rp_o, col_o, perm_o, w_o


def x_pair(g, dtype):
    """(device features, the same values as host fp32, oracle keyword)."""
    if dtype == torch.float32:
        return dev(g.x), g.x, {"x": g.x}
    return bf16_dev(g.x_bf16), graphgen.bf16_to_f32(g.x_bf16), {"x_bf16": g.x_bf16}


def compare_aggregate(ref, rp_o, out, out_max, argout, reduce, dtype):
    deg = np.diff(rp_o)
    if reduce & mp.MP_SUM:
        e = scaled_error(host_f32(out), ref["sum"], ref["scale"])
        assert e <= TOL[dtype], f"sum error {e}"
    if reduce & mp.MP_MEAN:
        e = scaled_error(host_f32(out), ref["mean"], ref["scale"] / np.maximum(deg, 1)[:, None])
        assert e <= TOL[dtype], f"mean error {e}"
    if reduce & mp.MP_MAX:
        assert np.array_equal(argout.cpu().numpy().astype(np.int64), ref["argmax"]), "argmax"
        assert np.array_equal(host_f32(out_max).view(np.uint32), ref["max"].view(np.uint32)), "max"


# ---- gather ------------------------------------------------------------------------------

@pytest.mark.parametrize("xdtype,msgdtype,weighted", [
    (torch.float32, torch.float32, False), (torch.float32, torch.float32, True),
    (torch.bfloat16, torch.float32, False), (torch.bfloat16, torch.float32, True),
    (torch.bfloat16, torch.bfloat16, False)])
def test_gather(mixed, xdtype, msgdtype, weighted):
    g, rp_o, col_o, perm_o, w_o = mixed
    x, _, kw = x_pair(g, xdtype)
    w = dev(w_o) if weighted else None
    msg = mp.message_gather(dev(col_o), x, w=w, msg_dtype=msgdtype)
    torch.cuda.synchronize()
    ref = oracle.message_gather(col_o, w=w_o if weighted else None, **kw)
    assert np.array_equal(host_f32(msg).view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("F", [1, 3, 8, 24, 100, 128, 300, 520])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_gather_feature_widths_and_offsets(F, dtype):
    """Every chunk width (odd F forces single elements), and a table view that
    starts one element into its buffer (misaligned for vector accesses)."""
    rng = np.random.default_rng(F)
    n, E = 400, 5003
    x32 = rng.standard_normal((n, F)).astype(np.float32)
    idx = rng.integers(0, n, E).astype(np.int32)
    w = rng.standard_normal(E).astype(np.float32)
    for offset in (0, 1):
        if dtype == torch.float32:
            buf = dev(np.concatenate([np.zeros(offset, np.float32), x32.ravel()]))
            kw = {"x": x32}
        else:
            xb = graphgen.f32_to_bf16(x32)
            buf = bf16_dev(np.concatenate([np.zeros(offset, np.uint16), xb.ravel()]))
            kw = {"x_bf16": xb}
        x = buf[offset:].view(n, F)
        msg = mp.message_gather(dev(idx), x, w=dev(w))
        torch.cuda.synchronize()
        ref = oracle.message_gather(idx, w=w, **kw)
        assert np.array_equal(host_f32(msg).view(np.uint32), ref.view(np.uint32)), offset


def test_csr_rows_and_destination_gather(mixed):
    g, rp_o, col_o, _, _ = mixed
    rp = dev(rp_o.astype(np.int32))
    row = mp.csr_rows(rp, g.E)
    row_o = np.repeat(np.arange(g.n_dst), np.diff(rp_o)).astype(np.int32)
    assert np.array_equal(row.cpu().numpy(), row_o)
    # x_i of every edge: gather of the destination rows (a square graph)
    xi = mp.message_gather(row, dev(g.x))
    torch.cuda.synchronize()
    assert np.array_equal(host_f32(xi), oracle.message_gather(row_o, x=g.x))


# ---- edge-mask callback ----------------------------------------------------------------------

@pytest.mark.parametrize("by_perm", [False, True])
@pytest.mark.parametrize("in_place", [False, True])
def test_scale(mixed, by_perm, in_place):
    g, rp_o, col_o, perm_o, _ = mixed
    rng = np.random.default_rng(2)
    mask = rng.uniform(0.0, 1.0, g.E).astype(np.float32)
    m_o = oracle.message_gather(col_o, x=g.x)
    idx = perm_o.astype(np.int32) if by_perm else None
    msg = dev(m_o)
    out = mp.message_scale(msg, dev(mask), idx=None if idx is None else dev(idx),
                           out=msg if in_place else None)
    torch.cuda.synchronize()
    ref = oracle.message_scale(m_o, mask, idx)
    assert np.array_equal(out.cpu().numpy().view(np.uint32), ref.view(np.uint32))


# ---- aggregation of materialized messages ------------------------------------------------------

@pytest.mark.parametrize("reduce", list(REDUCES))
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("use_plan", [False, True])
def test_aggregate(mixed, reduce, dtype, use_plan):
    g, rp_o, col_o, _, _ = mixed
    x, _, kw = x_pair(g, dtype)
    rp = dev(rp_o.astype(np.int32))
    msg = mp.message_gather(dev(col_o), x, msg_dtype=dtype)
    plan = mp.Plan(rp, g.E, g.F, dtype) if use_plan else None
    r = REDUCES[reduce]
    out, out_max, argout = mp.message_aggregate(rp, msg, r, plan=plan)
    torch.cuda.synchronize()
    ref = oracle.aggregate_messages(rp_o, **({"msg": oracle.message_gather(col_o, **kw)}))
    compare_aggregate(ref, rp_o, out, out_max, argout, r, dtype)


@pytest.mark.parametrize("thresholds", [(8, 64, 16), (1, 2, 1)])
def test_aggregate_plan_regimes(mixed, thresholds):
    """Small hub thresholds send most rows through the hub-chunk path."""
    g, rp_o, col_o, _, _ = mixed
    rp = dev(rp_o.astype(np.int32))
    msg = mp.message_gather(dev(col_o), dev(g.x))
    plan = mp.Plan(rp, g.E, g.F, torch.float32, opts=thresholds)
    out, out_max, argout = mp.message_aggregate(rp, msg, mp.MP_SUM | mp.MP_MAX, plan=plan)
    torch.cuda.synchronize()
    ref = oracle.aggregate_messages(rp_o, oracle.message_gather(col_o, x=g.x))
    compare_aggregate(ref, rp_o, out, out_max, argout, mp.MP_SUM | mp.MP_MAX, torch.float32)


@pytest.mark.parametrize("use_plan", [False, True])
@pytest.mark.parametrize("weighted", [False, True])
def test_identity_callback_equals_fused_spmm(mixed, use_plan, weighted):
    """Unweighted fp32 features: the same kernels over the same values in the
    same order, so every output equals the fused call bitwise.  Weighted: the
    fused sum may contract the product into its add (one rounding fewer), so
    sums agree to the tolerance; max and argmax stay bitwise equal."""
    g, rp_o, col_o, _, w_o = mixed
    rp, col, x = dev(rp_o.astype(np.int32)), dev(col_o), dev(g.x)
    w = dev(w_o) if weighted else None
    plan = mp.Plan(rp, g.E, g.F, torch.float32) if use_plan else None
    r = mp.MP_SUM | mp.MP_MAX
    a = mp.spmm_materialized(rp, col, x, r, w=w, plan=plan)
    b = mp.spmm(rp, col, x, r, w=w, plan=plan)
    torch.cuda.synchronize()
    assert torch.equal(a[1], b[1]) and torch.equal(a[2], b[2])
    if not weighted:
        assert torch.equal(a[0], b[0])
    else:
        ref = oracle.spmm(rp_o, col_o, x=g.x, w=w_o)
        assert scaled_error(host_f32(a[0]), ref["sum"], ref["scale"]) <= 1e-5
        assert scaled_error(host_f32(b[0]), ref["sum"], ref["scale"]) <= 1e-5


@pytest.mark.parametrize("reduce", ["sum", "mean+max"])
@pytest.mark.parametrize("use_plan", [False, True])
def test_edge_mask_callback(mixed, reduce, use_plan):
    """The explainer's callback: messages times a per-COO-edge mask, applied
    through the library on the call's stream."""
    g, rp_o, col_o, perm_o, w_o = mixed
    mask = np.random.default_rng(5).uniform(0.0, 1.0, g.E).astype(np.float32)
    rp, col, x, w = dev(rp_o.astype(np.int32)), dev(col_o), dev(g.x), dev(w_o)
    perm, maskd = dev(perm_o.astype(np.int32)), dev(mask)
    plan = mp.Plan(rp, g.E, g.F, torch.float32) if use_plan else None
    r = REDUCES[reduce]
    out, out_max, argout, msg = mp.spmm_materialized(
        rp, col, x, r, w=w, plan=plan,
        callback=lambda m: mp.message_scale(m, maskd, idx=perm, out=m))
    torch.cuda.synchronize()
    ref, m_o = oracle.spmm_materialized(
        rp_o, col_o, x=g.x, w=w_o,
        callback=lambda m: oracle.message_scale(m, mask, perm_o.astype(np.int32)))
    assert np.array_equal(msg.cpu().numpy().view(np.uint32), m_o.view(np.uint32))
    compare_aggregate(ref, rp_o, out, out_max, argout, r, torch.float32)


def test_torch_callback_perturbation(mixed):
    """A callback written with torch ops (enqueued on the current stream):
    drop every third message and halve the rest (exact operations)."""
    g, rp_o, col_o, _, _ = mixed
    rp, col, x = dev(rp_o.astype(np.int32)), dev(col_o), dev(g.x)

    def c_torch(m):
        m.mul_(0.5)
        m[::3] = 0.0

    def c_np(m):
        m = m * np.float32(0.5)
        m[::3] = 0.0
        return m

    out, out_max, argout, _ = mp.spmm_materialized(rp, col, x, mp.MP_MEAN | mp.MP_MAX,
                                                   callback=c_torch)
    torch.cuda.synchronize()
    ref, _ = oracle.spmm_materialized(rp_o, col_o, x=g.x, callback=c_np)
    compare_aggregate(ref, rp_o, out, out_max, argout, mp.MP_MEAN | mp.MP_MAX, torch.float32)


def test_callback_failure_leaves_outputs_untouched(mixed):
    g, rp_o, col_o, _, _ = mixed
    rp, col, x = dev(rp_o.astype(np.int32)), dev(col_o), dev(g.x)
    E, F = g.E, g.F
    msg = torch.empty(E, F, device=DEV)
    out = torch.full((g.n_dst, F), 7.0, device=DEV)

    def bad(m):
        raise RuntimeError("callback refused")

    c = mp.MESSAGE_FN(lambda *a: 1)
    with pytest.raises(mp.MPError) as e:
        mp.mp_spmm_materialized(None, rp, mp.MP_I32, col, None, x, mp.MP_F32, g.n_src, g.n_dst,
                                E, F, msg, mp.MP_F32, c, None, mp.MP_SUM, out, mp.MP_F32, None,
                                mp.MP_F32, None, None, 0)
    assert e.value.status == mp.MP_ERR_CALLBACK
    with pytest.raises(mp.MPError) as e:
        mp.spmm_materialized(rp, col, x, mp.MP_SUM, callback=bad)
    assert isinstance(e.value.__cause__, RuntimeError)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
    # the gather ran before the callback
    assert np.array_equal(msg.cpu().numpy(), oracle.message_gather(col_o, x=g.x))


def test_empty_graph():
    rp = torch.zeros(6, dtype=torch.int32, device=DEV)
    col = torch.empty(1, dtype=torch.int32, device=DEV)[:0]
    x = torch.randn(4, 8, device=DEV)
    out, out_max, argout, msg = mp.spmm_materialized(rp, col, x, mp.MP_SUM | mp.MP_MAX)
    torch.cuda.synchronize()
    assert msg.shape == (0, 8)
    assert bool((out == 0).all()) and bool((argout == -1).all()) and bool((out_max == 0).all())
    d = mp.message_backward(rp, torch.randn(5, 8, device=DEV), mp.MP_SUM, E=0)
    assert d.shape == (0, 8)


# ---- gradients ---------------------------------------------------------------------------------

@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
@pytest.mark.parametrize("gdtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("itype", [torch.int32, torch.int64])
def test_message_backward(mixed, reduce, gdtype, itype):
    g, rp_o, col_o, _, _ = mixed
    G = np.random.default_rng(9).standard_normal((g.n_dst, g.F)).astype(np.float32)
    Gb = graphgen.f32_to_bf16(G)
    rp = dev(rp_o.astype(np.int32 if itype == torch.int32 else np.int64))
    msg = mp.message_gather(dev(col_o), dev(g.x))
    _, _, argout = mp.message_aggregate(rp, msg, mp.MP_MAX)
    Gd = dev(G) if gdtype == torch.float32 else bf16_dev(Gb)
    dmsg = mp.message_backward(rp, Gd, REDUCES[reduce], E=g.E, argout=argout)
    torch.cuda.synchronize()
    ref_agg = oracle.aggregate_messages(rp_o, oracle.message_gather(col_o, x=g.x))
    gk = {"g": G} if gdtype == torch.float32 else {"g_bf16": Gb}
    ref = oracle.message_backward(rp_o, reduce, argout=ref_agg["argmax"], **gk)
    assert np.array_equal(dmsg.cpu().numpy().view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("F", [1, 3, 100, 300, 520])
@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
def test_message_backward_shapes(F, reduce):
    """Rows of 0 to 70,000 edges (a row's gradient streamed to many message
    rows), feature counts with 1-, 2- and 4-element chunks and rows wider
    than one pass of 64 chunks; argmax positions drawn within each row."""
    degs = np.array([0, 1, 5, 70_000, 0, 130, 2, 64, 65])
    n_dst = degs.size
    rp_o = np.concatenate([[0], np.cumsum(degs)]).astype(np.int64)
    E = int(rp_o[-1])
    rng = np.random.default_rng(F)
    G = rng.standard_normal((n_dst, F)).astype(np.float32)
    am = np.full((n_dst, F), -1, np.int64)
    for v in range(n_dst):
        if degs[v]:
            am[v] = rp_o[v] + rng.integers(0, degs[v], F)
    dmsg = mp.message_backward(dev(rp_o.astype(np.int32)), dev(G), REDUCES[reduce], E=E,
                               argout=dev(am.astype(np.int32)))
    torch.cuda.synchronize()
    ref = oracle.message_backward(rp_o, reduce, argout=am, g=G)
    assert np.array_equal(dmsg.cpu().numpy().view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("adtype,bdtype", [(torch.float32, torch.float32),
                                           (torch.bfloat16, torch.float32),
                                           (torch.float32, torch.bfloat16),
                                           (torch.bfloat16, torch.bfloat16)])
@pytest.mark.parametrize("F", [1, 5, 64, 100, 300])
def test_edge_dot(adtype, bdtype, F):
    rng = np.random.default_rng(F)
    E, n_b = 7001, 500
    a32 = rng.standard_normal((E, F)).astype(np.float32)
    b32 = rng.standard_normal((n_b, F)).astype(np.float32)
    bidx = rng.integers(0, n_b, E).astype(np.int32)
    oidx = rng.permutation(E).astype(np.int32)
    ak = {"a": a32} if adtype == torch.float32 else {"a_bf16": graphgen.f32_to_bf16(a32)}
    bk = {"b": b32} if bdtype == torch.float32 else {"b_bf16": graphgen.f32_to_bf16(b32)}
    ad = dev(a32) if adtype == torch.float32 else bf16_dev(ak["a_bf16"])
    bd = dev(b32) if bdtype == torch.float32 else bf16_dev(bk["b_bf16"])
    for bi, oi in ((bidx, oidx), (bidx, None)):
        out = mp.edge_dot(ad, bd, bidx=dev(bi), oidx=None if oi is None else dev(oi))
        again = mp.edge_dot(ad, bd, bidx=dev(bi), oidx=None if oi is None else dev(oi))
        torch.cuda.synchronize()
        assert torch.equal(out, again)  # a fixed reduction order
        ref, sc = oracle.edge_dot(bidx=bi, oidx=oi, **ak, **bk)
        e = scaled_error(out.cpu().numpy(), ref, sc)
        assert e <= 1e-5, e
    # both tables edge-indexed (the mask gradient: a = dL/d(masked), b = messages)
    bb = dev(rng.standard_normal((E, F)).astype(np.float32))
    out = mp.edge_dot(dev(a32), bb)
    torch.cuda.synchronize()
    ref, sc = oracle.edge_dot(a=a32, b=bb.cpu().numpy())
    assert scaled_error(out.cpu().numpy(), ref, sc) <= 1e-5


def test_explainer_chain(mixed):
    """One explainer step through the library: gather, edge-mask callback,
    mean aggregation, dL/dmsg, the mask gradient (COO order), the callback's
    input gradient, dL/dx over the transposed CSR with forward positions as
    columns, and dL/dw; each compared with the oracle's chain."""
    g, rp_o, col_o, perm_o, w_o = mixed
    rng = np.random.default_rng(4)
    mask = rng.uniform(0.1, 1.0, g.E).astype(np.float32)
    G = rng.standard_normal((g.n_dst, g.F)).astype(np.float32)
    perm32 = perm_o.astype(np.int32)
    rp, col, x, w = dev(rp_o.astype(np.int32)), dev(col_o), dev(g.x), dev(w_o)
    perm, maskd = dev(perm32), dev(mask)

    m_pre = mp.message_gather(col, x, w=w)
    m = mp.message_scale(m_pre, maskd, idx=perm)
    out, _, _ = mp.message_aggregate(rp, m, mp.MP_MEAN)
    dm = mp.message_backward(rp, dev(G), mp.MP_MEAN, E=g.E)
    dmask = mp.edge_dot(dm, m_pre, oidx=perm)
    dpre = mp.message_scale(dm, maskd, idx=perm)
    rpT, colT, posT, wT = mp.csr_transpose(rp, col, g.n_src, val=w)
    gx, _, _ = mp.spmm(rpT, posT, dpre, mp.MP_SUM, w=wT)
    gw = mp.edge_dot(dpre, x, bidx=col)
    torch.cuda.synchronize()

    m_pre_o = oracle.message_gather(col_o, x=g.x, w=w_o)
    m_o = oracle.message_scale(m_pre_o, mask, perm32)
    agg = oracle.aggregate_messages(rp_o, m_o)
    e = scaled_error(host_f32(out), agg["mean"], agg["scale"] / np.maximum(np.diff(rp_o), 1)[:, None])
    assert e <= 1e-5, e
    dm_o = oracle.message_backward(rp_o, "mean", g=G)
    assert np.array_equal(dm.cpu().numpy(), dm_o)
    dmask_o, s1 = oracle.edge_dot(a=dm_o, b=m_pre_o, oidx=perm32)
    assert scaled_error(dmask.cpu().numpy(), dmask_o, s1) <= 1e-5
    dpre_o = oracle.message_scale(dm_o, mask, perm32)
    assert np.array_equal(dpre.cpu().numpy(), dpre_o)
    gx_o, s2 = oracle.message_backward_x(col_o, g.n_src, dpre_o, w=w_o)
    assert scaled_error(gx.cpu().numpy(), gx_o, s2) <= 1e-5
    gw_o, s3 = oracle.edge_dot(a=dpre_o, b=g.x, bidx=col_o)
    assert scaled_error(gw.cpu().numpy(), gw_o, s3) <= 1e-5


def test_deterministic(mixed):
    g, rp_o, col_o, _, w_o = mixed
    rp, col, x, w = dev(rp_o.astype(np.int32)), dev(col_o), dev(g.x), dev(w_o)
    plan = mp.Plan(rp, g.E, g.F, torch.float32)
    a = mp.spmm_materialized(rp, col, x, mp.MP_MEAN | mp.MP_MAX, w=w, plan=plan)
    b = mp.spmm_materialized(rp, col, x, mp.MP_MEAN | mp.MP_MAX, w=w, plan=plan)
    torch.cuda.synchronize()
    for u, v in zip(a, b):
        assert torch.equal(u, v)


def test_chunglu_124M_materialized_sampled():
    """The 124M-edge graph in the explainer benchmark's configuration (fp32
    features, 49.5 GB of fp32 messages): gathered messages and the mask
    callback on sampled positions, sum and max of sampled rows (every
    hub-sized row plus 20k random rows), and dL/dmsg of sampled positions,
    all against the oracle."""
    g = graphgen.workload("chunglu-124M", seed=0, bf16=False)
    rp_o, col_o, perm_o, _ = oracle.coo_to_csr(g.src, g.dst, g.n_dst)
    rp, col, x = dev(rp_o.astype(np.int32)), dev(col_o), dev(g.x)
    mask = graphgen.uniform_f32(3, 9, g.E) * np.float32(0.5) + np.float32(0.5)
    perm32 = perm_o.astype(np.int32)
    plan = mp.Plan(rp, g.E, g.F, torch.float32)
    maskd, perm = dev(mask), dev(perm32)
    out, out_max, argout, msg = mp.spmm_materialized(
        rp, col, x, mp.MP_SUM | mp.MP_MAX, plan=plan,
        callback=lambda m: mp.message_scale(m, maskd, idx=perm, out=m))
    torch.cuda.synchronize()
    pos = np.unique(graphgen.uniform_ints(12, 5, 200_000, g.E).astype(np.int64))
    m_s = msg[dev(pos)].cpu().numpy()
    ref_m = oracle.message_scale(oracle.message_gather(col_o[pos], x=g.x), mask, perm32[pos])
    assert np.array_equal(m_s.view(np.uint32), ref_m.view(np.uint32))
    print("[note] sampled messages ok", file=sys.stderr, flush=True)
    deg = np.diff(rp_o)
    rows = np.unique(np.concatenate([np.nonzero(deg >= 2048)[0],
                                     graphgen.uniform_ints(11, 5, 20_000, g.n_dst)])).astype(np.int64)
    # the oracle aggregates the sampled rows' messages (recomputed on the host)
    seg = np.concatenate([[0], np.cumsum(deg[rows])]).astype(np.int64)
    p_rows = np.concatenate([np.arange(rp_o[r], rp_o[r + 1]) for r in rows])
    m_rows = oracle.message_scale(oracle.message_gather(col_o[p_rows], x=g.x), mask,
                                  perm32[p_rows])
    ref = oracle.aggregate_messages(seg, m_rows)
    e = scaled_error(host_f32(out)[rows], ref["sum"], ref["scale"])
    assert e <= 1e-5, e
    am = argout.cpu().numpy()[rows].astype(np.int64)
    # argout is a global message row; the sampled table renumbers positions
    shift = (rp_o[rows] - seg[:-1])[:, None]
    assert np.array_equal(am, np.where(ref["argmax"] >= 0, ref["argmax"] + shift, -1))
    assert np.array_equal(host_f32(out_max)[rows].view(np.uint32), ref["max"].view(np.uint32))
    print("[note] sampled rows ok", file=sys.stderr, flush=True)
    del msg
    # dL/dmsg of the max on every edge of the sampled rows, from the oracle's
    # argmax of those rows
    G = graphgen.normal_f32(0, 11, g.n_dst * g.F).reshape(g.n_dst, g.F)
    dmsg = mp.message_backward(rp, dev(G), mp.MP_MAX, E=g.E, argout=argout)
    torch.cuda.synchronize()
    d_s = dmsg[dev(p_rows)].cpu().numpy()
    ref_d = oracle.message_backward(seg, "max", g=G[rows], argout=ref["argmax"])
    assert np.array_equal(d_s.view(np.uint32), ref_d.view(np.uint32))
