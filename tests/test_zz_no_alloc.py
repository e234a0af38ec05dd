"""mp_spmm_noalloc, the aggregation entry point for callers that cannot
allocate device memory, against mp_spmm (the same kernels with a caller
workspace), through the C ABI: two calls in a row, the second with a smaller
input (the static scratch array keeps the first call's partials), with plans
whose small thresholds give many hub chunks, so the scratch is really used.
Outputs must be bit-identical to mp_spmm's with the same plan; a call whose
hub partials exceed the array is rejected before anything is enqueued."""
import sys

import numpy as np
import pytest
import torch

import graphgen
import oracle
import paper_2507_16991_amd as mp

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def both(g, dtype, reduce, weighted, opts):
    rp_o, col_o, _, w_o = oracle.coo_to_csr(g.src, g.dst, g.n_dst, val=g.w)
    rp, col = dev(rp_o.astype(np.int32)), dev(col_o)
    w = dev(w_o) if weighted else None
    x = dev(g.x) if dtype == torch.float32 else dev(g.x_bf16.view(np.int16)).view(torch.bfloat16)
    plan = mp.Plan(rp, g.E, g.F, dtype, opts=opts)
    need = mp.mp_spmm_workspace(plan.handle, reduce)
    assert 0 < need <= mp.MP_NOALLOC_SCRATCH_BYTES
    ref = mp.spmm(rp, col, x, reduce, w=w, plan=plan)
    hs = bool(reduce & (mp.MP_SUM | mp.MP_MEAN))
    hm = bool(reduce & mp.MP_MAX)
    N, F = g.n_dst, g.F
    out = torch.full((N, F), 7.0, device=DEV) if hs else None
    out_max = torch.full((N, F), 7.0, device=DEV) if hm else None
    argout = torch.full((N, F), -7, dtype=torch.int32, device=DEV) if hm else None
    mp.mp_spmm_noalloc(plan.handle, rp, mp.MP_I32, col, w, x, mp.MP_F32 if dtype == torch.float32
                       else mp.MP_BF16, g.n_src, N, F, F, reduce, out, mp.MP_F32, out_max,
                       mp.MP_F32, argout)
    torch.cuda.synchronize()
    for a, b in zip(ref, (out, out_max, argout)):
        if a is not None:
            assert torch.equal(a.view(torch.int32), b.view(torch.int32)), "differs from mp_spmm"
    return need


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_noalloc_equals_spmm_two_calls(dtype):
    big = graphgen.chung_lu_graph(3, 20_000, 400_000, 64, dmax=20_000.0)
    big.w = graphgen.uniform_f32(3, 7, big.E)
    small = graphgen.mixed_graph(4, n=900, e=12_000, f=64)
    for reduce, weighted in ((mp.MP_SUM | mp.MP_MAX, False), (mp.MP_MEAN, True),
                             (mp.MP_MAX, True)):
        n1 = both(big, dtype, reduce, weighted, (8, 64, 16))
        n2 = both(small, dtype, reduce, weighted, (8, 64, 16))
        assert n2 < n1, "the second call is the smaller one"
        sys.stderr.write(f"noalloc {dtype} reduce {reduce}: scratch {n1} then {n2} bytes\n")


def test_noalloc_rejects_oversized_partials():
    """One row of 4096 edges cut into 2048 chunks at F = 4096: the sum|max
    partials need 2048 * 4096 * 12 bytes > MP_NOALLOC_SCRATCH_BYTES."""
    F, n_src, E = 4096, 16, 4096
    src = (np.arange(E) % n_src).astype(np.int32)
    dst = np.zeros(E, np.int32)
    rp_o, col_o, _, _ = oracle.coo_to_csr(src, dst, 1, n_src=n_src)
    rp, col = dev(rp_o.astype(np.int32)), dev(col_o)
    x = torch.zeros(n_src, F, device=DEV)
    plan = mp.Plan(rp, E, F, torch.float32, opts=(1, 2, 1))
    assert mp.mp_spmm_workspace(plan.handle, mp.MP_SUM | mp.MP_MAX) > mp.MP_NOALLOC_SCRATCH_BYTES
    out = torch.full((1, F), 3.0, device=DEV)
    out_max = torch.full((1, F), 3.0, device=DEV)
    argout = torch.full((1, F), 5, dtype=torch.int32, device=DEV)
    with pytest.raises(mp.MPError) as e:
        mp.mp_spmm_noalloc(plan.handle, rp, mp.MP_I32, col, None, x, mp.MP_F32, n_src, 1, F, F,
                           mp.MP_SUM | mp.MP_MAX, out, mp.MP_F32, out_max, mp.MP_F32, argout)
    assert e.value.status == -5
    torch.cuda.synchronize()
    assert bool((out == 3.0).all()) and bool((argout == 5).all()), "outputs untouched"
    # the sum alone (4 bytes per partial) fits
    mp.mp_spmm_noalloc(plan.handle, rp, mp.MP_I32, col, None, x, mp.MP_F32, n_src, 1, F, F,
                       mp.MP_SUM, out, mp.MP_F32, None, mp.MP_F32, None)
    torch.cuda.synchronize()
    assert bool((out == 0.0).all())
