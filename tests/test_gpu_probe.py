"""The bandwidth probes (include/mp_probe.h) through the C ABI.  Every word a
probe loads is folded into an XOR, so the XOR of all sink words equals the
XOR of every word the probe was asked to read: an exact check that each probe
reads exactly its input (the read: the whole buffer; the gather: row idx[p]
for every p, once per index).  The scatter's output is compared whole."""
import numpy as np
import pytest
import torch

import paper_2507_16991_amd as mp

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def xor_all(a: np.ndarray) -> int:
    return int(np.bitwise_xor.reduce(a.view(np.uint32).ravel()))


def sink():
    return torch.zeros(mp.MP_PROBE_SINK_WORDS, dtype=torch.int32, device=DEV)


@pytest.mark.parametrize("nbytes", [16, 4096, 1 << 20, (1 << 24) + 48])
def test_probe_read_and_copy(nbytes):
    rng = np.random.default_rng(nbytes)
    h = rng.integers(0, 2**32, nbytes // 4, dtype=np.uint32)
    d = torch.from_numpy(h.view(np.int32)).to(DEV)
    s = sink()
    mp.mp_probe_read(d, nbytes, s)
    out = torch.empty_like(d)
    mp.mp_probe_copy(d, out, nbytes)
    torch.cuda.synchronize()
    assert xor_all(s.cpu().numpy()) == xor_all(h)
    assert torch.equal(out, d)


@pytest.mark.parametrize("row_bytes,stride", [(16, 16), (400, 400), (256, 256), (200 + 8, 256),
                                              (1024, 1024), (48, 64)])
@pytest.mark.parametrize("n", [0, 1, 63, 1000, 70_001])
def test_probe_gather(row_bytes, stride, n):
    if row_bytes % 16:
        pytest.skip("row bytes must be whole 16-byte chunks")
    rng = np.random.default_rng(n + row_bytes)
    rows = 5000
    tab = rng.integers(0, 2**32, rows * stride // 4, dtype=np.uint32)
    idx = rng.integers(0, rows, n).astype(np.int32)
    s = sink()
    mp.mp_probe_gather(torch.from_numpy(idx).to(DEV) if n else torch.zeros(1, dtype=torch.int32,
                                                                            device=DEV),
                       n, torch.from_numpy(tab.view(np.int32)).to(DEV), stride, row_bytes, s)
    torch.cuda.synchronize()
    t2 = tab.reshape(rows, stride // 4)[:, :row_bytes // 4]
    expect = xor_all(t2[idx]) if n else 0
    assert xor_all(s.cpu().numpy()) == expect


@pytest.mark.parametrize("elem_bytes", [4, 8])
@pytest.mark.parametrize("n", [1, 63, 1000, 70_001, 1 << 20])
def test_probe_scatter(elem_bytes, n):
    """out[dest[i]] = in[i] for a random permutation dest (exact)."""
    rng = np.random.default_rng(n + elem_bytes)
    dt = np.int64 if elem_bytes == 8 else np.int32
    h = rng.integers(-2**31, 2**31, n).astype(dt)
    dest = rng.permutation(n).astype(np.int32)
    d_in = torch.from_numpy(h).to(DEV)
    out = torch.zeros_like(d_in)
    mp.mp_probe_scatter(d_in, torch.from_numpy(dest).to(DEV), n, elem_bytes, out)
    torch.cuda.synchronize()
    expect = np.empty_like(h)
    expect[dest] = h
    assert np.array_equal(out.cpu().numpy(), expect)
