"""Checks of the seeded input generators (not part of the method).

SplitMix64 is re-derived here in pure Python from its published definition;
bf16 rounding is checked against torch's round-to-nearest-even conversion; the
samplers are checked for range, moments, frequencies and thread-count
independence.
"""
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

import graphgen

M64 = (1 << 64) - 1
G = 0x9E3779B97F4A7C15


def mix(z):
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def test_splitmix_published_sequence():
    # SplitMix64 started at state 0: first outputs (reference values of the
    # published generator: state += G; output = mix(state)).
    L = graphgen._L()
    assert L.gg_draw(0, 0) == 0xE220A8397B1DCDAF
    assert L.gg_draw(0, 1) == 0x6E789E6AA1B965F4
    assert L.gg_draw(0, 2) == 0x06C45D188009454F
    for i in range(3):
        assert L.gg_draw(0, i) == mix((G * (i + 1)) & M64)


def test_key_and_draw_formula():
    seed, stream = 7, 3
    key = mix((mix((seed + G) & M64) ^ ((stream * G + 0x632BE59BD9B4E019) & M64)) & M64)
    d = graphgen.draws(seed, stream, 5)
    assert [int(v) for v in d] == [mix((key + (i + 1) * G) & M64) for i in range(5)]


def test_uniform_ints_range_and_formula():
    a = graphgen.uniform_ints(1, 1, 1000, 37)
    assert a.min() >= 0 and a.max() < 37
    d = graphgen.draws(1, 1, 10)
    assert a[:10].tolist() == [(int(v) * 37) >> 64 for v in d]


def test_uniform_f32_exact_grid():
    u = graphgen.uniform_f32(0, 3, 100000)
    assert np.all(np.abs(u) < 1) and np.all(u != 0)
    k = (u.astype(np.float64) * 2 ** 24 + 2 ** 24 - 1) / 2
    assert np.all(k == np.round(k))
    assert abs(u.mean()) < 0.01


def test_normal_moments():
    z = graphgen.normal_f32(0, 3, 400000).astype(np.float64)
    assert abs(z.mean()) < 0.01 and abs(z.std() - 1) < 0.01


def test_bf16_matches_torch_rne():
    x = np.concatenate([graphgen.normal_f32(1, 3, 100000),
                        np.array([1.00390625, 1.01171875, -1.00390625, 0.0, -0.0, 3.4e38],
                                 np.float32)])
    ours = graphgen.f32_to_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_permutation_is_permutation():
    p = graphgen.permutation(0, 4, 10007)
    assert np.array_equal(np.sort(p), np.arange(10007))


def test_alias_frequencies():
    n, e, beta = 50, 400000, 0.9
    perm = np.arange(n, dtype=np.int32)
    s = graphgen.powerlaw_endpoints(0, 2, n, e, beta, perm)
    pr = np.arange(1, n + 1, dtype=np.float64) ** -beta
    pr /= pr.sum()
    freq = np.bincount(s, minlength=n) / e
    assert np.max(np.abs(freq - pr) / np.sqrt(pr / e)) < 5.0


def test_gcn_weights_formula():
    g = graphgen.workload("powerlaw-1.2M", seed=0, scale=0.05)
    od = np.bincount(g.src, minlength=g.n_src).astype(np.float64)
    idg = np.bincount(g.dst, minlength=g.n_dst).astype(np.float64)
    ref = (1.0 / np.sqrt(od[g.src] * idg[g.dst])).astype(np.float32)
    assert np.array_equal(g.w, ref)


def test_chunglu_beta_fit():
    b = graphgen.fit_beta(2_449_029, 123_718_280, 17_000.0)
    assert abs(b - graphgen.CHUNGLU_124M_BETA) < 5e-5


def test_powerlaw_workload_shape():
    g = graphgen.workload("powerlaw-1.2M", seed=0)
    deg = np.bincount(g.dst, minlength=g.n_dst)
    assert g.E == 1_166_243 and g.n_dst == 169_343
    assert 30_000 < deg.max() < 80_000        # expected top in-degree ~52k
    assert 0.12 < (deg == 0).mean() < 0.24    # ~18% empty rows


def test_thread_count_independence():
    code = ("import graphgen, hashlib; g = graphgen.workload('powerlaw-1.2M', seed=5, scale=0.2);"
            "h = hashlib.sha1(); [h.update(a.tobytes()) for a in (g.src, g.dst, g.x, g.w)];"
            "print(h.hexdigest())")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    outs = []
    for t in ("1", "5"):
        env = dict(os.environ, OMP_NUM_THREADS=t, PYTHONPATH=root)
        outs.append(subprocess.check_output([sys.executable, "-c", code], env=env, cwd=root))
    assert outs[0] == outs[1]


def test_uniform_bf16_is_rounding_of_uniform_f32():
    a = graphgen.uniform_bf16(3, 3, 50_000)
    b = graphgen.f32_to_bf16(graphgen.uniform_f32(3, 3, 50_000))
    assert np.array_equal(a, b)
