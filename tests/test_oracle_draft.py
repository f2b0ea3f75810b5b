"""Pins for oracle.draft: exact rational inverse-CDF sampling on dyadic
inputs, the sampling theorem, closed forms, and the identity between K
single-query decode steps and one causal window (torch SDPA in fp64)."""
import math
from fractions import Fraction

import numpy as np
import torch
from scipy import stats

from oracle.draft import draft_request, sample


def _grid_uniforms(rng, n):
    return (rng.integers(0, 1 << 24, n) * 2.0**-24).astype(np.float32)


def test_sample_matches_exact_rational_inverse_cdf():
    # small integer weights and uniforms on the 2^-24 grid: every prefix sum and
    # u * total is exact in fp64, so the oracle must equal the rational definition
    rng = np.random.default_rng(0)
    for _ in range(300):
        v = int(rng.integers(1, 40))
        w = rng.integers(0, 5, v).astype(np.float64)
        if w.sum() == 0:
            w[int(rng.integers(0, v))] = 1.0
        u = _grid_uniforms(rng, 1)
        got = int(sample(w[None], u)[0])
        tau = Fraction(float(u[0])) * int(w.sum())
        run, want = Fraction(0), None
        for t in range(v):
            run += int(w[t])
            if run > tau:
                want = t
                break
        assert got == want


def test_sample_boundaries_and_degenerate_rows():
    w = np.array([[1.0, 3.0, 0.0, 4.0]])
    for u, y in ((0.0, 0), (0.125 - 2**-24, 0), (0.125, 1), (0.5 - 2**-24, 1), (0.5, 3),
                 (1.0 - 2**-24, 3)):
        assert sample(w, np.array([u]))[0] == y
    assert sample(np.zeros((1, 7)), np.array([0.3]))[0] == -1       # no mass
    one_hot = np.zeros((5, 9))
    one_hot[np.arange(5), [0, 8, 3, 3, 7]] = 0.25
    np.testing.assert_array_equal(sample(one_hot, np.array([0.0, 0.1, 0.5, 0.9, 1 - 2**-24])),
                                  [0, 8, 3, 3, 7])
    # rounding past the total: the last token with mass
    assert sample(np.array([[0.5, 0.5, 0.0]]), np.array([1.0]))[0] == 1


def test_samples_follow_the_row():
    rng = np.random.default_rng(1)
    row = rng.exponential(size=12) * (rng.random(12) > 0.25)
    u = _grid_uniforms(rng, 50000)
    draws = sample(np.broadcast_to(row, (len(u), 12)), u)
    counts = np.bincount(draws, minlength=12)
    assert counts[row == 0].sum() == 0
    nz = row > 0
    assert stats.chisquare(counts[nz], row[nz] / row.sum() * len(u)).pvalue > 1e-4
    # power: a uniform row is rejected
    assert stats.chisquare(counts[nz], np.full(nz.sum(), len(u) / nz.sum())).pvalue < 1e-6


def _sdpa_causal(q, k, v, scale):
    """q [n][Hq][D] at the last n positions of k, v [L][Hkv][D] (torch, fp64)."""
    n, length = q.shape[0], k.shape[0]
    pos = length - n + np.arange(n)
    mask = torch.as_tensor(np.arange(length)[None, :] <= pos[:, None])
    o = torch.nn.functional.scaled_dot_product_attention(
        torch.as_tensor(q).permute(1, 0, 2)[None], torch.as_tensor(k).permute(1, 0, 2)[None],
        torch.as_tensor(v).permute(1, 0, 2)[None], attn_mask=mask, scale=scale, enable_gqa=True)
    return o[0].permute(1, 0, 2).numpy()


def test_decode_steps_equal_one_causal_window():
    rng = np.random.default_rng(2)
    for p_len, n_steps, hq, hkv, d in ((0, 1, 2, 1, 8), (5, 4, 16, 8, 16), (31, 6, 4, 2, 32),
                                       (16, 3, 8, 8, 8)):
        kc = rng.standard_normal((p_len, hkv, d))
        vc = rng.standard_normal((p_len, hkv, d))
        qs = rng.standard_normal((n_steps, hq, d))
        ks = rng.standard_normal((n_steps, hkv, d))
        vs = rng.standard_normal((n_steps, hkv, d))
        probs = rng.random((n_steps, 10))
        u = _grid_uniforms(rng, n_steps)
        scale = 1.0 / math.sqrt(d)
        o, x = draft_request(kc, vc, qs, ks, vs, probs, u, scale)
        ref = _sdpa_causal(qs, np.concatenate([kc, ks]), np.concatenate([vc, vs]), scale)
        np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)
        np.testing.assert_array_equal(x, sample(probs, u))


def test_zero_scale_step_averages_cache_and_new_rows():
    # scale 0: step i's output is the mean of the P + i + 1 values it can see
    rng = np.random.default_rng(3)
    p_len, n_steps, hq, hkv, d = 7, 3, 4, 2, 8
    kc, vc = rng.standard_normal((2, p_len, hkv, d))
    ks, vs = rng.standard_normal((2, n_steps, hkv, d))
    qs = rng.standard_normal((n_steps, hq, d))
    o, _ = draft_request(kc, vc, qs, ks, vs, np.ones((n_steps, 3)), np.zeros(n_steps), 0.0)
    allv = np.concatenate([vc, vs])
    for i in range(n_steps):
        for h in range(hq):
            np.testing.assert_allclose(o[i, h], allv[:p_len + i + 1, h // 2].mean(0), atol=1e-14)


def test_a_dominant_new_key_returns_its_value():
    # a new key aligned with the query and scaled up takes all the weight
    rng = np.random.default_rng(4)
    kc, vc = rng.standard_normal((2, 9, 1, 4))
    qs = np.ones((2, 1, 4))
    ks = np.stack([np.full((1, 4), -50.0), np.full((1, 4), 50.0)])
    vs = rng.standard_normal((2, 1, 4))
    o, _ = draft_request(kc, vc, qs, ks, vs, np.ones((2, 3)), np.zeros(2), 1.0)
    np.testing.assert_allclose(o[1, 0], vs[1, 0], atol=1e-12)
    assert np.abs(o[0, 0] - vs[0, 0]).max() > 1e-3      # step 0's new key scores -200
