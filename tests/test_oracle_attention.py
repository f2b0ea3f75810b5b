"""Pins for oracle.attention: a library routine (torch SDPA in fp64 on the CPU),
closed forms and structural special cases."""
import math

import numpy as np
import pytest
import torch

from oracle.attention import verify_attention_request


def _rand(rng, n_q, hq, hkv, length, d):
    q = rng.standard_normal((n_q, hq, d))
    k = rng.standard_normal((length, hkv, d))
    v = rng.standard_normal((length, hkv, d))
    return q, k, v


def _sdpa(q, k, v, scale):
    n_q, length = q.shape[0], k.shape[0]
    pos = length - n_q + np.arange(n_q)
    mask = torch.as_tensor(np.arange(length)[None, :] <= pos[:, None])
    qt = torch.as_tensor(q).permute(1, 0, 2)[None]      # [1, Hq, n_q, D]
    kt = torch.as_tensor(k).permute(1, 0, 2)[None]      # [1, Hkv, L, D]
    vt = torch.as_tensor(v).permute(1, 0, 2)[None]
    o = torch.nn.functional.scaled_dot_product_attention(
        qt, kt, vt, attn_mask=mask, scale=scale, enable_gqa=True)
    return o[0].permute(1, 0, 2).numpy()


@pytest.mark.parametrize("n_q,hq,hkv,length,d", [
    (5, 4, 2, 37, 64), (1, 16, 8, 50, 16), (9, 32, 8, 9, 8), (3, 8, 8, 33, 32), (7, 4, 1, 16, 8)])
def test_matches_torch_sdpa_fp64(n_q, hq, hkv, length, d):
    rng = np.random.default_rng(n_q * 1000 + length)
    q, k, v = _rand(rng, n_q, hq, hkv, length, d)
    scale = 1.0 / math.sqrt(d)
    np.testing.assert_allclose(verify_attention_request(q, k, v, scale), _sdpa(q, k, v, scale),
                               rtol=0, atol=1e-12)


def test_window_equal_to_context_is_plain_causal_attention():
    rng = np.random.default_rng(1)
    q, k, v = _rand(rng, 6, 2, 2, 6, 8)
    o = verify_attention_request(q, k, v, 0.3)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.as_tensor(q).permute(1, 0, 2), torch.as_tensor(k).permute(1, 0, 2),
        torch.as_tensor(v).permute(1, 0, 2), is_causal=True, scale=0.3).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(o, ref, atol=1e-12, rtol=0)


def test_single_visible_key_returns_its_value():
    rng = np.random.default_rng(2)
    q, k, v = _rand(rng, 1, 4, 2, 1, 16)
    o = verify_attention_request(q, k, v, 0.125)
    for h in range(4):
        np.testing.assert_array_equal(o[0, h], v[0, h // 2])


def test_zero_scale_averages_visible_values():
    rng = np.random.default_rng(3)
    n_q, length = 4, 21
    q, k, v = _rand(rng, n_q, 4, 4, length, 8)
    o = verify_attention_request(q, k, v, 0.0)
    for j in range(n_q):
        pos = length - n_q + j
        np.testing.assert_allclose(o[j], v[:pos + 1].mean(axis=0), atol=1e-13, rtol=0)


def test_gqa_groups_are_contiguous():
    # KV head g holds the constant value g+1: head h must read exactly h//G + 1.
    rng = np.random.default_rng(4)
    hq, hkv = 8, 2
    q, k, _ = _rand(rng, 3, hq, hkv, 40, 16)
    v = np.empty((40, hkv, 16))
    for g in range(hkv):
        v[:, g, :] = g + 1
    o = verify_attention_request(q, k, v, 0.2)
    for h in range(hq):
        np.testing.assert_allclose(o[:, h, :], h // (hq // hkv) + 1, atol=1e-13)


def test_causal_window_only_sees_the_past():
    # a huge value on the last key is visible only to the last query
    rng = np.random.default_rng(5)
    n_q, length = 5, 30
    q, k, v = _rand(rng, n_q, 2, 2, length, 8)
    v2 = v.copy()
    v2[length - 1] += 1e6
    a = verify_attention_request(q, k, v, 0.25)
    b = verify_attention_request(q, k, v2, 0.25)
    np.testing.assert_array_equal(a[:n_q - 1], b[:n_q - 1])
    assert np.all(np.abs(b[n_q - 1] - a[n_q - 1]) > 1.0)


def test_rows_are_convex_combinations():
    rng = np.random.default_rng(6)
    q, k, _ = _rand(rng, 4, 4, 2, 25, 8)
    ones = np.ones((25, 2, 8))
    np.testing.assert_allclose(verify_attention_request(q * 3, k, ones, 1.0), 1.0, atol=1e-13)
