"""Pins for oracle.accept: exact special cases, the inverse-CDF convention on
exactly representable weights, and the speculative-sampling theorem (the
emitted token is distributed as the target row) by chi-square."""
import numpy as np
import pytest
from scipy import stats

from oracle.accept import (accept_request, acceptance_length, inverse_cdf,
                           residual_weights, spec_accept)


def _probs(rng, vocab, sigma=1.0):
    z = sigma * rng.standard_normal(vocab)
    p = np.exp(z - z.max())
    return (p / p.sum()).astype(np.float32)


def test_identical_rows_accept_everything():
    rng = np.random.default_rng(0)
    k, vocab = 5, 50
    p = np.stack([_probs(rng, vocab) for _ in range(k + 1)])
    q = p[:k].copy()
    for trial in range(200):
        x = rng.integers(0, vocab, k)
        u = (rng.integers(0, 1 << 24, k + 1) * 2.0**-24).astype(np.float32)
        assert acceptance_length(p, q, x, u) == k


def test_zero_target_probability_rejects():
    rng = np.random.default_rng(1)
    k, vocab = 4, 20
    p = np.stack([_probs(rng, vocab) for _ in range(k + 1)])
    q = np.stack([_probs(rng, vocab) for _ in range(k)])
    x = np.array([3, 7, 11, 2])
    p[2, 11] = 0.0
    u = np.zeros(k + 1, np.float32) + np.float32(1e-7)   # accepts whenever p(x) > 0 ... almost
    n = acceptance_length(p, q, x, u)
    assert n <= 2


def test_one_hot_residual_is_forced():
    vocab, t_star = 10, 6
    p = np.zeros((2, vocab), np.float32)
    q = np.zeros((1, vocab), np.float32)
    p[0, t_star] = 1.0
    q[0, 2] = 1.0                       # proposal 2 has p = 0: rejected
    p[1, 0] = 1.0
    n, tok = accept_request(p, q, np.array([2]), np.array([0.3, 0.77], np.float32))
    assert n == 0 and list(tok) == [t_star, -1]


def test_exact_tie_is_accepted():
    p = np.array([[0.25, 0.75], [0.5, 0.5]], np.float32)
    q = np.array([[0.5, 0.5]], np.float32)
    # u * q(x) = 0.5 * 0.5 = 0.25 = p(x): accepted (<=)
    assert acceptance_length(p, q, np.array([0]), np.array([0.5, 0.1], np.float32)) == 1
    assert acceptance_length(p, q, np.array([0]), np.array([0.5 + 2**-24, 0.1], np.float32)) == 0


def test_inverse_cdf_boundaries_on_exact_weights():
    w = np.array([0.25, 0.25, 0.0, 0.5])
    assert inverse_cdf(w, 0.0) == 0
    assert inverse_cdf(w, 0.25 - 2**-24) == 0
    assert inverse_cdf(w, 0.25) == 1          # C(0) = 0.25 is not > 0.25
    assert inverse_cdf(w, 0.5) == 3           # the zero-weight token 2 is skipped
    assert inverse_cdf(w, 1.0 - 2**-24) == 3
    assert inverse_cdf(np.array([0.5, 0.5, 0.0]), 1.0) == 1   # overflow: last positive weight


def test_zero_weight_tokens_are_never_drawn():
    w = np.array([0.0, 0.3, 0.0, 0.0, 0.7, 0.0])
    for u in np.arange(0, 1 << 12) * 2.0**-12:
        assert w[inverse_cdf(w, u)] > 0


def test_residual_rule_and_fallback():
    p = np.array([[0.5, 0.25, 0.25], [0.2, 0.2, 0.6]], np.float32)
    q = np.array([[0.25, 0.5, 0.25]], np.float32)
    np.testing.assert_array_equal(residual_weights(p, q, 0), [0.25, 0.0, 0.0])
    np.testing.assert_array_equal(residual_weights(p, q, 1), p[1].astype(np.float64))
    same = np.array([[0.5, 0.5], [0.1, 0.9]], np.float32)
    np.testing.assert_array_equal(residual_weights(same, same[:1], 0), [0.5, 0.5])


def test_out_of_vocabulary_proposal_is_rejected():
    p = np.full((2, 4), 0.25, np.float32)
    assert acceptance_length(p, p[:1], np.array([4]), np.array([0.0, 0.5], np.float32)) == 0


def _simulate(p, q, trials, seed):
    rng = np.random.default_rng(seed)
    k, vocab = q.shape
    qq = q.astype(np.float64)
    xs = np.stack([rng.choice(vocab, size=trials, p=qq[i] / qq[i].sum()) for i in range(k)], 1)
    us = (rng.integers(0, 1 << 24, (trials, k + 1)) * 2.0**-24).astype(np.float32)
    first, second = [], []
    for x, u in zip(xs, us):
        n, tok = accept_request(p, q, x, u)
        first.append(tok[0])
        if n >= 1:
            second.append(tok[1])
    return np.array(first), np.array(second)


def test_emitted_tokens_follow_the_target_rows():
    # speculative-sampling theorem: token 0 ~ p_0 and, given proposal 0 was
    # accepted, token 1 ~ p_1, whatever the draft rows are.
    rng = np.random.default_rng(7)
    vocab = 6
    p = np.stack([_probs(rng, vocab, 1.5) for _ in range(3)]).astype(np.float64)
    q = np.stack([_probs(rng, vocab, 1.5) for _ in range(2)]).astype(np.float64)
    p = (p / p.sum(1, keepdims=True)).astype(np.float32)
    q = (q / q.sum(1, keepdims=True)).astype(np.float32)
    first, second = _simulate(p, q, 60000, 11)
    for tokens, row in ((first, p[0]), (second, p[1])):
        counts = np.bincount(tokens, minlength=vocab)
        r64 = row.astype(np.float64)
        exp = r64 / r64.sum() * len(tokens)
        assert stats.chisquare(counts, exp).pvalue > 1e-4
    # the residual alone is NOT distributed as p_0 (the test has power)
    w = np.maximum(0, p[0] - q[0]).astype(np.float64)
    counts = np.bincount(first, minlength=vocab)
    w = np.maximum(w / w.sum(), 1e-12)
    assert stats.chisquare(counts, w / w.sum() * len(first)).pvalue < 1e-6


def test_acceptance_probability_is_min_one_ratio():
    rng = np.random.default_rng(8)
    p = np.array([[0.1, 0.6, 0.3], [1/3, 1/3, 1/3]], np.float32)
    q = np.array([[0.4, 0.2, 0.4]], np.float32)
    for x, expect in ((0, 0.25), (1, 1.0), (2, 0.75)):
        u = (rng.integers(0, 1 << 24, 40000) * 2.0**-24).astype(np.float32)
        acc = np.mean([acceptance_length(p, q, np.array([x]), np.array([ui, 0.5], np.float32))
                       for ui in u])
        assert abs(acc - expect) < 0.01


def test_ragged_batch_layout():
    # request r, row i: every row is one-hot at token 10r + i and the proposal
    # is that token, so the emitted tokens spell out which rows were read.
    depth = [2, 0, 3]
    bs, vocab = len(depth), 64
    q_indptr = np.concatenate([[0], np.cumsum(np.array(depth) + 1)])
    p = np.zeros((q_indptr[-1], vocab), np.float32)
    q = np.zeros((q_indptr[-1] - bs, vocab), np.float32)
    x = np.zeros(q_indptr[-1] - bs, np.int32)
    for r, k in enumerate(depth):
        for i in range(k + 1):
            p[q_indptr[r] + i, 10 * r + i] = 1.0
        for i in range(k):
            q[q_indptr[r] - r + i, 10 * r + i] = 1.0
            x[q_indptr[r] - r + i] = 10 * r + i
    u = np.full(q_indptr[-1], 0.5, np.float32)
    acc, out = spec_accept(p, q, x, u, q_indptr)
    assert list(acc) == depth
    assert list(out) == [0, 1, 2, 10, 20, 21, 22, 23]
