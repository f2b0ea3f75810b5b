"""Oracle for speculative acceptance with residual resampling.

The paper relies on the standard speculative-sampling rule of the works it
builds on (Leviathan et al. 2023; Chen et al. 2023, cited in Sections 1 and 2)
without restating it.  Written out for one request with K proposals x_0..x_{K-1}
drawn from draft rows q_0..q_{K-1}, target rows p_0..p_K and uniforms
u_0..u_K:

1. Proposal i is accepted when u_i * q_i(x_i) <= p_i(x_i); n is the first i
   that is not accepted, or K if all are.  (Equivalent to u_i <= p_i/q_i; the
   product of two fp32 values is exact in fp64, so the comparison is exact.)
2. If n < K, one token is drawn from the residual weights
   w(t) = max(0, p_n(t) - q_n(t)); if n = K, from p_K (the bonus token).
   Should the residual have no mass (p_n = q_n in fp32), p_n is used.
3. The draw is the inverse CDF: y = min{t : C(t) > u_K * S}, with C the
   inclusive prefix sum of w in token order and S = C(V-1), all in fp64.  If
   rounding leaves no such t, y is the last token of positive weight.
4. The request emits x_0..x_{n-1} then y; the remaining K - n slots hold -1.

A proposal token outside [0, V) is treated as not accepted.
"""
import numpy as np


def acceptance_length(p_rows, q_rows, draft, u):
    """Step 1: the number n of accepted proposals."""
    k = len(draft)
    vocab = p_rows.shape[1]
    for i in range(k):
        x = int(draft[i])
        if not (0 <= x < vocab):
            return i
        if not (float(u[i]) * float(q_rows[i][x]) <= float(p_rows[i][x])):
            return i
    return k


def residual_weights(p_rows, q_rows, n):
    """Step 2: the fp64 weights the emitted token is drawn from."""
    k = q_rows.shape[0]
    if n < k:
        w = np.maximum(0.0, p_rows[n].astype(np.float64) - q_rows[n].astype(np.float64))
        if np.cumsum(w)[-1] == 0.0:
            w = p_rows[n].astype(np.float64)
        return w
    return p_rows[k].astype(np.float64)


def inverse_cdf(w, u):
    """Step 3: y = min{t : C(t) > u * C(V-1)} over the sequential fp64 prefix sums."""
    c = np.cumsum(w)
    tau = float(u) * c[-1]
    y = int(np.searchsorted(c, tau, side="right"))
    if y >= len(w):
        y = int(np.nonzero(w > 0)[0][-1])
    return y


def accept_request(p_rows, q_rows, draft, u):
    """One request: returns (n, tokens) with tokens of length K + 1."""
    k = len(draft)
    n = acceptance_length(p_rows, q_rows, draft, u)
    y = inverse_cdf(residual_weights(p_rows, q_rows, n), u[k])
    tokens = np.full(k + 1, -1, dtype=np.int64)
    tokens[:n] = np.asarray(draft[:n])
    tokens[n] = y
    return n, tokens


def spec_accept(p_target, q_draft, draft_tokens, uniforms, q_indptr, requests=None):
    """The whole batch (or the listed requests) in the ragged layout.

    Request r owns target rows / uniforms / output slots q_indptr[r] .. q_indptr[r+1]-1
    and draft rows / tokens q_indptr[r] - r .. q_indptr[r+1] - r - 2.
    Returns (accepted_len [bs], out_tokens [total_q]); unlisted requests get -1.
    """
    bs = len(q_indptr) - 1
    acc = np.full(bs, -1, dtype=np.int64)
    out = np.full(int(q_indptr[-1]), -1, dtype=np.int64)
    for r in (range(bs) if requests is None else requests):
        a, b = int(q_indptr[r]), int(q_indptr[r + 1])
        k = b - a - 1
        n, tok = accept_request(p_target[a:b], q_draft[a - r:a - r + k],
                                draft_tokens[a - r:a - r + k], uniforms[a:b])
        acc[r] = n
        out[a:b] = tok
    return acc, out
