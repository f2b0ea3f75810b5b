"""Oracle for the draft stage that precedes a verification round -- TEST
INFRASTRUCTURE (imported only by the test suite, the smoke check and the CPU
baseline of the benchmark).

Each speculative iteration runs the draft stage before the target stage
(Eq. 1).  The draft model proposes a chain of K tokens autoregressively: at
step i it processes one token (the anchor at step 0, proposal x_{i-1} after),
whose K/V it appends to its paged cache, attends with that token's single
query over the whole cache, and draws x_i from its output distribution q_i
(speculative decoding as the paper builds on it, Sections 1 and 2; proposal
depth d, Appendix H).  The draft model's projections and vocabulary head need
its weights and lie outside this oracle: per step the query, the new K/V row
and q_i are inputs.

* ``sample``       -- x ~ w by inverse CDF with one uniform: the first token
                      whose running sum exceeds u times the row total, the
                      same convention as the acceptance step's resampling;
                      a row without mass yields -1.
* ``draft_request`` -- the K steps of one request, in order: append, attend
                      (one query at the newest position), sample.
"""
import numpy as np

from .attention import verify_attention_request


def sample(rows, u):
    """rows: [n][V] nonnegative weights (any total), u: [n] in [0, 1) -> int64 [n].

    y = min{t : C(t) > u * C(V-1)} over sequential fp64 prefix sums C; if
    rounding leaves no such t, the last token with positive weight; -1 when
    the row has no mass."""
    rows = np.asarray(rows, dtype=np.float64)
    out = np.full(len(rows), -1, dtype=np.int64)
    for i, w in enumerate(rows):
        c = np.cumsum(w)
        if not c[-1] > 0.0:
            continue
        tau = float(u[i]) * c[-1]
        y = int(np.searchsorted(c, tau, side="right"))
        if y >= len(w):
            y = int(np.nonzero(w > 0)[0][-1])
        out[i] = y
    return out


def draft_request(k_ctx, v_ctx, q_steps, k_steps, v_steps, probs, u, scale):
    """The K draft steps of one request.

    k_ctx, v_ctx: [P][Hkv][D], the cache before the stage (P tokens; the
    anchor is not in it yet).  Step i appends k_steps[i], v_steps[i]
    ([Hkv][D]) at position P + i, attends with q_steps[i] ([Hq][D]) over
    positions 0 .. P + i, and draws x_i from probs[i] ([V]) with u[i].
    Returns (o [K][Hq][D] float64, x [K] int64)."""
    n_steps = len(q_steps)
    k = np.asarray(k_ctx, dtype=np.float64)
    v = np.asarray(v_ctx, dtype=np.float64)
    o = np.zeros((n_steps,) + np.shape(q_steps)[1:], dtype=np.float64)
    for i in range(n_steps):
        k = np.concatenate([k, np.asarray(k_steps[i], dtype=np.float64)[None]])
        v = np.concatenate([v, np.asarray(v_steps[i], dtype=np.float64)[None]])
        o[i] = verify_attention_request(np.asarray(q_steps[i], dtype=np.float64)[None], k, v,
                                        scale)[0]
    x = sample(probs, u)
    return o, x
