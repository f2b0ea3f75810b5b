"""Oracle for grouped-query verification attention over a request's KV cache.

In a verification round the target model scores a request's anchor token and
its K proposal tokens in one forward pass (Section 1; Appendix G.2 counts this
work as anchor-plus-proposal tokens; Appendix H: requests start post-prefill
with an anchor token and depth d proposals).  The KV cache already holds the
states of all L_r tokens, window included (Section 3: the cache is
append-dominant).  Query j of the n_q = K_r + 1 window sits at position
L_r - n_q + j and sees keys 0 .. L_r - n_q + j (causal within the window).
Query heads share KV heads in contiguous groups: head h reads KV head
h // (Hq / Hkv).

Plain definition, in fp64:  o = softmax(scale * K q) V  per (head, query).
"""
import numpy as np


def verify_attention_request(q, k, v, scale):
    """q: [n_q][Hq][D]; k, v: [L][Hkv][D] (float64) -> o [n_q][Hq][D] float64."""
    n_q, hq, _ = q.shape
    length, hkv, _ = k.shape
    group = hq // hkv
    o = np.zeros(q.shape, dtype=np.float64)
    for h in range(hq):
        g = h // group
        for j in range(n_q):
            pos = length - n_q + j
            scores = scale * (k[:pos + 1, g, :] @ q[j, h, :])
            w = np.exp(scores - scores.max())
            o[j, h, :] = (w / w.sum()) @ v[:pos + 1, g, :]
    return o
