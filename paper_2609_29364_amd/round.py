"""One verification round composed on one HIP stream (Algorithm 1: Run starts
once InputReady, KVReady and WorkerReady hold; on one GPU that join is stream
order): kv_gather, then verify_attention for every layer, then spec_accept."""
from . import kv_gather, verify_attention, spec_accept


def verify_round(k_pool, v_pool, k_stage, v_stage, src_ids, dst_ids, q, block_table, seq_lens,
                 q_indptr, max_q_per_seq, max_seq_len, accept=None, out=None, workspace=None,
                 scale=None):
    """Run the round; returns (out, accepted_len, out_tokens).

    Pools and staging planes are stacked over layers ([layers][blocks][...]);
    q and out are [layers][total_q][Hq][D].  ``accept`` is None (no acceptance
    step) or (p_target, q_draft, draft_tokens, uniforms, max_k).
    """
    kv_gather(k_stage, v_stage, k_pool, v_pool, src_ids, dst_ids)
    outs = []
    for layer in range(k_pool.shape[0]):
        o = None if out is None else out[layer]
        outs.append(verify_attention(q[layer], k_pool[layer], v_pool[layer], block_table,
                                     seq_lens, q_indptr, max_q_per_seq, max_seq_len, scale=scale,
                                     out=o, workspace=workspace))
    acc = tok = None
    if accept is not None:
        p, qd, x, u, max_k = accept
        acc, tok = spec_accept(p, qd, x, u, q_indptr, max_k)
    return outs if out is None else out, acc, tok
