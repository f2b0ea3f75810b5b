"""One verification round composed on one HIP stream (Algorithm 1: Run starts
once InputReady, KVReady and WorkerReady hold; on one GPU that join is stream
order): the KV-state preparation of the arriving requests, verification
attention for every layer, then spec_accept.  The preparation runs either as
its own gather before the layers, or fused into each layer's attention pass
(the layer's staged tiles are read once, used and written to the pool)."""
from . import kv_gather, verify_attention, gather_verify_attention, spec_accept


def verify_round(k_pool, v_pool, k_stage, v_stage, src_ids, dst_ids, q, block_table, seq_lens,
                 q_indptr, max_q_per_seq, max_seq_len, accept=None, out=None, workspace=None,
                 scale=None, stage_table=None):
    """Run the round; returns (out, accepted_len, out_tokens).

    Pools and staging planes are stacked over layers ([layers][blocks][...]);
    q and out are [layers][total_q][Hq][D].  With ``stage_table`` ([bs][max
    blocks] staging ids of arriving requests, -1 in entry 0 for resident ones)
    the preparation is fused into the attention passes and src_ids/dst_ids are
    not used; otherwise the (src_ids, dst_ids) pairs are gathered first.
    ``accept`` is None (no acceptance step) or (p_target, q_draft,
    draft_tokens, uniforms, max_k).
    """
    if stage_table is None:
        kv_gather(k_stage, v_stage, k_pool, v_pool, src_ids, dst_ids)
    outs = []
    for layer in range(k_pool.shape[0]):
        o = None if out is None else out[layer]
        if stage_table is None:
            outs.append(verify_attention(q[layer], k_pool[layer], v_pool[layer], block_table,
                                         seq_lens, q_indptr, max_q_per_seq, max_seq_len,
                                         scale=scale, out=o, workspace=workspace))
        else:
            outs.append(gather_verify_attention(q[layer], k_pool[layer], v_pool[layer],
                                                k_stage[layer], v_stage[layer], block_table,
                                                stage_table, seq_lens, q_indptr, max_q_per_seq,
                                                max_seq_len, scale=scale, out=o,
                                                workspace=workspace))
    acc = tok = None
    if accept is not None:
        p, qd, x, u, max_k = accept
        acc, tok = spec_accept(p, qd, x, u, q_indptr, max_k)
    return outs if out is None else out, acc, tok
