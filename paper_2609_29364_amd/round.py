"""One verification round composed on one HIP stream (Algorithm 1: Run starts
once InputReady, KVReady and WorkerReady hold; on one GPU that join is stream
order): the KV-state preparation of the arriving requests, then per layer the
append of the window's new K/V rows (when given) and verification attention,
then spec_accept and the commit of accepted lengths.  The preparation runs
either as its own gather before the layers, or fused into each layer's
attention pass (the layer's staged tiles are read once, used and written to
the pool)."""
from . import (kv_gather, verify_attention, gather_verify_attention, spec_accept, kv_append,
               commit_lengths)


def verify_round(k_pool, v_pool, k_stage, v_stage, src_ids, dst_ids, q, block_table, seq_lens,
                 q_indptr, max_q_per_seq, max_seq_len, accept=None, out=None, workspace=None,
                 scale=None, stage_table=None, window_kv=None, committed=None):
    """Run the round; returns (out, accepted_len, out_tokens).

    Pools and staging planes are stacked over layers ([layers][blocks][...]);
    q and out are [layers][total_q][Hq][D].  With ``stage_table`` ([bs][max
    blocks] staging ids of arriving requests, -1 in entry 0 for resident ones)
    the preparation is fused into the attention passes and src_ids/dst_ids are
    not used; otherwise the (src_ids, dst_ids) pairs are gathered first.
    ``accept`` is None (no acceptance step) or (p_target, q_draft,
    draft_tokens, uniforms, max_k).  ``window_kv`` is None (the pools already
    hold the window's K/V) or per-layer (k_new, v_new) rows [total_q][Hkv][D]
    appended before that layer's attention (into the staging bank for arriving
    requests of the fused path, whose blocks the pass then moves to the pool).  With acceptance and a
    ``committed`` int32 [bs] tensor, the committed lengths are written there.
    """
    if stage_table is None:
        kv_gather(k_stage, v_stage, k_pool, v_pool, src_ids, dst_ids)
    elif window_kv is not None:
        # fused preparation: an arriving request's blocks are still in the staging
        # bank, so its window rows go there and the pass moves whole blocks to the pool
        import torch
        arriving = stage_table[:, :1] >= 0
        pool_table = torch.where(arriving, torch.full_like(block_table, -1), block_table)
        stage_rows = torch.where(arriving, stage_table, torch.full_like(stage_table, -1))
    outs = []
    for layer in range(k_pool.shape[0]):
        o = None if out is None else out[layer]
        if window_kv is not None:
            kn, vn = window_kv[layer]
            if stage_table is None:
                kv_append(k_pool[layer], v_pool[layer], kn, vn, block_table, seq_lens, q_indptr)
            else:
                kv_append(k_pool[layer], v_pool[layer], kn, vn, pool_table, seq_lens, q_indptr)
                kv_append(k_stage[layer], v_stage[layer], kn, vn, stage_rows, seq_lens, q_indptr)
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
        if committed is not None:
            commit_lengths(seq_lens, q_indptr, acc, out=committed)
    return outs if out is None else out, acc, tok
