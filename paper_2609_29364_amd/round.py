"""One verification round composed on one HIP stream (Algorithm 1: Run starts
once InputReady, KVReady and WorkerReady hold; on one GPU that join is stream
order): the KV-state preparation of the arriving requests, then per layer the
append of the window's new K/V rows (when given) and verification attention,
then spec_accept and the commit of accepted lengths.  The preparation runs
either as its own gather before the layers, or fused into each layer's
attention pass (the layer's staged tiles are read once, used and written to
the pool).

The draft stage that precedes it (Eq. 1) is composed the same way: K steps of
append, single-query attention and sampling."""
from . import (kv_gather, verify_attention, gather_verify_attention, spec_accept, kv_append,
               commit_lengths, sample, accept_workspace_size)

# Batches below this many requests prepare with the separate gather even when a
# stage table is given: there the fused pass is bound by each wave's chain of
# span steps and measured slower than gather + attention (verify_8b-shaped
# requests: 4 requests 68 against 50 us, 8 requests 78 against 54 us; from
# about 16 requests on the fused pass is as fast or faster).
FUSED_MIN_BATCH = 16


def verify_round(k_pool, v_pool, k_stage, v_stage, src_ids, dst_ids, q, block_table, seq_lens,
                 q_indptr, max_q_per_seq, max_seq_len, accept=None, out=None, workspace=None,
                 scale=None, stage_table=None, window_kv=None, committed=None,
                 append_tables=None, accept_workspace=None, prepare="auto"):
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
    requests of the fused path, whose blocks the pass then moves to the pool;
    ``append_tables`` = fused_tables(block_table, stage_table), if given).  With
    acceptance and a ``committed`` int32 [bs] tensor, the committed lengths are
    written there; ``accept_workspace`` is spec_accept's workspace.

    ``prepare``: "auto" lets a batch of fewer than FUSED_MIN_BATCH requests
    given both a stage table and the (src_ids, dst_ids) pairs take the
    separate gather (the caller states the two describe the same preparation,
    with ids in range), the faster path for such batches; "fused" keeps the
    fused pass whenever a stage table is given; "gather" always gathers first.
    """
    if prepare not in ("auto", "fused", "gather"):
        raise ValueError(f"prepare must be 'auto', 'fused' or 'gather', not {prepare!r}")
    if stage_table is not None and src_ids is not None and (
            prepare == "gather" or (prepare == "auto" and seq_lens.numel() < FUSED_MIN_BATCH)):
        stage_table = None
    if stage_table is None:
        kv_gather(k_stage, v_stage, k_pool, v_pool, src_ids, dst_ids)
    elif window_kv is not None:
        # fused preparation: an arriving request's blocks are still in the staging
        # bank, so its window rows go there and the pass moves whole blocks to the pool
        pool_table, stage_rows = append_tables or fused_tables(block_table, stage_table)
    outs = []
    for layer in range(k_pool.shape[0]):
        o = None if out is None else out[layer]
        if window_kv is not None:
            kn, vn = window_kv[layer]
            if stage_table is None:
                kv_append(k_pool[layer], v_pool[layer], kn, vn, block_table, seq_lens, q_indptr)
            else:
                kv_append(k_pool[layer], v_pool[layer], kn, vn, pool_table, seq_lens, q_indptr)
                if k_stage[layer].numel():
                    kv_append(k_stage[layer], v_stage[layer], kn, vn, stage_rows, seq_lens,
                              q_indptr)
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
        acc, tok = spec_accept(p, qd, x, u, q_indptr, max_k, workspace=accept_workspace)
        if committed is not None:
            commit_lengths(seq_lens, q_indptr, acc, out=committed)
    return outs if out is None else out, acc, tok


def fused_tables(block_table, stage_table):
    """Append tables for the fused preparation, (pool_table, stage_rows): arriving
    requests (staging id in entry 0) write into their staged blocks, resident
    ones into the pool.  Batch metadata: build once per batch and pass as
    ``append_tables``."""
    import torch
    arriving = stage_table[:, :1] >= 0
    pool_table = torch.where(arriving, torch.full_like(block_table, -1), block_table)
    stage_rows = torch.where(arriving, stage_table, torch.full_like(stage_table, -1))
    return pool_table, stage_rows


def draft_stage(k_pool, v_pool, q, k_new, v_new, probs, uniforms, block_table, lens, q_indptr,
                max_seq_len, k_stage=None, v_stage=None, src_ids=None, dst_ids=None,
                stage_table=None, tokens=None, out=None, workspace=None, scale=None,
                append_tables=None, sample_workspace=None):
    """K draft steps of one layer on one stream; returns (out, tokens).

    Step i processes one token per request (the anchor, then proposal i-1): it
    appends that token's K/V rows k_new[i], v_new[i] ([bs][Hkv][D]) at
    position lens[i][r] - 1, attends with q[i] ([bs][Hq][D]) over positions
    0 .. lens[i][r] - 1 into out[i], and draws proposal i from the draft rows
    probs[:, i] with uniforms[i] into tokens[:, i].

    probs: fp32 [bs][K][V] and tokens: int32 [bs][K] are request-major, the
    q_draft / draft_tokens layout spec_accept takes; uniforms: fp32 [K][bs];
    lens: int32 [K][bs] (step i: the step-0 lengths plus i); q_indptr: int32
    [bs+1] = 0, 1, .., bs.  Arriving requests are prepared before step 0, by
    the (src_ids, dst_ids) gather from the staging planes, or with
    ``stage_table`` fused into step 0's attention pass (their step-0 rows are
    appended into the staged blocks, which the pass moves to the pool;
    ``append_tables`` = fused_tables(block_table, stage_table), if given).
    ``sample_workspace``: accept_workspace_size(bs, V) bytes, one for all steps."""
    import torch
    n_steps, bs = lens.shape
    if sample_workspace is None:
        sample_workspace = torch.empty(accept_workspace_size(bs, probs.shape[-1]),
                                       dtype=torch.uint8, device=probs.device)
    if tokens is None:
        tokens = torch.empty((bs, n_steps), dtype=torch.int32, device=probs.device)
    if out is None:
        out = torch.empty_like(q)
    if stage_table is None:
        if src_ids is not None and src_ids.numel():
            kv_gather(k_stage, v_stage, k_pool, v_pool, src_ids, dst_ids)
    else:
        pool_table, stage_rows = append_tables or fused_tables(block_table, stage_table)
    for i in range(n_steps):
        if stage_table is not None and i == 0:
            kv_append(k_pool, v_pool, k_new[i], v_new[i], pool_table, lens[i], q_indptr)
            if k_stage.numel():      # no staged blocks when nothing arrives
                kv_append(k_stage, v_stage, k_new[i], v_new[i], stage_rows, lens[i], q_indptr)
            gather_verify_attention(q[i], k_pool, v_pool, k_stage, v_stage, block_table,
                                    stage_table, lens[i], q_indptr, 1, max_seq_len, scale=scale,
                                    out=out[i], workspace=workspace)
        else:
            kv_append(k_pool, v_pool, k_new[i], v_new[i], block_table, lens[i], q_indptr)
            verify_attention(q[i], k_pool, v_pool, block_table, lens[i], q_indptr, 1,
                             max_seq_len, scale=scale, out=out[i], workspace=workspace)
        sample(probs[:, i], uniforms[i], out=tokens[:, i], workspace=sample_workspace)
    return out, tokens
