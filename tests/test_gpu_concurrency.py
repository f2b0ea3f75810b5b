"""Calls on different streams with disjoint outputs may run at the same time
(the library's threading contract): a fused preparation + attention pass,
a separate attention pass and an acceptance, each on a stream of its own
(default priority), launched back to back without waiting, then every
result against the oracle."""

import numpy as np
import pytest
import torch

import oracle
import paper_2609_29364_amd as nsd
from workload import custom_config, make_meta, make_layer, make_accept
from parity import i32, u16, check_attention, check_accept

pytestmark = pytest.mark.gpu


def _inputs(cfg, dev):
    meta = make_meta(cfg)
    lay = make_layer(cfg, meta, 0, "cpu")
    return meta, lay, {n: getattr(lay, n).to(dev).contiguous()
                       for n in ("k_pool", "v_pool", "k_stage", "v_stage", "q")}


def test_streams_run_independent_calls_concurrently(device):
    cfg_a = custom_config(seed=90, bs=40, num_q_heads=32, num_kv_heads=8, head_dim=128,
                          ctx_lo=200, ctx_hi=1500, k_lo=4, k_hi=4, n_arriving=12,
                          pool_blocks=None, vocab=4096)
    cfg_b = custom_config(seed=91, bs=33, num_q_heads=16, num_kv_heads=8, head_dim=128,
                          ctx_lo=50, ctx_hi=900, k_lo=0, k_hi=3, n_arriving=0,
                          pool_blocks=None, vocab=0)
    meta_a, lay_a, t_a = _inputs(cfg_a, device)
    meta_b, lay_b, t_b = _inputs(cfg_b, device)
    acc_in = make_accept(cfg_a, meta_a, "cpu")
    acc_dev = [x.to(device) for x in (acc_in.p_target, acc_in.q_draft, acc_in.draft_tokens,
                                       acc_in.uniforms)]
    out_a = torch.empty_like(t_a["q"])
    out_b = torch.empty_like(t_b["q"])
    ws_a = nsd.new_workspace(nsd.verify_attention_workspace_size(
        cfg_a.bs, cfg_a.num_q_heads, cfg_a.num_kv_heads, cfg_a.head_dim, meta_a.max_q,
        meta_a.max_seq_len), device)
    ws_b = nsd.new_workspace(nsd.verify_attention_workspace_size(
        cfg_b.bs, cfg_b.num_q_heads, cfg_b.num_kv_heads, cfg_b.head_dim, meta_b.max_q,
        meta_b.max_seq_len), device)
    ws_c = torch.empty(nsd.accept_workspace_size(cfg_a.bs, cfg_a.vocab), dtype=torch.uint8,
                       device=device)
    acc_len = torch.empty(cfg_a.bs, dtype=torch.int32, device=device)
    acc_tok = torch.empty(meta_a.total_q, dtype=torch.int32, device=device)
    qi_a = i32(meta_a.q_indptr, device)
    tabs_a = [i32(x, device) for x in (meta_a.block_table, meta_a.stage_table, meta_a.seq_lens)]
    tabs_b = [i32(x, device) for x in (meta_b.block_table, meta_b.seq_lens, meta_b.q_indptr)]
    torch.cuda.synchronize()

    streams = [torch.cuda.Stream(device) for _ in range(3)]
    for rep in range(3):   # several rounds of the three calls, each stream back to back
        with torch.cuda.stream(streams[0]):
            nsd.gather_verify_attention(t_a["q"], t_a["k_pool"], t_a["v_pool"], t_a["k_stage"],
                                        t_a["v_stage"], tabs_a[0], tabs_a[1], tabs_a[2], qi_a,
                                        meta_a.max_q, meta_a.max_seq_len, out=out_a,
                                        workspace=ws_a)
        with torch.cuda.stream(streams[1]):
            nsd.verify_attention(t_b["q"], t_b["k_pool"], t_b["v_pool"], tabs_b[0], tabs_b[1],
                                 tabs_b[2], meta_b.max_q, meta_b.max_seq_len, out=out_b,
                                 workspace=ws_b)
        with torch.cuda.stream(streams[2]):
            nsd.spec_accept(*acc_dev, qi_a, int(meta_a.depth.max()), accepted_len=acc_len,
                            out_tokens=acc_tok, workspace=ws_c)
    torch.cuda.synchronize()

    # the fused pass moved the arriving blocks (the pool after it equals the
    # gather's result; repeating the pass rewrites the same bytes)
    ref_k, ref_v = oracle.gather.kv_gather(u16(lay_a.k_stage)[None], u16(lay_a.v_stage)[None],
                                           u16(lay_a.k_pool)[None], u16(lay_a.v_pool)[None],
                                           meta_a.src_ids, meta_a.dst_ids)
    assert np.array_equal(u16(t_a["k_pool"]), ref_k[0])
    assert np.array_equal(u16(t_a["v_pool"]), ref_v[0])
    check_attention(meta_a, lay_a, out_a, range(cfg_a.bs))
    check_attention(meta_b, lay_b, out_b, range(cfg_b.bs))
    check_accept(acc_in.p_target.numpy(), acc_in.q_draft.numpy(), acc_in.draft_tokens.numpy(),
                 acc_in.uniforms.numpy(), meta_a.q_indptr, acc_len.cpu().numpy(),
                 acc_tok.cpu().numpy())
