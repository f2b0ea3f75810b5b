"""A verification round captured in a HIP graph: the library allocates nothing,
records no memory sets and waits for nothing inside a call, so the fused
preparation + attention pass and the acceptance can be captured once and
replayed.  Each replay (with eager library work and synchronisations between
the replays) must reproduce the eager results exactly, and those match the
oracle."""

import numpy as np
import pytest
import torch

import oracle
import paper_2609_29364_amd as nsd
from workload import custom_config, make_meta, make_layer, make_accept
from parity import i32, u16, check_attention, check_accept

pytestmark = pytest.mark.gpu


def test_round_replays_from_a_graph(device):
    cfg = custom_config(seed=95, bs=48, num_q_heads=32, num_kv_heads=8, head_dim=128,
                        ctx_lo=100, ctx_hi=1200, k_lo=2, k_hi=4, n_arriving=16, pool_blocks=None,
                        vocab=8192)
    meta = make_meta(cfg)
    lay = make_layer(cfg, meta, 0, "cpu")
    t = {n: getattr(lay, n).to(device).contiguous()
         for n in ("k_pool", "v_pool", "k_stage", "v_stage", "q")}
    acc_in = make_accept(cfg, meta, "cpu")
    p, qd, xt, u = (x.to(device) for x in (acc_in.p_target, acc_in.q_draft, acc_in.draft_tokens,
                                            acc_in.uniforms))
    bt, st, sl, qi = (i32(x, device) for x in (meta.block_table, meta.stage_table, meta.seq_lens,
                                               meta.q_indptr))
    max_k = int(meta.depth.max())
    ws = nsd.new_workspace(nsd.verify_attention_workspace_size(
        cfg.bs, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, meta.max_q, meta.max_seq_len),
        device)
    aws = torch.empty(nsd.accept_workspace_size(cfg.bs, cfg.vocab), dtype=torch.uint8,
                      device=device)
    out = torch.empty_like(t["q"])
    acc_len = torch.empty(cfg.bs, dtype=torch.int32, device=device)
    acc_tok = torch.empty(meta.total_q, dtype=torch.int32, device=device)

    def round_():
        nsd.gather_verify_attention(t["q"], t["k_pool"], t["v_pool"], t["k_stage"], t["v_stage"],
                                    bt, st, sl, qi, meta.max_q, meta.max_seq_len, out=out,
                                    workspace=ws)
        nsd.spec_accept(p, qd, xt, u, qi, max_k, accepted_len=acc_len, out_tokens=acc_tok,
                        workspace=aws)

    # eager reference, checked against the oracle
    round_()
    torch.cuda.synchronize()
    ref_out, ref_len, ref_tok = out.clone(), acc_len.clone(), acc_tok.clone()
    check_attention(meta, lay, ref_out, range(cfg.bs))
    check_accept(acc_in.p_target.numpy(), acc_in.q_draft.numpy(), acc_in.draft_tokens.numpy(),
                 acc_in.uniforms.numpy(), meta.q_indptr, ref_len.cpu().numpy(),
                 ref_tok.cpu().numpy())
    ref_k, ref_v = oracle.gather.kv_gather(u16(lay.k_stage)[None], u16(lay.v_stage)[None],
                                           u16(lay.k_pool)[None], u16(lay.v_pool)[None],
                                           meta.src_ids, meta.dst_ids)

    side = torch.cuda.Stream(device)
    side.wait_stream(torch.cuda.current_stream(device))
    with torch.cuda.stream(side):   # one warm call on the capture stream
        round_()
    torch.cuda.current_stream(device).wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        round_()
    torch.cuda.synchronize()

    other_q = torch.randn_like(t["q"], dtype=torch.float32).to(torch.bfloat16)
    for rep in range(3):
        out.zero_()
        acc_len.fill_(-7)
        acc_tok.fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref_out), f"replay {rep}: attention output differs"
        assert torch.equal(acc_len, ref_len) and torch.equal(acc_tok, ref_tok), \
            f"replay {rep}: acceptance differs"
        assert np.array_equal(u16(t["k_pool"]), ref_k[0])
        assert np.array_equal(u16(t["v_pool"]), ref_v[0])
        # eager library work on other buffers between the replays
        nsd.verify_attention(other_q, t["k_pool"], t["v_pool"], bt, sl, qi, meta.max_q,
                             meta.max_seq_len)
        torch.cuda.synchronize()
