"""Closing the round on the GPU: the window append, the committed lengths and
the suffix writeback into the pinned host arena, each against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_29364_amd as nsd
from workload import CONFIGS, custom_config, make_meta, make_layer, make_accept, make_hostkv
from parity import i32, u16

pytestmark = pytest.mark.gpu


def _rows(meta, cfg, seed):
    g = torch.Generator(device="cpu").manual_seed(seed)
    shape = (meta.total_q, cfg.num_kv_heads, cfg.head_dim)
    return (torch.randn(shape, generator=g).to(torch.bfloat16),
            torch.randn(shape, generator=g).to(torch.bfloat16))


@pytest.mark.parametrize("cfg", [CONFIGS["tiny"],
                                 custom_config(seed=41, bs=7, k_lo=1, k_hi=6, head_dim=128,
                                               num_q_heads=8, num_kv_heads=4, pool_blocks=None)],
                         ids=["tiny", "ragged_d128"])
def test_append_matches_oracle(device, cfg):
    meta = make_meta(cfg)
    lay = make_layer(cfg, meta, 0, "cpu")
    kn, vn = _rows(meta, cfg, 3)
    kp, vp = lay.k_pool.to(device), lay.v_pool.to(device)
    nsd.kv_append(kp, vp, kn.to(device), vn.to(device), i32(meta.block_table, device),
                  i32(meta.seq_lens, device), i32(meta.q_indptr, device))
    torch.cuda.synchronize()
    rk, rv = oracle.commit.kv_append(u16(lay.k_pool), u16(lay.v_pool), u16(kn), u16(vn),
                                     meta.block_table, meta.seq_lens, meta.q_indptr)
    assert np.array_equal(u16(kp), rk) and np.array_equal(u16(vp), rv)


@pytest.mark.parametrize("head_dim", [64, 128])
def test_append_edges_match_oracle(device, head_dim):
    """Windows that cross a block boundary or span three blocks, block ids out
    of range inside a window, positions past the table and contexts shorter
    than the window.  The expected pools are the oracle's append applied token
    by token to the tokens that have a position in the table and a valid
    block id (the others are skipped); every other slot, including the rest
    of each 32-byte sector the kernel rewrites, must keep its bytes."""
    hkv, mbs, nb = 2, 4, 40
    rng = np.random.default_rng(7)
    # (seq_len, n_q, table row): block ids, -1 = invalid
    cases = [(19, 5, [3, 4, -1, -1]),          # slots 14, 15 | 0, 1, 2 of the next block
             (48, 40, [5, 6, 7, -1]),          # three blocks
             (16, 1, [8, -1, -1, -1]),         # the last slot of a block
             (33, 6, [9, -1, 10, -1]),         # the middle block invalid
             (30, 4, [11, nb + 3, -1, -1]),    # an id past the pool
             (70, 8, [12, 13, 14, 15]),        # positions past the table (64 slots)
             (3, 5, [16, -1, -1, -1]),         # context shorter than the window
             (1, 1, [17, -1, -1, -1])]
    sl = np.array([c[0] for c in cases], dtype=np.int32)
    nqs = np.array([c[1] for c in cases])
    qi = np.concatenate([[0], np.cumsum(nqs)]).astype(np.int32)
    bt = np.array([c[2] for c in cases], dtype=np.int32)
    tq = int(qi[-1])
    kp0 = torch.from_numpy(rng.integers(-30000, 30000, size=(nb, hkv, head_dim // 8, 16, 8),
                                        dtype=np.int16)).view(torch.bfloat16)
    vp0 = torch.from_numpy(rng.integers(-30000, 30000, size=(nb, hkv, head_dim, 16),
                                        dtype=np.int16)).view(torch.bfloat16)
    kn = torch.from_numpy(rng.integers(-30000, 30000, size=(tq, hkv, head_dim),
                                       dtype=np.int16)).view(torch.bfloat16)
    vn = torch.from_numpy(rng.integers(-30000, 30000, size=(tq, hkv, head_dim),
                                       dtype=np.int16)).view(torch.bfloat16)
    kp, vp = kp0.to(device), vp0.to(device)
    nsd.kv_append(kp, vp, kn.to(device), vn.to(device), i32(bt, device), i32(sl, device),
                  i32(qi, device))
    torch.cuda.synchronize()
    rk, rv = u16(kp0), u16(vp0)
    for r, (L, nq, row) in enumerate(cases):
        for j in range(nq):
            t = L - nq + j
            if t < 0 or t >= 16 * mbs or not 0 <= bt[r, t // 16] < nb:
                continue
            one = np.array([0, 1], dtype=np.int32)
            rk, rv = oracle.commit.kv_append(rk, rv, u16(kn)[qi[r] + j:qi[r] + j + 1],
                                             u16(vn)[qi[r] + j:qi[r] + j + 1], bt[r:r + 1],
                                             np.array([t + 1]), one)
    assert np.array_equal(u16(kp), rk) and np.array_equal(u16(vp), rv)


def test_append_and_commit_bindings_refuse_mismatched_shapes(device):
    """The binding checks every shape the kernels index with before launching:
    pools whose head_dim differs from the rows', a table of another batch
    size, and a commit output of the wrong length are refused, and nothing
    is written."""
    bf = torch.bfloat16
    kp = torch.zeros((8, 2, 64 // 8, 16, 8), dtype=bf, device=device)
    vp = torch.zeros((8, 2, 64, 16), dtype=bf, device=device)
    rows = torch.ones((3, 2, 128), dtype=bf, device=device)   # head_dim 128 against 64
    bt = torch.zeros((2, 4), dtype=torch.int32, device=device)
    sl = torch.tensor([3, 1], dtype=torch.int32, device=device)
    qi = torch.tensor([0, 2, 3], dtype=torch.int32, device=device)
    with pytest.raises(ValueError):
        nsd.kv_append(kp, vp, rows, rows, bt, sl, qi)
    rows64 = torch.ones((3, 2, 64), dtype=bf, device=device)
    with pytest.raises(ValueError):
        nsd.kv_append(kp, vp, rows64, rows64, bt[:1], sl, qi)
    with pytest.raises(ValueError):
        nsd.commit_lengths(sl, qi, sl, out=torch.empty(5, dtype=torch.int32, device=device))
    p = torch.full((3, 8), 0.125, dtype=torch.float32, device=device)
    u = torch.full((3,), 0.5, dtype=torch.float32, device=device)
    with pytest.raises(ValueError):   # accepted_len shorter than the batch
        nsd.spec_accept(p, p[:1], qi[:1], u, qi, 1,
                        accepted_len=torch.empty(1, dtype=torch.int32, device=device))
    torch.cuda.synchronize()
    assert not kp.any() and not vp.any()


def test_commit_lengths_matches_oracle(device):
    cfg = custom_config(seed=42, bs=50, k_lo=0, k_hi=8, pool_blocks=None, ctx_lo=20, ctx_hi=90)
    meta = make_meta(cfg)
    g = np.random.default_rng(2)
    acc = g.integers(-2, 11, meta.bs).astype(np.int32)      # out-of-range values are clamped
    out = nsd.commit_lengths(i32(meta.seq_lens, device), i32(meta.q_indptr, device),
                             i32(acc, device))
    torch.cuda.synchronize()
    k = np.diff(meta.q_indptr) - 1
    ref = oracle.commit.commit_lengths(meta.seq_lens, meta.q_indptr, np.clip(acc, 0, k))
    assert np.array_equal(out.cpu().numpy(), ref)


def test_round_close_writes_back_the_suffix(device):
    # round -> acceptance -> commit -> suffix writeback into the host arena, on the
    # GPU; every expected value comes from the oracle on the generator's inputs:
    # accepted lengths (oracle.accept), committed lengths (oracle.commit), the
    # pool after the preparation (oracle.gather) and the suffix blocks
    # (oracle.commit.writeback_pairs) copied into the arena as it was before
    from paper_2609_29364_amd.hostkv import writeback_pairs
    cfg = custom_config(seed=43, bs=6, k_lo=2, k_hi=5, n_arriving=2, pool_blocks=None)
    meta = make_meta(cfg)
    lay = make_layer(cfg, meta, 0, "cpu")
    host = make_hostkv(cfg, meta, lay)
    arena0 = (u16(host.k).copy(), u16(host.v).copy())
    host_len = meta.seq_lens - np.diff(meta.q_indptr)      # the window is new this round
    acc_cpu = make_accept(cfg, meta, "cpu")
    # GPU: the worker's order of calls; the writeback plan follows the GPU's own lengths
    kp, vp = lay.k_pool.to(device), lay.v_pool.to(device)
    nsd.kv_gather(lay.k_stage.to(device), lay.v_stage.to(device), kp, vp,
                  i32(meta.src_ids, device), i32(meta.dst_ids, device))
    acc, _ = nsd.spec_accept(acc_cpu.p_target.to(device), acc_cpu.q_draft.to(device),
                             acc_cpu.draft_tokens.to(device), acc_cpu.uniforms.to(device),
                             i32(meta.q_indptr, device), int(meta.depth.max()))
    new_len = nsd.commit_lengths(i32(meta.seq_lens, device), i32(meta.q_indptr, device), acc)
    torch.cuda.synchronize()
    src, dst = writeback_pairs(meta.block_table, host.extent, host_len, new_len.cpu().numpy())
    nsd.kv_writeback(kp, vp, host.k, host.v, i32(src, device), i32(dst, device))
    torch.cuda.synchronize()
    # oracle, from the generator's inputs only
    n_ref, _ = oracle.accept.spec_accept(acc_cpu.p_target.numpy(), acc_cpu.q_draft.numpy(),
                                         acc_cpu.draft_tokens.numpy(), acc_cpu.uniforms.numpy(),
                                         meta.q_indptr)
    len_ref = oracle.commit.commit_lengths(meta.seq_lens, meta.q_indptr, n_ref)
    pool_k, pool_v = oracle.gather.kv_gather(u16(lay.k_stage)[None], u16(lay.v_stage)[None],
                                             u16(lay.k_pool)[None], u16(lay.v_pool)[None],
                                             meta.src_ids, meta.dst_ids)
    s_ref, d_ref = oracle.commit.writeback_pairs(meta.block_table, host.extent, host_len,
                                                 len_ref)
    ref_k, ref_v = arena0[0].copy(), arena0[1].copy()
    ref_k[d_ref], ref_v[d_ref] = pool_k[0][s_ref], pool_v[0][s_ref]
    assert np.array_equal(acc.cpu().numpy(), n_ref)
    assert np.array_equal(new_len.cpu().numpy(), len_ref)
    assert np.array_equal(u16(host.k), ref_k) and np.array_equal(u16(host.v), ref_v)
    assert len(s_ref) > 0
    # the arena now holds every request's committed tokens (the generator's logical cache)
    from workload.layout import logical_kv_from_blocks
    from workload.synth import logical_kv
    for r in range(meta.bs):
        n = -(-int(len_ref[r]) // 16)
        e = int(host.extent[r])
        k, v = logical_kv_from_blocks(host.k[e:e + n], host.v[e:e + n], int(len_ref[r]))
        k0, v0 = logical_kv(meta, lay, r)
        assert torch.equal(k.view(torch.int16), k0[:int(len_ref[r])].view(torch.int16))
        assert torch.equal(v.view(torch.int16), v0[:int(len_ref[r])].view(torch.int16))


def test_host_alias_refuses_pageable(device):
    with pytest.raises(ValueError):
        nsd.host_alias(torch.zeros(16))
    t = torch.zeros(64, pin_memory=True)
    assert nsd.host_alias(t) is not None


@pytest.mark.parametrize("fused", [False, True])
def test_round_with_window_append(device, fused):
    # the pools start with the window slots poisoned; the round appends the window rows
    # (the logical K/V at the window positions) before attention, which must then match
    # the oracle on the logical cache; the committed lengths follow acceptance
    from paper_2609_29364_amd.round import verify_round
    from workload.synth import logical_kv
    cfg = custom_config(seed=44, bs=5, k_lo=1, k_hi=5, n_arriving=2, pool_blocks=None)
    meta = make_meta(cfg)
    lay = make_layer(cfg, meta, 0, "cpu")
    kn = torch.empty((meta.total_q, cfg.num_kv_heads, cfg.head_dim), dtype=torch.bfloat16)
    vn = torch.empty_like(kn)
    kp, vp = lay.k_pool.clone(), lay.v_pool.clone()
    ks, vs = lay.k_stage.clone(), lay.v_stage.clone()
    for r in range(meta.bs):
        a, b = int(meta.q_indptr[r]), int(meta.q_indptr[r + 1])
        L = int(meta.seq_lens[r])
        k, v = logical_kv(meta, lay, r)
        kn[a:b], vn[a:b] = k[L - (b - a):], v[L - (b - a):]
        # poison the window slots wherever this request's blocks live now
        table = meta.stage_table if meta.arriving[r] else meta.block_table
        pk, pv = (ks, vs) if meta.arriving[r] else (kp, vp)
        for t in range(L - (b - a), L):
            blk = int(table[r, t // 16])
            pk[blk, :, :, t % 16, :] = float("nan")
            pv[blk, :, :, t % 16] = float("nan")
    acc_in = make_accept(cfg, meta, device)
    committed = torch.empty(meta.bs, dtype=torch.int32, device=device)
    st = i32(meta.stage_table, device) if fused else None
    outs, acc, _ = verify_round(
        kp.to(device)[None].contiguous(), vp.to(device)[None].contiguous(),
        ks.to(device)[None].contiguous(), vs.to(device)[None].contiguous(),
        i32(meta.src_ids, device), i32(meta.dst_ids, device), lay.q.to(device)[None].contiguous(),
        i32(meta.block_table, device), i32(meta.seq_lens, device), i32(meta.q_indptr, device),
        meta.max_q, meta.max_seq_len,
        accept=(acc_in.p_target, acc_in.q_draft, acc_in.draft_tokens, acc_in.uniforms,
                int(meta.depth.max())),
        stage_table=st, window_kv=[(kn.to(device), vn.to(device))], committed=committed,
        prepare="fused" if fused else "gather")
    torch.cuda.synchronize()
    from parity import check_attention
    check_attention(meta, lay, outs[0], range(meta.bs))
    # the generator's inputs (drawn on the device), copied to the host
    n_ref, _ = oracle.accept.spec_accept(acc_in.p_target.cpu().numpy(),
                                         acc_in.q_draft.cpu().numpy(),
                                         acc_in.draft_tokens.cpu().numpy(),
                                         acc_in.uniforms.cpu().numpy(), meta.q_indptr)
    ref = oracle.commit.commit_lengths(meta.seq_lens, meta.q_indptr, n_ref)
    assert np.array_equal(acc.cpu().numpy(), n_ref)
    assert np.array_equal(committed.cpu().numpy(), ref)
