"""KV-state preparation from a pinned host arena (HostKV) through the DMA copy
plan into double-buffered device banks, then the fused gather + attention pass:
the worker pool must hold exactly what the oracle's gather gives, bank reuse must
never let a background copy overwrite a bank a round is still reading."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_29364_amd as nsd
from paper_2609_29364_amd.hostkv import DoubleBank, h2d_plan
from workload import CONFIGS, custom_config, make_meta, make_layer, make_hostkv
from parity import i32, u16, check_attention

pytestmark = pytest.mark.gpu


def _setup(cfg, device):
    meta = make_meta(cfg)
    lay = make_layer(cfg, meta, 0, "cpu")
    host = make_hostkv(cfg, meta, lay)
    bb = lay.k_stage[0].numel() * 2
    plan = h2d_plan(host.extent, meta.stage_table, meta.arriving, meta.seq_lens, bb)
    return meta, lay, host, plan


def _fused(meta, lay, kp, vp, ks, vs, device):
    return nsd.gather_verify_attention(lay.q.to(device), kp, vp, ks, vs,
                                       i32(meta.block_table, device), i32(meta.stage_table, device),
                                       i32(meta.seq_lens, device), i32(meta.q_indptr, device),
                                       meta.max_q, meta.max_seq_len)


def _expect_pool(meta, lay):
    return oracle.gather.kv_gather(u16(lay.k_stage)[None], u16(lay.v_stage)[None],
                                   u16(lay.k_pool)[None], u16(lay.v_pool)[None],
                                   meta.src_ids, meta.dst_ids)


@pytest.mark.parametrize("name", ["tiny", "shuffled"])
@pytest.mark.parametrize("chunk", [nsd.DEFAULT_CHUNK, 4096])
def test_h2d_then_fused_round(device, name, chunk):
    cfg = CONFIGS["tiny"] if name == "tiny" else custom_config(staging_order="shuffled", seed=10)
    meta, lay, host, plan = _setup(cfg, device)
    bank = DoubleBank(lay.k_stage.shape, lay.v_stage.shape, device)
    bank.k[0].fill_(float("nan"))
    bank.v[0].fill_(float("nan"))
    bank.prepare(0, host.k, host.v, plan, plan, chunk_bytes=chunk)
    torch.cuda.current_stream(device).wait_event(bank.ready(0))
    kp, vp = lay.k_pool.to(device), lay.v_pool.to(device)
    ks, vs = bank.bank(0)
    out = _fused(meta, lay, kp, vp, ks, vs, device)
    torch.cuda.synchronize()
    # the bank holds the staged blocks, byte for byte
    ids = torch.as_tensor(meta.src_ids, dtype=torch.long)
    assert np.array_equal(u16(ks.cpu()[ids]), u16(lay.k_stage[ids]))
    assert np.array_equal(u16(vs.cpu()[ids]), u16(lay.v_stage[ids]))
    ref_k, ref_v = _expect_pool(meta, lay)
    assert np.array_equal(u16(kp.cpu()), ref_k[0]) and np.array_equal(u16(vp.cpu()), ref_v[0])
    check_attention(meta, lay, out, range(cfg.bs))


def test_d2h_plan_roundtrip(device):
    # writeback direction: scattered 4 KiB pieces of a device buffer into a pinned arena,
    # with chunks smaller than the merged runs
    g = torch.Generator(device="cpu").manual_seed(5)
    src = torch.randint(0, 255, (64 * 4096,), dtype=torch.uint8, generator=g)
    dev = src.to(device)
    host = torch.zeros(80 * 4096, dtype=torch.uint8, pin_memory=True)
    perm = np.random.default_rng(3).permutation(80)[:64]
    plan = np.stack([np.arange(64) * 4096, perm * 4096, np.full(64, 4096)], axis=1)
    plan[10:20, 1] = (np.arange(10) + 70) * 4096     # a run of ten contiguous pieces
    nsd.copy_plan(dev, host, plan, chunk_bytes=12288)
    torch.cuda.synchronize()
    ref = np.zeros(80 * 4096, dtype=np.uint8)
    for s, d, n in plan:
        ref[d:d + n] = src.numpy()[s:s + n]
    assert np.array_equal(host.numpy(), ref)


def test_copy_plan_rejects_pageable_memory(device):
    host = torch.zeros(4096, dtype=torch.uint8)           # not pinned
    dev = torch.zeros(4096, dtype=torch.uint8, device=device)
    with pytest.raises(ValueError):
        nsd.copy_plan(host, dev, [[0, 0, 4096]])
    st = nsd.lib().nsd_copy_plan(host.data_ptr(), 4096, dev.data_ptr(), 4096,
                                 np.array([0, 0, 4096], dtype=np.int64).ctypes.data, 1, 1 << 20,
                                 nsd.COPY_H2D, None)
    assert st == 3 and b"pinned" in nsd.lib().nsd_last_error()


def test_double_banked_rounds(device):
    # four rounds alternating two banks, each round with KV of its own (different layers),
    # so a bank refilled before its round had read it would show up as a wrong pool
    cfg = custom_config(seed=13, bs=6, n_arriving=3, pool_blocks=None)
    meta = make_meta(cfg)
    lays = [make_layer(cfg, meta, i, "cpu") for i in range(4)]
    hosts = [make_hostkv(cfg, meta, lay) for lay in lays]
    bb = lays[0].k_stage[0].numel() * 2
    plan = h2d_plan(hosts[0].extent, meta.stage_table, meta.arriving, meta.seq_lens, bb)
    bank = DoubleBank(lays[0].k_stage.shape, lays[0].v_stage.shape, device)
    stream = torch.cuda.current_stream(device)
    pools, outs = [], []
    bank.prepare(0, hosts[0].k, hosts[0].v, plan, plan)
    for i in range(4):
        if i + 1 < 4:
            bank.prepare(i + 1, hosts[i + 1].k, hosts[i + 1].v, plan, plan)
        stream.wait_event(bank.ready(i))
        kp, vp = lays[i].k_pool.to(device), lays[i].v_pool.to(device)
        ks, vs = bank.bank(i)
        outs.append(_fused(meta, lays[i], kp, vp, ks, vs, device))
        bank.done(i, stream)
        pools.append((kp, vp))
    torch.cuda.synchronize()
    for i, ((kp, vp), out) in enumerate(zip(pools, outs)):
        ref_k, ref_v = _expect_pool(meta, lays[i])
        assert np.array_equal(u16(kp.cpu()), ref_k[0]) and np.array_equal(u16(vp.cpu()), ref_v[0])
        check_attention(meta, lays[i], out, range(cfg.bs))


@pytest.mark.parametrize("window", [None, 64 << 10], ids=["all_queued", "window_64k"])
def test_banked_rounds_with_export(device, window):
    # the whole bank lifecycle (Eq. E.2) over four rounds on two banks: round
    # i+1's H2D (bounded to 64 KiB groups of 4 KiB chunks, or queued at once)
    # while round i computes; after round i, acceptance and the committed
    # lengths, then its export -- the committed suffix written back into round
    # i's arena on the D2H stream -- before the bank is Free again.  Every
    # round's pool, attention, committed lengths and arena against the oracle
    # (expected values from the generator's inputs only).
    from paper_2609_29364_amd.hostkv import writeback_pairs
    from workload import make_accept
    cfg = custom_config(seed=14, bs=6, k_lo=2, k_hi=5, n_arriving=3, pool_blocks=None)
    meta = make_meta(cfg)
    lays = [make_layer(cfg, meta, i, "cpu") for i in range(4)]
    hosts = [make_hostkv(cfg, meta, lay) for lay in lays]
    host_len = meta.seq_lens - np.diff(meta.q_indptr)
    # the arena holds the tokens persisted before the round; a resident request's
    # blocks from host_len on are stale there (a marker value), so only the
    # export can make them right (arriving requests' blocks are restored from
    # the arena first, so theirs stay whole)
    for h in hosts:
        for r in np.nonzero(~meta.arriving)[0]:
            j0, j1 = int(host_len[r]) // 16, meta.nblk(r)
            e = int(h.extent[r])
            h.k[e + j0:e + j1] = 7.0
            h.v[e + j0:e + j1] = 7.0
    arenas0 = [(u16(h.k).copy(), u16(h.v).copy()) for h in hosts]
    a_cpu = make_accept(cfg, meta, "cpu")
    a_dev = [t.to(device) for t in (a_cpu.p_target, a_cpu.q_draft, a_cpu.draft_tokens,
                                    a_cpu.uniforms)]
    bb = lays[0].k_stage[0].numel() * 2
    plan = h2d_plan(hosts[0].extent, meta.stage_table, meta.arriving, meta.seq_lens, bb)
    chunk = 4096 if window else nsd.DEFAULT_CHUNK
    bank = DoubleBank(lays[0].k_stage.shape, lays[0].v_stage.shape, device)
    stream = torch.cuda.current_stream(device)
    qi = i32(meta.q_indptr, device)
    pools, outs, lens = [], [], []
    bank.prepare(0, hosts[0].k, hosts[0].v, plan, plan, chunk_bytes=chunk, window_bytes=window)
    for i in range(4):
        if i + 1 < 4:
            bank.prepare(i + 1, hosts[i + 1].k, hosts[i + 1].v, plan, plan, chunk_bytes=chunk,
                         window_bytes=window)
        bank.computing(i, stream)
        kp, vp = lays[i].k_pool.to(device), lays[i].v_pool.to(device)
        ks, vs = bank.bank(i)
        outs.append(_fused(meta, lays[i], kp, vp, ks, vs, device))
        acc, _ = nsd.spec_accept(*a_dev, qi, int(meta.depth.max()))
        new_len = nsd.commit_lengths(i32(meta.seq_lens, device), qi, acc)
        nl = new_len.cpu().numpy()               # the control path reads the lengths
        src, dst = writeback_pairs(meta.block_table, hosts[i].extent, host_len, nl)
        s_d, d_d = i32(src, device), i32(dst, device)
        h = hosts[i]
        bank.export(i, stream, lambda s, kp=kp, vp=vp, h=h, s_d=s_d, d_d=d_d:
                    nsd.kv_writeback(kp, vp, h.k, h.v, s_d, d_d))
        pools.append((kp, vp))
        lens.append(nl)
    torch.cuda.synchronize()
    n_ref, _ = oracle.accept.spec_accept(a_cpu.p_target.numpy(), a_cpu.q_draft.numpy(),
                                         a_cpu.draft_tokens.numpy(), a_cpu.uniforms.numpy(),
                                         meta.q_indptr)
    len_ref = oracle.commit.commit_lengths(meta.seq_lens, meta.q_indptr, n_ref)
    for i, ((kp, vp), out) in enumerate(zip(pools, outs)):
        ref_k, ref_v = _expect_pool(meta, lays[i])
        assert np.array_equal(u16(kp.cpu()), ref_k[0]) and np.array_equal(u16(vp.cpu()), ref_v[0])
        check_attention(meta, lays[i], out, range(cfg.bs))
        assert np.array_equal(lens[i], len_ref)
        s_ref, d_ref = oracle.commit.writeback_pairs(meta.block_table, hosts[i].extent, host_len,
                                                     len_ref)
        ak, av = arenas0[i][0].copy(), arenas0[i][1].copy()
        ak[d_ref], av[d_ref] = ref_k[0][s_ref], ref_v[0][s_ref]
        assert not np.array_equal(ak, arenas0[i][0])      # the export has work to do
        assert np.array_equal(u16(hosts[i].k), ak) and np.array_equal(u16(hosts[i].v), av)
