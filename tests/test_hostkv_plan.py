"""Host-side logic of the HostKV preparation (no GPU): the arena layout keeps
each request's logical KV at its extent, and the H2D plan maps every arriving
block from its arena block to the staging id its stage table names, matching
the gather's (staging id, pool id) pairs."""
import numpy as np
import torch

from paper_2609_29364_amd.hostkv import h2d_plan
from workload import CONFIGS, custom_config, make_meta, make_layer, make_hostkv
from workload.synth import logical_kv
from workload.layout import logical_kv_from_blocks


def _round(cfg):
    meta = make_meta(cfg)
    lay = make_layer(cfg, meta, 0, "cpu")
    return meta, lay, make_hostkv(cfg, meta, lay, pin=False)


def test_arena_holds_every_request_at_its_extent():
    for cfg in (CONFIGS["tiny"], custom_config(staging_order="shuffled", seed=10)):
        meta, lay, host = _round(cfg)
        # extents are disjoint and within the arena
        order = np.argsort(host.extent)
        ends = host.extent[order] + host.capacity[order]
        assert np.all(host.extent[order][1:] >= ends[:-1]) and ends[-1] <= host.k.shape[0]
        for r in range(meta.bs):
            n = meta.nblk(r)
            assert host.capacity[r] >= n
            kb, vb = host.k[host.extent[r]:host.extent[r] + n], host.v[host.extent[r]:host.extent[r] + n]
            k, v = logical_kv_from_blocks(kb, vb, int(meta.seq_lens[r]))
            k0, v0 = logical_kv(meta, lay, r)
            assert torch.equal(k.view(torch.int16), k0.view(torch.int16))
            assert torch.equal(v.view(torch.int16), v0.view(torch.int16))


def test_plan_moves_each_arriving_block_to_its_staging_id():
    cfg = custom_config(staging_order="shuffled", seed=11, bs=6, n_arriving=4, pool_blocks=None)
    meta, lay, host = _round(cfg)
    bb = host.k[0].numel() * 2
    plan = h2d_plan(host.extent, meta.stage_table, meta.arriving, meta.seq_lens, bb)
    # brute force: one triple per arriving block, in request order
    want = []
    for r in range(meta.bs):
        if not meta.arriving[r]:
            continue
        for j in range(meta.nblk(r)):
            want.append(((host.extent[r] + j) * bb, meta.stage_table[r, j] * bb, bb))
    assert np.array_equal(plan, np.array(want, dtype=np.int64))
    # the destination blocks are exactly the gather's staging ids, each once
    assert sorted((plan[:, 1] // bb).tolist()) == sorted(meta.src_ids.tolist())
    # applying the plan on the host reproduces the staging pool at those ids
    hk = host.k.view(torch.uint8).numpy().reshape(-1)
    st = np.zeros(lay.k_stage.numel() * 2, dtype=np.uint8)
    for s, d, n in plan:
        st[d:d + n] = hk[s:s + n]
    ref = lay.k_stage.view(torch.uint8).numpy().reshape(-1)
    for i in meta.src_ids:
        assert np.array_equal(st[i * bb:(i + 1) * bb], ref[i * bb:(i + 1) * bb])


def test_plan_of_a_round_with_no_arrivals_is_empty():
    cfg = custom_config(n_arriving=0, seed=12)
    meta, lay, host = _round(cfg)
    assert h2d_plan(host.extent, meta.stage_table, meta.arriving, meta.seq_lens, 4096).shape == (0, 3)


def test_writeback_pairs_match_the_oracle():
    import oracle
    from paper_2609_29364_amd.hostkv import writeback_pairs
    g = np.random.default_rng(4)
    bs = 30
    bt = g.permutation(bs * 16).reshape(bs, 16).astype(np.int32)
    extent = np.cumsum(np.r_[0, g.integers(17, 20, bs - 1)])
    host = g.integers(0, 180, bs)
    new = host + g.integers(0, 60, bs)
    new = np.minimum(new, 256)
    new[3] = host[3]
    s1, d1 = writeback_pairs(bt, extent, host, new)
    s2, d2 = oracle.commit.writeback_pairs(bt, extent, host, new)
    assert np.array_equal(s1, s2) and np.array_equal(d1, d2)


def test_plans_refuse_offsets_they_cannot_represent():
    # negative extents or staging ids and byte offsets past 2^63 - 1 are
    # refused instead of wrapping around
    import pytest
    import paper_2609_29364_amd as nsd
    from paper_2609_29364_amd.hostkv import writeback_pairs
    st = np.array([[3, 4]], np.int32)
    lens = np.array([20], np.int32)
    arriving = np.array([1], np.uint8)
    ok = h2d_plan(np.array([5], np.int64), st, arriving, lens, 4096)
    assert ok.tolist() == [[5 * 4096, 3 * 4096, 4096], [6 * 4096, 4 * 4096, 4096]]
    for extent, table, block_bytes in (([-1], st, 4096), ([5], np.array([[3, -2]], np.int32), 4096),
                                       ([2**31 - 1], st, 2**40), ([0], st, 2**62),
                                       ([2**62], st, 2)):
        with pytest.raises(nsd.NsdError):
            h2d_plan(np.array(extent, np.int64), table, arriving, lens, block_bytes)
    # the largest representable offsets still plan
    big = h2d_plan(np.array([2**31], np.int64), st, arriving, lens, 2**31)
    assert big[1].tolist() == [(2**31 + 1) * 2**31, 4 * 2**31, 2**31]
    bt = np.array([[7, 8]], np.int32)
    assert [x.tolist() for x in writeback_pairs(bt, np.array([10], np.int64), np.array([0]),
                                                np.array([20]))] == [[7, 8], [10, 11]]
    with pytest.raises(nsd.NsdError):
        writeback_pairs(bt, np.array([-3], np.int64), np.array([0]), np.array([20]))
    with pytest.raises(nsd.NsdError):
        writeback_pairs(bt, np.array([2**31], np.int64), np.array([0]), np.array([20]))
