"""Pins of the round-closing oracle (oracle/commit.py): the append lands every
window row where the paged layout says (read back through the input generator's
own layout routine), nothing else moves; committed lengths follow the closed
forms of acceptance; the writeback suffix is exactly the blocks holding new
tokens."""
import numpy as np
import torch

from oracle.commit import kv_append, commit_lengths, writeback_pairs
from workload import custom_config, make_meta
from workload.layout import logical_kv_from_blocks


def _rows(meta, hkv, d, seed):
    g = np.random.default_rng(seed)
    return (g.integers(0, 60000, (meta.total_q, hkv, d)).astype(np.uint16),
            g.integers(0, 60000, (meta.total_q, hkv, d)).astype(np.uint16))


def test_append_lands_rows_in_their_slots_and_nothing_else():
    cfg = custom_config(seed=40, bs=5, k_lo=1, k_hi=6, pool_blocks=None)
    meta = make_meta(cfg)
    hkv, d = cfg.num_kv_heads, cfg.head_dim
    kp = np.full((meta.num_blocks, hkv, d // 8, 16, 8), 7, dtype=np.uint16)
    vp = np.full((meta.num_blocks, hkv, d, 16), 9, dtype=np.uint16)
    kn, vn = _rows(meta, hkv, d, 1)
    ok, ov = kv_append(kp, vp, kn, vn, meta.block_table, meta.seq_lens, meta.q_indptr)
    touched_k = np.zeros(kp.shape, dtype=bool)
    for r in range(meta.bs):
        n = meta.nblk(r)
        ids = meta.block_table[r, :n]
        L = int(meta.seq_lens[r])
        a, b = int(meta.q_indptr[r]), int(meta.q_indptr[r + 1])
        k, v = logical_kv_from_blocks(torch.from_numpy(ok[ids].view(np.int16)),
                                      torch.from_numpy(ov[ids].view(np.int16)), L)
        # the window rows read back through the layout routine
        assert np.array_equal(k[L - (b - a):].numpy().view(np.uint16), kn[a:b])
        assert np.array_equal(v[L - (b - a):].numpy().view(np.uint16), vn[a:b])
        # the prefix is untouched
        assert np.all(k[:L - (b - a)].numpy().view(np.uint16) == 7)
        assert np.all(v[:L - (b - a)].numpy().view(np.uint16) == 9)
    # count of changed elements = window rows x heads x dims, in each plane
    assert int((ok != 7).sum()) == meta.total_q * hkv * d
    assert int((ov != 9).sum()) == meta.total_q * hkv * d


def test_commit_lengths_closed_forms():
    L = np.array([100, 64, 33, 17])
    qi = np.array([0, 5, 6, 10, 12])            # K = 4, 0, 3, 1
    assert np.array_equal(commit_lengths(L, qi, [4, 0, 3, 1]), L)            # all accepted
    assert np.array_equal(commit_lengths(L, qi, [0, 0, 0, 0]), L - [4, 0, 3, 1])
    n = np.array([2, 0, 1, 0])
    # the anchor plus the accepted proposals stay: L' = (L - n_q) + 1 + n
    assert np.array_equal(commit_lengths(L, qi, n), L - np.diff(qi) + 1 + n)


def test_writeback_suffix_is_the_blocks_of_new_tokens():
    g = np.random.default_rng(3)
    bs = 40
    bt = np.arange(bs * 20).reshape(bs, 20)[:, ::-1].copy()
    extent = np.cumsum(np.r_[0, np.full(bs - 1, 23)])
    host = g.integers(0, 200, bs)
    new = host + g.integers(0, 40, bs)
    new[0] = host[0]                              # nothing new: nothing written
    src, dst = writeback_pairs(bt, extent, host, new)
    want = []
    for r in range(bs):
        for blk in sorted({t // 16 for t in range(host[r], new[r])}):
            want.append((bt[r, blk], extent[r] + blk))
    assert list(zip(src.tolist(), dst.tolist())) == [tuple(map(int, w)) for w in want]
