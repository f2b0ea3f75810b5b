"""The seeded generator draws what each workload names, reproducibly."""
import numpy as np
import pytest
import torch

from workload import CONFIGS, custom_config, make_meta, make_layer, make_accept
from workload.synth import logical_kv


@pytest.mark.parametrize("name", list(CONFIGS))
def test_meta_matches_the_recipe(name):
    cfg = CONFIGS[name]
    m = make_meta(cfg)
    m2 = make_meta(cfg)
    assert np.array_equal(m.seq_lens, m2.seq_lens) and np.array_equal(m.block_table, m2.block_table)
    assert m.seq_lens.min() >= cfg.ctx_lo and m.seq_lens.max() <= cfg.ctx_hi
    assert m.depth.min() >= cfg.k_lo and m.depth.max() <= cfg.k_hi
    assert m.arriving.sum() == cfg.n_arriving
    used = np.concatenate([m.block_table[r, :m.nblk(r)] for r in range(cfg.bs)])
    assert len(np.unique(used)) == len(used) and used.min() >= 0 and used.max() < m.num_blocks
    assert np.all(m.block_table[:, :][m.block_table < 0] == -1)
    # the plan covers exactly the arriving requests' blocks, destinations distinct
    assert m.n_pairs == sum(m.nblk(r) for r in range(cfg.bs) if m.arriving[r])
    assert len(np.unique(m.dst_ids)) == m.n_pairs
    assert sorted(m.src_ids) == list(range(m.stage_num_blocks))
    assert m.q_indptr[-1] == (m.depth + 1).sum()


def test_ragged_depth_draw():
    m = make_meta(CONFIGS["full_depth"])
    assert set(np.unique(m.depth)) <= set(range(1, 9)) and len(np.unique(m.depth)) > 4


@pytest.mark.parametrize("order", ["extent", "shuffled"])
def test_tiny_layer_poison_and_canary(order):
    cfg = custom_config(staging_order=order)
    m = make_meta(cfg)
    lay = make_layer(cfg, m, 0, "cpu")
    for r in range(cfg.bs):
        k, v = logical_kv(m, lay, r)
        assert k.shape == (m.seq_lens[r], cfg.num_kv_heads, cfg.head_dim)
        assert not torch.isnan(k.float()).any() and not torch.isnan(v.float()).any()
    # arriving destinations are NaN before the gather
    for d in m.dst_ids:
        assert torch.isnan(lay.k_pool[d].float()).all() and torch.isnan(lay.v_pool[d].float()).all()
    # unowned blocks are finite canaries
    owned = set(np.concatenate([m.block_table[r, :m.nblk(r)] for r in range(cfg.bs)]).tolist())
    for b in set(range(m.num_blocks)) - owned:
        assert torch.isfinite(lay.k_pool[b].float()).all()
    # tail slots of the last block are NaN
    for r in range(cfg.bs):
        s = int(m.seq_lens[r]) % 16
        if s and not m.arriving[r]:
            blk = lay.v_pool[m.block_table[r, m.nblk(r) - 1]]
            assert torch.isnan(blk[:, :, s:].float()).all() and torch.isfinite(blk[:, :, :s].float()).all()


def test_accept_inputs():
    cfg = CONFIGS["tiny"]
    m = make_meta(cfg)
    a = make_accept(cfg, m, "cpu")
    assert a.p_target.shape == (m.total_q, cfg.vocab) and a.q_draft.shape == (m.total_q - cfg.bs, cfg.vocab)
    assert torch.allclose(a.p_target.double().sum(1), torch.ones(m.total_q, dtype=torch.float64), atol=1e-5)
    u = a.uniforms.double() * 2**24
    assert torch.equal(u, u.floor()) and a.uniforms.min() >= 0 and a.uniforms.max() < 1
    assert a.draft_tokens.min() >= 0 and a.draft_tokens.max() < cfg.vocab


def test_draft_tokens_follow_draft_rows():
    # Gumbel-max draws: the mean draft probability of the drawn token equals
    # E_q[q(x)] = sum q^2, checked over many rows.
    cfg = custom_config(bs=64, vocab=50, ctx_lo=16, ctx_hi=16, k_lo=8, k_hi=8, n_arriving=0, pool_blocks=None)
    m = make_meta(cfg)
    a = make_accept(cfg, m, "cpu")
    q = a.q_draft.double()
    drawn = q[torch.arange(q.shape[0]), a.draft_tokens.long()]
    expect = (q * q).sum(1)
    assert abs(drawn.mean().item() - expect.mean().item()) < 4 * expect.std().item() / np.sqrt(len(q)) + 0.01
