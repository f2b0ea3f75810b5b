"""Randomised GPU parity: many small verification rounds with random shapes,
every request checked against the oracle.

Each case draws a batch size, KV-head count and group size (query heads per KV
head), head dimension, per-request context lengths and draft depths (ragged),
an arriving set (none, all, or a random subset), a staging order, and a wave
count for the attention's work split (few waves: mostly whole items; many:
items cut into partials merged by the second kernel).  The same round runs
through the separate gather + attention and through the fused pass, and an
acceptance step runs on random rows.  The cases are seeded, so a failure
names its case and reproduces."""
import numpy as np
import pytest

from workload import custom_config, make_meta
from test_gpu_round_small import _check_all

pytestmark = pytest.mark.gpu

N_CASES = 400


def _case(seed):
    rng = np.random.default_rng(1000 + seed)
    d = int(rng.choice([64, 128]))
    hkv = int(rng.choice([1, 2, 4, 8]))
    max_q = int(rng.integers(1, 10))
    groups = [g for g in (1, 2, 4, 8) if g * max_q <= 64]
    group = int(rng.choice(groups))
    bs = int(rng.integers(1, 41))
    lens = rng.integers(1, 700, bs)
    lens = np.where(rng.random(bs) < 0.15, rng.integers(1, 17, bs), lens)   # some very short
    depth = np.minimum(rng.integers(0, max_q, bs), lens - 1)
    kind = rng.choice(["none", "all", "some"], p=[0.15, 0.15, 0.7])
    arriving = {"none": np.zeros(bs, bool), "all": np.ones(bs, bool),
                "some": rng.random(bs) < 0.4}[kind]
    vocab = int(rng.choice([0, 64, 1000, 4096, 16388]))   # 16388: 65 chunks, the two-kernel path
    cfg = custom_config(seed=2000 + seed, bs=bs, num_q_heads=group * hkv, num_kv_heads=hkv,
                        head_dim=d, vocab=vocab, n_arriving=int(arriving.sum()),
                        pool_blocks=None, k_lo=0, k_hi=max_q - 1,
                        staging_order=str(rng.choice(["extent", "shuffled"])))
    meta = make_meta(cfg, seq_lens=lens, depth=depth, arriving=arriving)
    waves = [None, 4, 8, 12, 36][int(rng.integers(0, 5))]
    return cfg, meta, waves


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_round(device, seed):
    cfg, meta, waves = _case(seed)
    print(f"case {seed}: bs={cfg.bs} heads={cfg.num_q_heads}/{cfg.num_kv_heads} "
          f"D={cfg.head_dim} max_q={meta.max_q} arriving={int(meta.arriving.sum())} "
          f"vocab={cfg.vocab} waves={waves}", flush=True)
    for fused in (False, True):
        _check_all(cfg, meta, device, waves=waves, fused=fused)
