"""The one-launch acceptance and sampling kernel (a workgroup per row, used
once a batch has a row for every CU) at the vocabulary sizes where its
one-wave draw gives each lane the longest run of chunk sums (2^19 weights:
32 chunks per lane), against the oracle."""
import numpy as np
import pytest
import torch

import paper_2609_29364_amd as nsd
from workload import custom_config, make_meta, make_accept
from parity import check_accept, check_samples, i32

pytestmark = pytest.mark.gpu

ROWS = 300   # more rows than the MI355X has CUs, so the one-launch kernel runs


@pytest.mark.parametrize("vocab", [1000, 151936, 1 << 19])
def test_sample_one_launch_matches_oracle(device, vocab):
    g = torch.Generator(device=device).manual_seed(vocab + 1)
    rows = torch.rand(ROWS, vocab, generator=g, device=device) ** 6
    rows[1] = 0.0                                   # no mass: -1
    rows[2] = 0.0
    rows[2, vocab - 1] = 3.0                        # one token, at the end
    rows[3, : vocab // 2] = 0.0                     # zero head
    rows[4] *= 1e-30                                # tiny total
    rows[5, 1:] = 0.0                               # one token, at the start
    u = (torch.randint(0, 1 << 24, (ROWS,), generator=g, device=device) * 2.0**-24).float()
    u[0] = 0.0
    u[6] = 1.0 - 2.0**-24
    got = nsd.sample(rows, u)
    torch.cuda.synchronize()
    got = got.cpu().numpy()
    assert got[1] == -1 and got[2] == vocab - 1 and got[5] == 0
    check_samples(rows.cpu().numpy(), u.cpu().numpy(), got)


def test_accept_one_launch_at_the_largest_vocabulary(device):
    cfg = custom_config(seed=77, bs=264, num_q_heads=4, num_kv_heads=2, head_dim=64,
                        ctx_lo=16, ctx_hi=64, k_lo=0, k_hi=3, n_arriving=0, pool_blocks=None,
                        vocab=1 << 19)
    meta = make_meta(cfg)
    acc = make_accept(cfg, meta, device)
    qi = i32(meta.q_indptr, device)
    al, tok = nsd.spec_accept(acc.p_target, acc.q_draft, acc.draft_tokens, acc.uniforms, qi,
                              int(meta.depth.max()))
    torch.cuda.synchronize()
    check_accept(acc.p_target.cpu().numpy(), acc.q_draft.cpu().numpy(),
                 acc.draft_tokens.cpu().numpy(), acc.uniforms.cpu().numpy(), meta.q_indptr,
                 al.cpu().numpy(), tok.cpu().numpy())
    # both outcomes occur: rejections (residual rows) and full acceptances (bonus rows)
    n = al.cpu().numpy()
    assert (n < meta.depth).any() and (n == meta.depth).any()
