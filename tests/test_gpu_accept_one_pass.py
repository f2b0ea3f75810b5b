"""The one-launch acceptance and sampling kernel (a workgroup per row, used
when a batch has exactly one row per CU or at least 1.375) at the vocabulary
sizes where its one-wave draw gives each lane the longest run of chunk sums
(2^19 weights: 32 chunks per lane), the empty-residual fallback of both
acceptance paths over many chunks, and strided sampling at the full
vocabulary on both sampling paths, against the oracle."""
import numpy as np
import pytest
import torch

import paper_2609_29364_amd as nsd
from workload import custom_config, make_meta, make_accept
from parity import check_accept, check_samples, i32

pytestmark = pytest.mark.gpu

ROWS = 400   # over 1.375 rows per CU of the MI355X (256 CUs): the one-launch kernel


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


@pytest.mark.parametrize("bs", [300, 360])
def test_accept_at_the_largest_vocabulary(device, bs):
    # 300 requests (just over one per CU) take the two-kernel path, 360 the
    # one-launch kernel
    cfg = custom_config(seed=77, bs=bs, num_q_heads=4, num_kv_heads=2, head_dim=64,
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


@pytest.mark.parametrize("bs", [6, ROWS])
def test_empty_residual_draws_from_the_target_row(device, bs):
    # every proposal lies outside the vocabulary (rejected) and q_0 = p_0, so
    # every residual is empty and the token is drawn from p_0 itself; 16388
    # weights are 65 chunks (more than one per lane of the one-wave draw), so
    # 6 requests take the two-kernel path and ROWS the one-launch kernel
    vocab = 16388
    g = torch.Generator(device=device).manual_seed(bs)
    q_indptr = np.arange(0, 2 * bs + 1, 2, dtype=np.int32)
    p = torch.rand(2 * bs, vocab, generator=g, device=device) ** 4
    p[0, :] = 0.0
    p[0, vocab - 3] = 1.0                               # a one-token target row
    q = p[0::2].contiguous()                            # q_0 = p_0 exactly
    x = torch.full((bs,), vocab + 5, dtype=torch.int32, device=device)
    u = (torch.randint(0, 1 << 24, (2 * bs,), generator=g, device=device) * 2.0**-24).float()
    acc, tok = nsd.spec_accept(p, q, x, u, i32(q_indptr, device), 1)
    torch.cuda.synchronize()
    acc, tok = acc.cpu().numpy(), tok.cpu().numpy()
    assert (acc == 0).all() and tok[0] == vocab - 3
    check_accept(p.cpu().numpy(), q.cpu().numpy(), x.cpu().numpy(), u.cpu().numpy(), q_indptr,
                 acc, tok)


@pytest.mark.parametrize("n", [64, ROWS])
def test_sample_strided_rows_at_full_vocabulary(device, n):
    # step i of request-major [n][K][V] draft rows (row stride K * V) into
    # column i of [n][K] tokens (stride K), at the draft vocabulary, on the
    # two-kernel path (64 rows) and the one-launch kernel (ROWS rows)
    vocab, k = 151936, 3
    g = torch.Generator(device=device).manual_seed(n + 3)
    probs = torch.rand(n, k, vocab, generator=g, device=device) ** 8
    u = (torch.randint(0, 1 << 24, (k, n), generator=g, device=device) * 2.0**-24).float()
    tok = torch.full((n, k), -7, dtype=torch.int32, device=device)
    for i in range(k):
        nsd.sample(probs[:, i], u[i], out=tok[:, i])
    torch.cuda.synchronize()
    tok, u = tok.cpu().numpy(), u.cpu().numpy()
    for i in range(k):
        check_samples(probs[:, i].cpu().numpy(), u[i], tok[:, i])
