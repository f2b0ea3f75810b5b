"""The draft stage on the GPU: inverse-CDF sampling and K steps of append,
single-query attention and sampling, against oracle.draft; and its hand-off
into the acceptance step (draft rows and tokens in the layout spec_accept
reads)."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_29364_amd as nsd
from paper_2609_29364_amd.round import draft_stage
from workload import CONFIGS, custom_config, make_draft
from workload.synth import logical_kv
from parity import ATTN_ATOL, check_accept, check_samples, i32

pytestmark = pytest.mark.gpu


def _grid(g, shape):
    return (torch.randint(0, 1 << 24, shape, generator=g) * 2.0**-24).to(torch.float32)


@pytest.mark.parametrize("vocab", [4, 1000, 4096, 16388, 151936, 1 << 19])
def test_sample_matches_oracle(device, vocab):
    g = torch.Generator().manual_seed(vocab)
    n = 64
    rows = torch.softmax(2.0 * torch.randn(n, vocab, generator=g, dtype=torch.float64), 1)
    rows = rows.to(torch.float32)
    rows[1] = 0.0                                   # no mass: -1
    rows[2] = 0.0
    rows[2, vocab - 1] = 3.0                        # one token, at the end
    rows[3, : vocab // 2] = 0.0                     # zero head
    rows[4] *= 1e-30                                # tiny total
    u = _grid(g, (n,))
    u[0] = 0.0
    u[5] = 1.0 - 2.0**-24
    got = nsd.sample(rows.to(device), u.to(device))
    torch.cuda.synchronize()
    got = got.cpu().numpy()
    assert got[1] == -1 and got[2] == vocab - 1
    check_samples(rows.numpy(), u.numpy(), got)


def test_sample_strided_rows_and_tokens(device):
    # step i of a request-major [bs][K][V] draft block writes tokens [bs][K] column i
    g = torch.Generator().manual_seed(7)
    bs, k, vocab = 33, 5, 1000
    probs = torch.softmax(2.0 * torch.randn(bs, k, vocab, generator=g, dtype=torch.float64), 2)
    probs = probs.to(torch.float32)
    u = _grid(g, (k, bs))
    pd = probs.to(device)
    tok = torch.full((bs, k), -7, dtype=torch.int32, device=device)
    for i in range(k):
        nsd.sample(pd[:, i], u[i].to(device), out=tok[:, i])
    torch.cuda.synchronize()
    tok = tok.cpu().numpy()
    for i in range(k):
        check_samples(probs[:, i].numpy(), u[i].numpy(), tok[:, i])


def test_sample_rejects_bad_arguments(device):
    p = torch.rand(4, 1000, device=device)
    u = torch.rand(4, device=device)
    with pytest.raises(nsd.NsdError):
        nsd.sample(torch.rand(4, 1002, device=device)[:, :999].contiguous(), u)   # vocab % 4
    with pytest.raises(ValueError):
        nsd.sample(p.t(), torch.rand(1000, device=device))                      # strided rows
    with pytest.raises(ValueError):
        nsd.sample(p, u[:3])
    assert nsd.sample(p[:0], u[:0]).numel() == 0


def _run_stage(dd, device, fused):
    meta, lay = dd.meta, dd.layer
    kp, vp = lay.k_pool.clone(), lay.v_pool.clone()
    ks, vs = lay.k_stage.clone(), lay.v_stage.clone()
    qi = i32(np.arange(meta.bs + 1), device)
    kw = dict(k_stage=ks, v_stage=vs)
    if fused:
        kw["stage_table"] = i32(meta.stage_table, device)
    else:
        kw.update(src_ids=i32(meta.src_ids, device), dst_ids=i32(meta.dst_ids, device))
    out, tok = draft_stage(kp, vp, dd.q, dd.k_new, dd.v_new, dd.probs, dd.uniforms,
                           i32(meta.block_table, device), dd.lens, qi, int(meta.seq_lens.max()),
                           **kw)
    torch.cuda.synchronize()
    return out, tok


def _check_stage(dd, out, tok, requests):
    cfg, meta = dd.meta.cfg, dd.meta
    scale = 1.0 / math.sqrt(cfg.head_dim)
    o = out.float().cpu().numpy()
    assert np.isfinite(o).all()
    probs = dd.probs.cpu().numpy()
    u = dd.uniforms.cpu().numpy()
    tok = tok.cpu().numpy()
    worst = 0.0
    for r in requests:
        k, v = logical_kv(meta, dd.layer, r)
        p = int(dd.prefix[r])
        ref, _ = oracle.draft.draft_request(
            k[:p].double().cpu().numpy(), v[:p].double().cpu().numpy(),
            dd.q[:, r].double().cpu().numpy(), dd.k_new[:, r].double().cpu().numpy(),
            dd.v_new[:, r].double().cpu().numpy(), probs[r], u[:, r], scale)
        err = float(np.abs(o[:, r] - ref).max())
        worst = max(worst, err)
        assert err <= ATTN_ATOL, f"request {r} (P={p}): max error {err}"
    # every proposal of every request
    check_samples(probs.reshape(-1, probs.shape[-1]), u.T.reshape(-1), tok.reshape(-1))
    return worst


@pytest.mark.parametrize("fused", [False, True], ids=["gather", "fused"])
@pytest.mark.parametrize("cfg,steps", [
    (custom_config(seed=50, bs=6, ctx_lo=17, ctx_hi=90, k_lo=0, k_hi=0, n_arriving=2,
                   pool_blocks=None), 4),
    (custom_config(seed=51, bs=9, ctx_lo=1, ctx_hi=40, k_lo=0, k_hi=0, n_arriving=4,
                   num_q_heads=16, num_kv_heads=8, head_dim=128, pool_blocks=None), 7),
    (custom_config(seed=52, bs=5, ctx_lo=30, ctx_hi=33, k_lo=0, k_hi=0, n_arriving=5,
                   pool_blocks=None), 16),
    (custom_config(seed=54, bs=3, ctx_lo=5, ctx_hi=40, k_lo=0, k_hi=0, n_arriving=0,
                   pool_blocks=None), 3),
], ids=["tiny_k4", "c2heads_k7", "all_arriving_k16", "none_arriving_k3"])
def test_draft_stage_matches_oracle(device, cfg, steps, fused):
    dd = make_draft(cfg, steps, 1000, device)
    out, tok = _run_stage(dd, device, fused)
    _check_stage(dd, out, tok, range(cfg.bs))


@pytest.mark.parametrize("fused", [False, True], ids=["gather", "fused"])
def test_draft_stage_decode_shape(device, fused):
    # the draft-side decode shape: bs 512, 16 q / 8 kv heads, D 128, contexts
    # 512..2048, a quarter arriving; four proposals over a 151936-token vocabulary
    cfg = CONFIGS["draft_decode"]
    dd = make_draft(cfg, 4, 151936, device)
    out, tok = _run_stage(dd, device, fused)
    meta = dd.meta
    arr = np.nonzero(meta.arriving)[0]
    res = np.nonzero(~meta.arriving)[0]
    order = np.argsort(meta.seq_lens)
    pick = sorted(set([int(order[0]), int(order[-1])] + list(arr[:5]) + list(res[:5])))
    _check_stage(dd, out, tok, pick)


def test_draft_tokens_feed_acceptance(device):
    # draft stage -> verification acceptance: the stage's rows and tokens are
    # spec_accept's q_draft and draft_tokens as they stand
    cfg = custom_config(seed=53, bs=8, ctx_lo=20, ctx_hi=70, k_lo=0, k_hi=0, n_arriving=3,
                        pool_blocks=None)
    k, vocab = 4, 1000
    dd = make_draft(cfg, k, vocab, device)
    _, tok = _run_stage(dd, device, True)
    g = torch.Generator().manual_seed(9)
    p = torch.softmax(2.0 * torch.randn(cfg.bs * (k + 1), vocab, generator=g,
                                        dtype=torch.float64), 1).to(torch.float32)
    u = _grid(g, (cfg.bs * (k + 1),))
    qi = np.arange(cfg.bs + 1, dtype=np.int32) * (k + 1)
    acc, out = nsd.spec_accept(p.to(device), dd.probs.view(-1, vocab), tok.view(-1),
                               u.to(device), i32(qi, device), k)
    torch.cuda.synchronize()
    # the oracle draws the proposals itself from the generator's draft rows and
    # uniforms, then accepts them: nothing it receives came from the library
    rows = dd.probs.cpu().numpy()                                   # [bs][K][V]
    x_ref = oracle.draft.sample(rows.reshape(-1, vocab),
                                dd.uniforms.cpu().numpy().T.reshape(-1)).reshape(cfg.bs, k)
    tok_gpu = tok.cpu().numpy()
    # proposals equal except within the CDF-boundary tolerance (checked by check_samples)
    check_samples(rows.reshape(-1, vocab), dd.uniforms.cpu().numpy().T.reshape(-1),
                  tok_gpu.reshape(-1))
    same = [r for r in range(cfg.bs) if np.array_equal(tok_gpu[r], x_ref[r])]
    assert len(same) == cfg.bs
    ref_acc, ref_tok = oracle.accept.spec_accept(p.numpy(), rows.reshape(-1, vocab),
                                                 x_ref.reshape(-1).astype(np.int32), u.numpy(), qi)
    check_accept(p.numpy(), rows.reshape(-1, vocab), x_ref.reshape(-1).astype(np.int32),
                 u.numpy(), qi, acc.cpu().numpy(), out.cpu().numpy())
    assert np.array_equal(acc.cpu().numpy(), ref_acc)
