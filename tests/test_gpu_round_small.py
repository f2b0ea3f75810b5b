"""GPU parity on small rounds: every step against the oracle, element by element,
plus edge cases (ragged depths, L mod 16 in {0, 1, 15}, L = n_q, every GQA
group size, both head dims).  The attention's work decomposition is forced
through few waves (most items whole) and the device's full wave count (most
items cut into partials) through the library's wave-count hook."""

import numpy as np
import pytest
import torch

import oracle
import paper_2609_29364_amd as nsd
from paper_2609_29364_amd.round import verify_round, FUSED_MIN_BATCH
from workload import CONFIGS, custom_config, make_meta, make_layer, make_accept
from parity import i32, u16, check_attention, check_accept

pytestmark = pytest.mark.gpu


def _run_round(cfg, meta, dev, layers=None, accept=True, waves=None, fused=False, prepare=None):
    layers = layers or [make_layer(cfg, meta, l, "cpu") for l in range(cfg.num_layers)]
    stack = lambda name: torch.stack([getattr(l, name) for l in layers]).to(dev).contiguous()
    kp, vp, ks, vs, q = (stack(n) for n in ("k_pool", "v_pool", "k_stage", "v_stage", "q"))
    acc_in = make_accept(cfg, meta, "cpu") if (accept and cfg.vocab) else None
    acc_dev = None
    if acc_in is not None:
        acc_dev = (acc_in.p_target.to(dev), acc_in.q_draft.to(dev), acc_in.draft_tokens.to(dev),
                   acc_in.uniforms.to(dev), int(meta.depth.max()))
    with nsd.attention_waves(waves):
        prepare = prepare or ("fused" if fused else "gather")
        st = i32(meta.stage_table, dev) if prepare != "gather" else None
        outs, acc, tok = verify_round(kp, vp, ks, vs, i32(meta.src_ids, dev),
                                      i32(meta.dst_ids, dev), q, i32(meta.block_table, dev),
                                      i32(meta.seq_lens, dev), i32(meta.q_indptr, dev),
                                      meta.max_q, meta.max_seq_len, accept=acc_dev,
                                      stage_table=st, prepare=prepare)
        torch.cuda.synchronize()
    return layers, kp, vp, outs, acc_in, acc, tok


def _check_all(cfg, meta, dev, **kw):
    layers, kp, vp, outs, acc_in, acc, tok = _run_round(cfg, meta, dev, **kw)
    ref_k, ref_v = oracle.gather.kv_gather(
        np.stack([u16(l.k_stage) for l in layers]), np.stack([u16(l.v_stage) for l in layers]),
        np.stack([u16(l.k_pool) for l in layers]), np.stack([u16(l.v_pool) for l in layers]),
        meta.src_ids, meta.dst_ids)
    assert np.array_equal(u16(kp), ref_k) and np.array_equal(u16(vp), ref_v)
    for l, lay in enumerate(layers):
        check_attention(meta, lay, outs[l], range(cfg.bs))
    if acc_in is not None:
        check_accept(acc_in.p_target.numpy(), acc_in.q_draft.numpy(),
                     acc_in.draft_tokens.numpy(), acc_in.uniforms.numpy(), meta.q_indptr,
                     acc.cpu().numpy(), tok.cpu().numpy())
    return outs


@pytest.mark.parametrize("fused", [False, True])
def test_tiny_round(device, fused):
    cfg = CONFIGS["tiny"]
    _check_all(cfg, make_meta(cfg), device, fused=fused)


@pytest.mark.parametrize("fused", [False, True])
def test_tiny_round_shuffled_staging(device, fused):
    cfg = custom_config(staging_order="shuffled", seed=10)
    _check_all(cfg, make_meta(cfg), device, fused=fused)


CASES = [
    # (Hq, Hkv, D, seq_lens, depths)
    (4, 4, 64, [16, 17, 31], [4, 0, 2]),
    (4, 2, 128, [1, 33, 47, 64], [0, 8, 3, 1]),
    (32, 8, 128, [5, 100, 513, 1024, 1500], [4, 4, 4, 4, 4]),
    (8, 1, 64, [8, 64, 65, 300], [7, 6, 5, 4]),
    (16, 8, 128, [1, 2, 15, 16, 17, 31, 32, 33], [0, 0, 0, 0, 0, 0, 0, 0]),
    (32, 8, 64, [9, 47, 48, 49, 95, 96], [8, 8, 8, 8, 8, 8]),
]


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("waves", [None, 4, 12])
@pytest.mark.parametrize("fused", [False, True])
def test_attention_edge_cases(device, case, waves, fused):
    hq, hkv, d, lens, depth = CASES[case]
    bs = len(lens)
    cfg = custom_config(seed=100 + case, bs=bs, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                        vocab=0, n_arriving=bs // 2, pool_blocks=None)
    arriving = np.arange(bs) % 2 == 1
    meta = make_meta(cfg, seq_lens=lens, depth=depth, arriving=arriving)
    _check_all(cfg, meta, device, waves=waves, fused=fused)


ARRIVING_SETS = {
    "none": [], "all": list(range(8)), "first": [0], "last": [7],
    "head_half": [0, 1, 2, 3], "tail_half": [4, 5, 6, 7], "scattered": [1, 2, 6],
}


@pytest.mark.parametrize("waves", [None, 4, 12])
@pytest.mark.parametrize("aset", sorted(ARRIVING_SETS))
def test_fused_arriving_sets(device, aset, waves):
    """The fused pass works on resident requests and arriving requests as two
    segments, each split over the waves on its own; every arriving set (none,
    all, one at either end, contiguous halves, scattered) gives the gather's
    bytes and the oracle's attention."""
    lens = [40, 300, 17, 129, 1, 64, 500, 33]
    depth = [3, 4, 0, 8, 0, 2, 5, 1]
    arriving = np.zeros(8, dtype=bool)
    arriving[ARRIVING_SETS[aset]] = True
    cfg = custom_config(seed=300, bs=8, num_q_heads=8, num_kv_heads=2, head_dim=128, vocab=0,
                        n_arriving=int(arriving.sum()), pool_blocks=None)
    meta = make_meta(cfg, seq_lens=lens, depth=depth, arriving=arriving)
    _check_all(cfg, meta, device, waves=waves, fused=True)


def test_ragged_batch_of_64(device):
    rng = np.random.default_rng(5)
    lens = rng.integers(1, 700, 64)
    depth = np.minimum(rng.integers(0, 9, 64), lens - 1)
    cfg = custom_config(seed=7, bs=64, num_q_heads=32, num_kv_heads=8, head_dim=128, vocab=2048,
                        n_arriving=20, pool_blocks=None, k_lo=0, k_hi=8)
    meta = make_meta(cfg, seq_lens=lens, depth=depth)
    for fused in (False, True):
        _check_all(cfg, meta, device, fused=fused)
        _check_all(cfg, meta, device, waves=8, fused=fused)
        _check_all(cfg, meta, device, waves=36, fused=fused)


@pytest.mark.parametrize("bs", [1, 4, 12])
def test_small_batches_of_long_requests(device, bs):
    """Small batches of verify_8b-shaped requests (32/8 heads, head_dim 128,
    contexts up to 4096, K = 4): the launch uses only about one wave per 20
    K/V blocks, and every item is cut into parts that the merge kernel
    combines.  Every request is checked, fused and not."""
    rng = np.random.default_rng(40 + bs)
    lens = rng.integers(1024, 4097, bs)
    depth = np.full(bs, 4)
    cfg = custom_config(seed=41 + bs, bs=bs, num_q_heads=32, num_kv_heads=8, head_dim=128,
                        vocab=4096, n_arriving=max(1, bs // 3), pool_blocks=None, k_lo=4,
                        k_hi=4)
    meta = make_meta(cfg, seq_lens=lens, depth=depth)
    for fused in (False, True):
        _check_all(cfg, meta, device, fused=fused)


@pytest.mark.parametrize("fused", [False, True])
def test_largest_batch(device, fused):
    """The largest batch the attention entry points take (8192 requests): the
    work order and span prefix of the whole batch sit in LDS.  Short contexts
    keep the oracle quick; every request is checked."""
    bs = 8192
    rng = np.random.default_rng(21)
    lens = rng.integers(1, 48, bs)
    depth = np.minimum(rng.integers(0, 4, bs), lens - 1)
    cfg = custom_config(seed=22, bs=bs, num_q_heads=4, num_kv_heads=2, head_dim=64, vocab=0,
                        n_arriving=int(0.3 * bs), pool_blocks=None, k_lo=0, k_hi=3)
    meta = make_meta(cfg, seq_lens=lens, depth=depth)
    _check_all(cfg, meta, device, fused=fused)
    # one request more than the limit is refused before any launch
    q = torch.zeros((bs + 1, 4, 64), dtype=torch.bfloat16, device=device)
    with pytest.raises(nsd.NsdError):
        nsd.verify_attention(q, torch.zeros((4, 2, 8, 16, 8), dtype=torch.bfloat16, device=device),
                             torch.zeros((4, 2, 64, 16), dtype=torch.bfloat16, device=device),
                             torch.zeros((bs + 1, 1), dtype=torch.int32, device=device),
                             torch.ones(bs + 1, dtype=torch.int32, device=device),
                             torch.arange(bs + 2, dtype=torch.int32, device=device), 1, 1)


def test_multi_layer_gather_subrange(device):
    cfg = custom_config(seed=3, num_layers=3)
    meta = make_meta(cfg)
    layers = [make_layer(cfg, meta, l, "cpu") for l in range(3)]
    stack = lambda name: torch.stack([getattr(l, name) for l in layers]).to(device).contiguous()
    kp, vp, ks, vs = (stack(n) for n in ("k_pool", "v_pool", "k_stage", "v_stage"))
    nsd.kv_gather(ks, vs, kp, vp, i32(meta.src_ids, device), i32(meta.dst_ids, device),
                  layer0=1, n_layers=1)
    torch.cuda.synchronize()
    ref_k, ref_v = oracle.gather.kv_gather(
        np.stack([u16(l.k_stage) for l in layers]), np.stack([u16(l.v_stage) for l in layers]),
        np.stack([u16(l.k_pool) for l in layers]), np.stack([u16(l.v_pool) for l in layers]),
        meta.src_ids, meta.dst_ids, layer0=1, n_layers=1)
    assert np.array_equal(u16(kp), ref_k) and np.array_equal(u16(vp), ref_v)


def test_gather_empty_plan_and_idempotence(device):
    cfg = CONFIGS["tiny"]
    meta = make_meta(cfg)
    lay = make_layer(cfg, meta, 0, "cpu")
    kp, vp = lay.k_pool.to(device), lay.v_pool.to(device)
    ks, vs = lay.k_stage.to(device), lay.v_stage.to(device)
    e = torch.zeros(0, dtype=torch.int32, device=device)
    nsd.kv_gather(ks, vs, kp, vp, e, e)
    torch.cuda.synchronize()
    assert np.array_equal(u16(kp), u16(lay.k_pool))
    src, dst = i32(meta.src_ids, device), i32(meta.dst_ids, device)
    nsd.kv_gather(ks, vs, kp, vp, src, dst)
    once = u16(kp).copy()
    nsd.kv_gather(ks, vs, kp, vp, src, dst)
    assert np.array_equal(u16(kp), once)


def test_attention_deterministic_and_permutation_invariant(device):
    cfg = custom_config(seed=21, bs=6, num_q_heads=32, num_kv_heads=8, head_dim=128, vocab=0,
                        ctx_lo=200, ctx_hi=900, n_arriving=0, pool_blocks=None)
    meta = make_meta(cfg)
    lay = make_layer(cfg, meta, 0, "cpu")
    q = lay.q.to(device)
    args = (i32(meta.seq_lens, device), i32(meta.q_indptr, device), meta.max_q, meta.max_seq_len)
    kp, vp = lay.k_pool.to(device), lay.v_pool.to(device)
    bt = i32(meta.block_table, device)
    o1 = nsd.verify_attention(q, kp, vp, bt, *args).clone()
    o2 = nsd.verify_attention(q, kp, vp, bt, *args).clone()
    # same logical cache under a different physical placement
    sigma = np.random.default_rng(1).permutation(meta.num_blocks)
    kp2, vp2 = torch.empty_like(kp), torch.empty_like(vp)
    sig = torch.as_tensor(sigma, device=device)
    kp2[sig] = kp
    vp2[sig] = vp
    bt2 = np.where(meta.block_table >= 0, sigma[np.maximum(meta.block_table, 0)], -1)
    o3 = nsd.verify_attention(q, kp2, vp2, i32(bt2, device), *args)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(o1.view(torch.int16), o3.view(torch.int16))
    check_attention(meta, lay, o1, range(cfg.bs))


@pytest.mark.parametrize("waves", [None, 8])
def test_workspace_reuse(device, waves):
    # calls that reuse one workspace (split partials of the previous call still in it),
    # alternating the fused and unfused entry points, agree bit for bit
    cfg = custom_config(seed=22, bs=5, num_q_heads=16, num_kv_heads=4, head_dim=128, vocab=0,
                        ctx_lo=300, ctx_hi=1200, k_lo=2, k_hi=2, n_arriving=2, pool_blocks=None)
    meta = make_meta(cfg)
    lay = make_layer(cfg, meta, 0, "cpu")
    with nsd.attention_waves(waves):
        n = nsd.verify_attention_workspace_size(cfg.bs, cfg.num_q_heads, cfg.num_kv_heads,
                                                cfg.head_dim, meta.max_q, meta.max_seq_len)
        ws = nsd.new_workspace(n, device)
        q = lay.q.to(device)
        sl, qi, bt = (i32(meta.seq_lens, device), i32(meta.q_indptr, device),
                      i32(meta.block_table, device))
        kp, vp = lay.k_pool.to(device), lay.v_pool.to(device)
        outs = []
        for fused in (False, True, True, False):
            k2, v2 = kp.clone(), vp.clone()
            if fused:
                o = nsd.gather_verify_attention(q, k2, v2, lay.k_stage.to(device),
                                                lay.v_stage.to(device), bt,
                                                i32(meta.stage_table, device), sl, qi,
                                                meta.max_q, meta.max_seq_len, workspace=ws)
            else:
                nsd.kv_gather(lay.k_stage.to(device), lay.v_stage.to(device), k2, v2,
                              i32(meta.src_ids, device), i32(meta.dst_ids, device))
                o = nsd.verify_attention(q, k2, v2, bt, sl, qi, meta.max_q, meta.max_seq_len,
                                         workspace=ws)
            torch.cuda.synchronize()
            outs.append(o.clone())
    assert torch.equal(outs[1].view(torch.int16), outs[2].view(torch.int16))
    assert torch.equal(outs[0].view(torch.int16), outs[3].view(torch.int16))
    for o in outs:
        check_attention(meta, lay, o, range(cfg.bs))


def test_out_of_range_block_ids_are_invisible(device):
    # a block id past the pool makes its tokens invisible; nothing faults
    cfg = custom_config(seed=31, bs=2, vocab=0, n_arriving=0, ctx_lo=64, ctx_hi=64, k_lo=0, k_hi=0,
                        pool_blocks=None)
    meta = make_meta(cfg)
    lay = make_layer(cfg, meta, 0, "cpu")
    bt = meta.block_table.copy()
    bt[1, 3] = meta.num_blocks + 1000   # last block of request 1: its 16 tokens vanish
    out = nsd.verify_attention(lay.q.to(device), lay.k_pool.to(device), lay.v_pool.to(device),
                               i32(bt, device), i32(meta.seq_lens, device),
                               i32(meta.q_indptr, device), 1, 64)
    torch.cuda.synchronize()
    check_attention(meta, lay, out, [0])
    # request 1's only query (position 63) lives in the dropped block: it sees tokens 0..47
    from workload.synth import logical_kv
    k, v = logical_kv(meta, lay, 1)
    qr = lay.q[1:2].double().numpy()
    ref = oracle.attention.verify_attention_request(qr, k[:48].double().numpy(),
                                                    v[:48].double().numpy(), 0.125)
    # the oracle places the query at the last visible position, which is the same set of keys
    assert np.abs(out[1:2].float().cpu().numpy() - ref).max() <= 2e-2


def test_fused_out_of_range_ids(device):
    # fused pass: a staging id past the staging pool hides its tokens and leaves the
    # destination unwritten; a destination id past the pool is not written, while its
    # (valid) staged tokens stay visible
    cfg = custom_config(seed=32, bs=2, vocab=0, n_arriving=2, ctx_lo=64, ctx_hi=64, k_lo=0,
                        k_hi=0, pool_blocks=None)
    meta = make_meta(cfg)
    lay = make_layer(cfg, meta, 0, "cpu")
    st = meta.stage_table.copy()
    bt = meta.block_table.copy()
    st[1, 3] = meta.stage_num_blocks + 100   # request 1: tokens 48..63 vanish, block not written
    bt[0, 2] = meta.num_blocks + 5           # request 0: block 2 not written, still attended
    kp, vp = lay.k_pool.to(device), lay.v_pool.to(device)
    out = nsd.gather_verify_attention(lay.q.to(device), kp, vp, lay.k_stage.to(device),
                                      lay.v_stage.to(device), i32(bt, device), i32(st, device),
                                      i32(meta.seq_lens, device), i32(meta.q_indptr, device), 1, 64)
    torch.cuda.synchronize()
    # pool: the pairs that stayed valid are copied, the two dropped blocks keep their bytes
    keep = [(int(meta.stage_table[r, b]), int(meta.block_table[r, b]))
            for r in range(2) for b in range(4) if (r, b) not in ((1, 3), (0, 2))]
    ref_k, ref_v = oracle.gather.kv_gather(u16(lay.k_stage)[None], u16(lay.v_stage)[None],
                                           u16(lay.k_pool)[None], u16(lay.v_pool)[None],
                                           np.array([a for a, _ in keep]),
                                           np.array([b for _, b in keep]))
    assert np.array_equal(u16(kp.cpu()), ref_k[0]) and np.array_equal(u16(vp.cpu()), ref_v[0])
    from workload.synth import logical_kv
    qs = lay.q.double().numpy()
    k0, v0 = logical_kv(meta, lay, 0)
    ref0 = oracle.attention.verify_attention_request(qs[0:1], k0.double().numpy(),
                                                     v0.double().numpy(), 0.125)
    k1, v1 = logical_kv(meta, lay, 1)
    ref1 = oracle.attention.verify_attention_request(qs[1:2], k1[:48].double().numpy(),
                                                     v1[:48].double().numpy(), 0.125)
    got = out.float().cpu().numpy()
    assert np.abs(got[0:1] - ref0).max() <= 2e-2
    assert np.abs(got[1:2] - ref1).max() <= 2e-2


# ---------------------------------------------------------------- acceptance

def _accept(dev, p, q, x, u, q_indptr, max_k):
    t = lambda a, dt: torch.as_tensor(np.ascontiguousarray(a), dtype=dt, device=dev)
    acc, tok = nsd.spec_accept(t(p, torch.float32), t(q, torch.float32) if max_k else None,
                               t(x, torch.int32) if max_k else None, t(u, torch.float32),
                               t(q_indptr, torch.int32), max_k)
    torch.cuda.synchronize()
    return acc.cpu().numpy(), tok.cpu().numpy()


def _probs(rng, rows, vocab, sigma=2.0):
    z = sigma * rng.standard_normal((rows, vocab))
    e = np.exp(z - z.max(1, keepdims=True))
    return (e / e.sum(1, keepdims=True)).astype(np.float32)


def _batch(depth):
    q_indptr = np.concatenate([[0], np.cumsum(np.array(depth) + 1)]).astype(np.int32)
    return q_indptr, int(q_indptr[-1]), len(depth)


def test_accept_random_ragged(device):
    rng = np.random.default_rng(0)
    depth = rng.integers(0, 9, 300)
    q_indptr, tq, bs = _batch(depth)
    vocab = 4096
    p = _probs(rng, tq, vocab, 1.0)
    q = _probs(rng, tq - bs, vocab, 1.0)
    x = np.array([rng.choice(vocab, p=row.astype(np.float64) / row.astype(np.float64).sum())
                  for row in q], dtype=np.int32)
    u = (rng.integers(0, 1 << 24, tq) * 2.0**-24).astype(np.float32)
    acc, tok = _accept(device, p, q, x, u, q_indptr, 8)
    check_accept(p, q, x, u, q_indptr, acc, tok)
    assert acc.max() >= 2   # some requests accept several proposals


def test_accept_identical_rows_accept_all(device):
    rng = np.random.default_rng(1)
    depth = [4] * 16
    q_indptr, tq, bs = _batch(depth)
    p = _probs(rng, tq, 1000)
    q = np.concatenate([p[q_indptr[r]:q_indptr[r] + 4] for r in range(bs)])
    x = rng.integers(0, 1000, tq - bs).astype(np.int32)
    u = (rng.integers(0, 1 << 24, tq) * 2.0**-24).astype(np.float32)
    acc, tok = _accept(device, p, q, x, u, q_indptr, 4)
    assert np.all(acc == 4)
    check_accept(p, q, x, u, q_indptr, acc, tok)


def _special_cases():
    """Five requests: forced one-hot residual, out-of-vocabulary proposal with
    an empty residual, exact tie, K = 0 at u = 1 - 2^-24, u on a CDF boundary."""
    vocab = 16
    depth = [1, 1, 1, 0, 2]
    q_indptr, tq, bs = _batch(depth)
    p = np.full((tq, vocab), 1.0 / vocab, np.float32)
    q = np.full((tq - bs, vocab), 1.0 / vocab, np.float32)
    x = np.zeros(tq - bs, np.int32)
    u = np.full(tq, 0.5, np.float32)
    # r0: one-hot residual forced: proposal 3 has p = 0, p_0 one-hot at 9
    a = q_indptr[0]
    p[a] = 0
    p[a, 9] = 1.0
    x[0] = 3
    # r1: out-of-vocabulary proposal with p_0 = q_0: rejected, residual empty -> draw from p_0
    x[1] = vocab + 5
    # r2: exact tie u*q = p -> accepted; bonus from p_1 one-hot at 12
    a = q_indptr[2]
    q[2] = 0
    q[2, 7] = 0.5
    p[a] = 0
    p[a, 7] = 0.25
    p[a, 1] = 0.75
    x[2] = 7
    p[a + 1] = 0
    p[a + 1, 12] = 1.0
    # r3: K = 0: plain draw from p_0 at u = 1 - 2^-24 -> the last token of weight
    a = q_indptr[3]
    p[a] = 0
    p[a, 2] = 0.5
    p[a, 5] = 0.5
    u[a] = np.float32(1 - 2**-24)
    # r4: u exactly on a CDF boundary of exactly representable weights
    a = q_indptr[4]
    x[3], x[4] = 0, 1
    p[a + 2] = np.array([0.25, 0.25, 0, 0.5] + [0] * 12, np.float32)
    u[a + 2] = 0.25
    return p, q, x, u, depth


def _check_special(acc, tok, q_indptr, r0=0):
    assert list(acc[r0:r0 + 5]) == [0, 0, 1, 0, 2]
    assert tok[q_indptr[r0]] == 9
    assert tok[q_indptr[r0 + 2]:q_indptr[r0 + 2] + 2].tolist() == [7, 12]
    assert tok[q_indptr[r0 + 3]] == 5
    assert tok[q_indptr[r0 + 4] + 2] == 1


def test_accept_special_cases(device):
    p, q, x, u, depth = _special_cases()
    q_indptr, _, _ = _batch(depth)
    acc, tok = _accept(device, p, q, x, u, q_indptr, 2)
    _check_special(acc, tok, q_indptr)
    check_accept(p, q, x, u, q_indptr, acc, tok)


def test_accept_special_cases_one_pass(device):
    """The same cases in a batch with more rows than the device has CUs, which
    takes the one-kernel path (one workgroup per row, sums kept in LDS)."""
    p, q, x, u, depth = _special_cases()
    reps = 60
    assert reps * len(depth) >= torch.cuda.get_device_properties(device).multi_processor_count
    q_indptr, _, _ = _batch(depth * reps)
    pt, qt = np.tile(p, (reps, 1)), np.tile(q, (reps, 1))
    xt, ut = np.tile(x, reps), np.tile(u, reps)
    acc, tok = _accept(device, pt, qt, xt, ut, q_indptr, 2)
    for rep in range(reps):
        _check_special(acc, tok, q_indptr, rep * len(depth))
    check_accept(pt, qt, xt, ut, q_indptr, acc, tok)


def test_accept_workspace_contents_do_not_matter(device):
    # the chunk sums are written before they are read: a workspace full of NaN
    # bytes, then reused across calls of different sizes, gives the same result
    rng = np.random.default_rng(5)
    out = []
    for depth, vocab in (([3, 0, 5, 1], 16388), ([2] * 9, 1000), ([3, 0, 5, 1], 16388)):
        q_indptr, tq, bs = _batch(depth)
        p = _probs(rng, tq, vocab)
        q = _probs(rng, tq - bs, vocab)
        x = rng.integers(0, vocab, tq - bs).astype(np.int32)
        u = (rng.integers(0, 1 << 24, tq) * 2.0**-24).astype(np.float32)
        out.append((p, q, x, u, q_indptr, max(depth)))
    ws = torch.full((nsd.accept_workspace_size(9, 16388),), 0xFF, dtype=torch.uint8,
                    device=device)
    t = lambda a, dt: torch.as_tensor(np.ascontiguousarray(a), dtype=dt, device=device)
    for p, q, x, u, q_indptr, mk in out:
        acc, tok = nsd.spec_accept(t(p, torch.float32), t(q, torch.float32), t(x, torch.int32),
                                   t(u, torch.float32), t(q_indptr, torch.int32), mk,
                                   workspace=ws)
        torch.cuda.synchronize()
        check_accept(p, q, x, u, q_indptr, acc.cpu().numpy(), tok.cpu().numpy())
    with pytest.raises(nsd.NsdError):
        nsd.spec_accept(t(p, torch.float32), t(q, torch.float32), t(x, torch.int32),
                        t(u, torch.float32), t(q_indptr, torch.int32), mk, workspace=ws[:64])


def test_first_token_follows_target_row(device):
    # speculative-sampling theorem on the GPU: 200k requests share (p_0, q_0)
    from scipy import stats
    rng = np.random.default_rng(3)
    vocab, bs = 8, 200000
    p0 = _probs(rng, 1, vocab, 1.0)[0]
    q0 = _probs(rng, 1, vocab, 1.0)[0]
    p1 = _probs(rng, 1, vocab, 1.0)[0]
    q_indptr, tq, _ = _batch([1] * bs)
    p = np.tile(np.stack([p0, p1]), (bs, 1))
    q = np.tile(q0[None], (bs, 1))
    qq = q0.astype(np.float64)
    x = rng.choice(vocab, size=bs, p=qq / qq.sum()).astype(np.int32)
    u = (rng.integers(0, 1 << 24, tq) * 2.0**-24).astype(np.float32)
    acc, tok = _accept(device, p, q, x, u, q_indptr, 1)
    counts = np.bincount(tok[q_indptr[:-1]], minlength=vocab)
    r64 = p0.astype(np.float64)
    assert stats.chisquare(counts, r64 / r64.sum() * bs).pvalue > 1e-4
    check_accept(p, q, x, u, q_indptr, acc, tok, requests=range(0, bs, 97))


@pytest.mark.parametrize("bs", [FUSED_MIN_BATCH - 1, FUSED_MIN_BATCH])
def test_auto_preparation_both_sides_of_the_threshold(device, bs):
    # verify_round's default preparation: below FUSED_MIN_BATCH requests the
    # separate gather, from it on the fused pass; both against the oracle
    cfg = custom_config(seed=70 + bs, bs=bs, num_q_heads=32, num_kv_heads=8, head_dim=128,
                        ctx_lo=200, ctx_hi=1500, k_lo=4, k_hi=4, n_arriving=bs // 3,
                        vocab=1000, pool_blocks=None)
    meta = make_meta(cfg)
    _check_all(cfg, meta, device, prepare="auto")


def test_fused_without_query_rows_still_prepares(device):
    # q_indptr all zero (no query rows): the fused call has nothing to attend,
    # but it still moves the arriving requests' blocks into the pool, as the
    # separate gather does
    cfg = custom_config(seed=75, bs=7, n_arriving=3, pool_blocks=None, vocab=0)
    meta = make_meta(cfg)
    lay = make_layer(cfg, meta, 0, "cpu")
    kp, vp = lay.k_pool.to(device), lay.v_pool.to(device)
    # one row of q and out (an empty tensor has no address); none is read or written
    q0 = torch.zeros((1, cfg.num_q_heads, cfg.head_dim), dtype=torch.bfloat16, device=device)
    qi = torch.zeros(cfg.bs + 1, dtype=torch.int32, device=device)
    out = nsd.gather_verify_attention(q0, kp, vp, lay.k_stage.to(device), lay.v_stage.to(device),
                                      i32(meta.block_table, device),
                                      i32(meta.stage_table, device), i32(meta.seq_lens, device),
                                      qi, meta.max_q, meta.max_seq_len)
    torch.cuda.synchronize()
    ref_k, ref_v = oracle.gather.kv_gather(u16(lay.k_stage)[None], u16(lay.v_stage)[None],
                                           u16(lay.k_pool)[None], u16(lay.v_pool)[None],
                                           meta.src_ids, meta.dst_ids)
    assert np.array_equal(u16(kp), ref_k[0]) and np.array_equal(u16(vp), ref_v[0])
