"""Seeded generation of one verification round's inputs.

Scalars (context lengths, proposal depths, the arriving set, block
permutations) come from numpy PCG64 streams keyed by (seed, stream).  Bulk
tensors come from torch generators keyed by (seed, stream, layer) on the device
that will hold them, so a workload is reproducible on any host for a given
device type.  Everything here is input drawing and byte layout; none of it
gathers, attends or accepts.

Input recipe (the distributions named for each workload):
* L_r integer-uniform in [ctx_lo, ctx_hi]; K_r integer-uniform in [k_lo, k_hi].
* Query/key/value elements N(0, 1) in fp32, rounded to bf16 (round to nearest
  even).
* Target and draft rows: softmax of N(0, 2^2) logits computed in fp64, then
  rounded to fp32 (not renormalised).
* Draft token i of a request is drawn from its draft row by the Gumbel-max rule
  on the fp64 draft logits.
* Uniforms are fp32 values on the 2^-24 grid in [0, 1).
* Exactly n_arriving requests arrive, chosen by a seeded permutation.  Their
  KV sits in a staging pool (per-request contiguous extents, the HostKV
  arrangement of Appendix E.1, or a shuffled arrangement) and their blocks in the
  worker pool hold NaN until gathered.
* Physical block ids of the worker pool are a seeded permutation of
  [0, num_blocks).  Slots past L_r in a request's last block hold NaN.  Pool
  blocks owned by no request keep random values (a canary for the gather).
"""
from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

from .configs import RoundConfig
from .layout import BLOCK_SIZE, k_block_shape, v_block_shape, logical_kv_from_blocks

# stream ids
S_CTX, S_ARRIVE, S_POOL_PERM, S_STAGE_PERM, S_DEPTH = 1, 2, 3, 4, 5
S_Q, S_K, S_V, S_P_LOGITS, S_Q_LOGITS, S_GUMBEL, S_UNIFORM = 6, 7, 8, 9, 10, 11, 12
S_K_STAGE, S_V_STAGE = 13, 14
S_DRAFT_Q, S_DRAFT_K, S_DRAFT_V, S_DRAFT_LOGITS, S_DRAFT_U = 15, 16, 17, 18, 19

_CHUNK = 1 << 26


def _np_rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream])))


def _torch_gen(seed: int, stream: int, layer: int, device) -> torch.Generator:
    s = np.random.SeedSequence([seed, stream, layer]).generate_state(1, dtype=np.uint64)[0]
    g = torch.Generator(device=device)
    g.manual_seed(int(s) & ((1 << 63) - 1))
    return g


@dataclass
class RoundMeta:
    cfg: RoundConfig
    seq_lens: np.ndarray        # int32 [bs], L_r including the query window
    depth: np.ndarray           # int32 [bs], K_r
    q_indptr: np.ndarray        # int32 [bs+1], n_q[r] = K_r + 1
    block_table: np.ndarray     # int32 [bs][max_blocks_per_seq], -1 past the request's blocks
    arriving: np.ndarray        # bool [bs]
    stage_table: np.ndarray     # int32 [bs][max_blocks_per_seq], staging ids (-1 if resident)
    src_ids: np.ndarray         # int32 [n_pairs], staging block ids
    dst_ids: np.ndarray         # int32 [n_pairs], worker-pool block ids
    num_blocks: int
    stage_num_blocks: int

    @property
    def bs(self): return self.cfg.bs

    @property
    def total_q(self): return int(self.q_indptr[-1])

    @property
    def max_q(self): return int((self.depth + 1).max()) if self.bs else 1

    @property
    def max_seq_len(self): return int(self.seq_lens.max()) if self.bs else 0

    @property
    def max_blocks_per_seq(self): return self.block_table.shape[1]

    @property
    def n_pairs(self): return len(self.src_ids)

    def nblk(self, r: int) -> int:
        return -(-int(self.seq_lens[r]) // BLOCK_SIZE)


def make_meta(cfg: RoundConfig, seq_lens=None, depth=None, arriving=None) -> RoundMeta:
    """Draw the round's scalars; explicit seq_lens/depth/arriving override the draw."""
    bs = cfg.bs
    if seq_lens is None:
        seq_lens = _np_rng(cfg.seed, S_CTX).integers(cfg.ctx_lo, cfg.ctx_hi + 1, size=bs)
    seq_lens = np.asarray(seq_lens, dtype=np.int32)
    if depth is None:
        depth = _np_rng(cfg.seed, S_DEPTH).integers(cfg.k_lo, cfg.k_hi + 1, size=bs)
    depth = np.asarray(depth, dtype=np.int32)
    if np.any(depth + 1 > seq_lens):
        raise ValueError("every request needs L_r >= K_r + 1")
    if arriving is None:
        arr_idx = np.sort(_np_rng(cfg.seed, S_ARRIVE).permutation(bs)[:cfg.n_arriving])
        arriving = np.zeros(bs, dtype=bool)
        arriving[arr_idx] = True
    arriving = np.asarray(arriving, dtype=bool)

    nb = -(-seq_lens.astype(np.int64) // BLOCK_SIZE)
    total = int(nb.sum())
    num_blocks = cfg.pool_blocks if cfg.pool_blocks is not None else total
    if total > num_blocks:
        raise ValueError(f"pool of {num_blocks} blocks cannot hold {total}")
    max_blocks = int(nb.max()) if bs else 1
    perm = _np_rng(cfg.seed, S_POOL_PERM).permutation(num_blocks).astype(np.int32)
    block_table = np.full((bs, max_blocks), -1, dtype=np.int32)
    off = 0
    for r in range(bs):
        block_table[r, :nb[r]] = perm[off:off + nb[r]]
        off += nb[r]

    n_stage = int(nb[arriving].sum())
    stage_ids = np.arange(n_stage, dtype=np.int32)
    if cfg.staging_order == "shuffled":
        stage_ids = _np_rng(cfg.seed, S_STAGE_PERM).permutation(n_stage).astype(np.int32)
    elif cfg.staging_order != "extent":
        raise ValueError(cfg.staging_order)
    stage_table = np.full((bs, max_blocks), -1, dtype=np.int32)
    src, dst = [], []
    off = 0
    for r in np.nonzero(arriving)[0]:
        ids = stage_ids[off:off + nb[r]]
        stage_table[r, :nb[r]] = ids
        src.append(ids)
        dst.append(block_table[r, :nb[r]])
        off += nb[r]
    src_ids = np.concatenate(src).astype(np.int32) if src else np.zeros(0, np.int32)
    dst_ids = np.concatenate(dst).astype(np.int32) if dst else np.zeros(0, np.int32)
    q_indptr = np.zeros(bs + 1, dtype=np.int32)
    q_indptr[1:] = np.cumsum(depth + 1)
    return RoundMeta(cfg, seq_lens, depth, q_indptr, block_table, arriving, stage_table,
                     src_ids, dst_ids, num_blocks, max(n_stage, 0))


@dataclass
class LayerData:
    """One layer's inputs: worker pool before the gather, staging pool, queries."""
    k_pool: torch.Tensor    # bf16 [num_blocks][Hkv][D/8][16][8]
    v_pool: torch.Tensor    # bf16 [num_blocks][Hkv][D][16]
    k_stage: torch.Tensor   # bf16 [stage_blocks][Hkv][D/8][16][8]
    v_stage: torch.Tensor   # bf16 [stage_blocks][Hkv][D][16]
    q: torch.Tensor         # bf16 [total_q][Hq][D]


def _fill_normal(out: torch.Tensor, gen: torch.Generator):
    flat = out.view(-1)
    n = flat.numel()
    for a in range(0, n, _CHUNK):
        b = min(n, a + _CHUNK)
        flat[a:b] = torch.randn(b - a, generator=gen, device=out.device, dtype=torch.float32)


def _poison_tails(k: torch.Tensor, v: torch.Tensor, blocks: np.ndarray, first_slot: np.ndarray):
    for s in range(1, BLOCK_SIZE):
        sel = blocks[first_slot == s]
        if len(sel):
            idx = torch.as_tensor(sel, dtype=torch.long, device=k.device)
            k[idx, :, :, s:, :] = float("nan")
            v[idx, :, :, s:] = float("nan")


def make_layer(cfg: RoundConfig, meta: RoundMeta, layer: int, device) -> LayerData:
    hkv, d = cfg.num_kv_heads, cfg.head_dim
    kshape, vshape = k_block_shape(hkv, d), v_block_shape(hkv, d)
    bf = torch.bfloat16
    k_pool = torch.empty((meta.num_blocks,) + kshape, dtype=bf, device=device)
    v_pool = torch.empty((meta.num_blocks,) + vshape, dtype=bf, device=device)
    k_stage = torch.empty((meta.stage_num_blocks,) + kshape, dtype=bf, device=device)
    v_stage = torch.empty((meta.stage_num_blocks,) + vshape, dtype=bf, device=device)
    q = torch.empty((meta.total_q, cfg.num_q_heads, d), dtype=bf, device=device)
    _fill_normal(k_pool, _torch_gen(cfg.seed, S_K, layer, device))
    _fill_normal(v_pool, _torch_gen(cfg.seed, S_V, layer, device))
    _fill_normal(k_stage, _torch_gen(cfg.seed, S_K_STAGE, layer, device))
    _fill_normal(v_stage, _torch_gen(cfg.seed, S_V_STAGE, layer, device))
    _fill_normal(q, _torch_gen(cfg.seed, S_Q, layer, device))

    # Arriving requests' worker-pool blocks are not valid until gathered.
    if meta.n_pairs:
        idx = torch.as_tensor(meta.dst_ids, dtype=torch.long, device=device)
        k_pool[idx] = float("nan")
        v_pool[idx] = float("nan")
    # Slots past L_r in each request's last block.
    last_slot = meta.seq_lens % BLOCK_SIZE
    tails = np.nonzero(last_slot)[0]
    res = tails[~meta.arriving[tails]]
    arr = tails[meta.arriving[tails]]
    nblk = -(-meta.seq_lens // BLOCK_SIZE)
    if len(res):
        _poison_tails(k_pool, v_pool, meta.block_table[res, nblk[res] - 1], last_slot[res])
    if len(arr):
        _poison_tails(k_stage, v_stage, meta.stage_table[arr, nblk[arr] - 1], last_slot[arr])
    return LayerData(k_pool, v_pool, k_stage, v_stage, q)


def logical_kv(meta: RoundMeta, layer: LayerData, r: int):
    """Request r's logical K/V [L_r][Hkv][D] as drawn (before any gather).

    Arriving requests are read from the staging pool, resident ones from the
    worker pool.
    """
    nb = meta.nblk(r)
    if meta.arriving[r]:
        ids = torch.as_tensor(meta.stage_table[r, :nb], dtype=torch.long, device=layer.k_stage.device)
        kb, vb = layer.k_stage[ids], layer.v_stage[ids]
    else:
        ids = torch.as_tensor(meta.block_table[r, :nb], dtype=torch.long, device=layer.k_pool.device)
        kb, vb = layer.k_pool[ids], layer.v_pool[ids]
    return logical_kv_from_blocks(kb, vb, int(meta.seq_lens[r]))


@dataclass
class AcceptData:
    p_target: torch.Tensor      # fp32 [total_q][V]: target rows, request r at q_indptr[r] + i
    q_draft: torch.Tensor       # fp32 [total_q - bs][V]: draft rows, request r at q_indptr[r] - r + i
    draft_tokens: torch.Tensor  # int32 [total_q - bs]
    uniforms: torch.Tensor      # fp32 [total_q]: K_r acceptance uniforms, then 1 sampling uniform


def _softmax_rows(out: torch.Tensor, gen: torch.Generator, sigma: float, gumbel_gen=None):
    """Fill out[rows][V] with fp32(softmax_fp64(N(0, sigma^2))); optionally draw one
    Gumbel-max token per row from the same fp64 logits."""
    rows, vocab = out.shape
    tokens = torch.empty(rows, dtype=torch.int32, device=out.device)
    step = max(1, (1 << 24) // max(vocab, 1))
    for a in range(0, rows, step):
        b = min(rows, a + step)
        z = sigma * torch.randn((b - a, vocab), generator=gen, device=out.device,
                                dtype=torch.float64)
        out[a:b] = torch.softmax(z, dim=1).to(torch.float32)
        if gumbel_gen is not None:
            u = torch.rand((b - a, vocab), generator=gumbel_gen, device=out.device,
                           dtype=torch.float64)
            tokens[a:b] = torch.argmax(z - torch.log(-torch.log(u)), dim=1).to(torch.int32)
    return tokens


def make_accept(cfg: RoundConfig, meta: RoundMeta, device) -> Optional[AcceptData]:
    if cfg.vocab == 0:
        return None
    nq, nd = meta.total_q, meta.total_q - meta.bs
    p = torch.empty((nq, cfg.vocab), dtype=torch.float32, device=device)
    qd = torch.empty((nd, cfg.vocab), dtype=torch.float32, device=device)
    _softmax_rows(p, _torch_gen(cfg.seed, S_P_LOGITS, 0, device), 2.0)
    tok = _softmax_rows(qd, _torch_gen(cfg.seed, S_Q_LOGITS, 0, device), 2.0,
                        gumbel_gen=_torch_gen(cfg.seed, S_GUMBEL, 0, device))
    ug = _torch_gen(cfg.seed, S_UNIFORM, 0, device)
    u = torch.randint(0, 1 << 24, (nq,), generator=ug, device=device, dtype=torch.int64)
    u = u.to(torch.float32) * (2.0 ** -24)
    return AcceptData(p, qd, tok, u)


@dataclass
class HostKV:
    """A pinned host KV arena for one layer (every request at a stable extent).

    Request r owns blocks [extent[r], extent[r] + capacity[r]) of each plane;
    its first ceil(L_r/16) blocks hold its logical KV (the staged blocks if it is
    arriving, its pool blocks if resident), the rest is reserved headroom."""
    k: torch.Tensor            # bf16 [arena_blocks][Hkv][D/8][16][8], pinned
    v: torch.Tensor            # bf16 [arena_blocks][Hkv][D][16], pinned
    extent: np.ndarray         # int64 [bs], first arena block of request r
    capacity: np.ndarray       # int64 [bs], blocks reserved for request r


def make_hostkv(cfg: RoundConfig, meta: RoundMeta, layer: LayerData, headroom_tokens: int = 64,
                seed_stream: int = 97, pin: bool = True) -> HostKV:
    """Host arena holding the round's KV the way HostKV keeps it: extents sized
    for the tokens so far plus generation headroom (Eq. E.1), laid out in a seeded
    order; the bytes come from the layer's staging pool and worker pool.  pin=False
    (no GPU present) gives the same arena in pageable memory."""
    nblk = -(-meta.seq_lens.astype(np.int64) // BLOCK_SIZE)
    cap = -(-(meta.seq_lens.astype(np.int64) + headroom_tokens) // BLOCK_SIZE)
    order = _np_rng(cfg.seed, seed_stream).permutation(meta.bs)
    extent = np.zeros(meta.bs, dtype=np.int64)
    off = 0
    for r in order:
        extent[r] = off
        off += int(cap[r])
    kshape, vshape = tuple(layer.k_pool.shape[1:]), tuple(layer.v_pool.shape[1:])
    hk = torch.zeros((off,) + kshape, dtype=torch.bfloat16, pin_memory=pin)
    hv = torch.zeros((off,) + vshape, dtype=torch.bfloat16, pin_memory=pin)
    src_k, src_v = layer.k_pool.cpu(), layer.v_pool.cpu()
    stg_k, stg_v = layer.k_stage.cpu(), layer.v_stage.cpu()
    for r in range(meta.bs):
        n = int(nblk[r])
        if meta.arriving[r]:
            ids = torch.as_tensor(meta.stage_table[r, :n], dtype=torch.long)
            hk[extent[r]:extent[r] + n] = stg_k[ids]
            hv[extent[r]:extent[r] + n] = stg_v[ids]
        else:
            ids = torch.as_tensor(meta.block_table[r, :n], dtype=torch.long)
            hk[extent[r]:extent[r] + n] = src_k[ids]
            hv[extent[r]:extent[r] + n] = src_v[ids]
    return HostKV(hk, hv, extent, cap)


@dataclass
class DraftData:
    """Inputs of a K-step draft stage over one layer.

    Request r enters with P_r = L_r - 1 tokens in its cache (L_r drawn as for a
    round, the anchor included); step i processes the token at position P_r + i.
    The block tables cover the last step's length P_r + K, and every slot at or
    past P_r holds NaN until a step appends it."""
    meta: RoundMeta             # seq_lens = P_r + K (tables sized for the last step), one query each
    layer: LayerData            # pools and staging planes (layer.q is not used)
    lens: torch.Tensor          # int32 [K][bs], step i's length P_r + i + 1
    q: torch.Tensor             # bf16 [K][bs][Hq][D]
    k_new: torch.Tensor         # bf16 [K][bs][Hkv][D]
    v_new: torch.Tensor         # bf16 [K][bs][Hkv][D]
    probs: torch.Tensor         # fp32 [bs][K][V], draft row of step i at [r][i]
    uniforms: torch.Tensor      # fp32 [K][bs]

    @property
    def steps(self): return self.lens.shape[0]

    @property
    def prefix(self): return self.meta.seq_lens - self.steps   # P_r


def _poison_positions(k, v, table, rows, pos):
    """NaN into slot pos % 16 of block table[row][pos // 16] for each (row, pos)."""
    if len(rows) == 0:
        return
    blk = torch.as_tensor(table[rows, pos // BLOCK_SIZE], dtype=torch.long, device=k.device)
    slot = torch.as_tensor(pos % BLOCK_SIZE, dtype=torch.long, device=k.device)
    k[blk, :, :, slot, :] = float("nan")
    v[blk, :, :, slot] = float("nan")


def make_draft(cfg: RoundConfig, steps: int, vocab: int, device) -> DraftData:
    """Draw a draft stage of ``steps`` proposals per request: contexts, the
    arriving set and block layout as for a round of ``cfg`` (one query per
    request), per-step queries and new K/V rows N(0, 1) in bf16, draft rows
    fp32(softmax_fp64(N(0, 2^2))) over ``vocab`` tokens, uniforms on the 2^-24
    grid."""
    if steps < 1:
        raise ValueError("a draft stage has at least one step")
    L = _np_rng(cfg.seed, S_CTX).integers(cfg.ctx_lo, cfg.ctx_hi + 1, size=cfg.bs)
    meta = make_meta(cfg, seq_lens=L - 1 + steps, depth=np.zeros(cfg.bs, dtype=np.int32))
    layer = make_layer(cfg, meta, 0, device)
    # the cache holds P_r tokens; the positions the steps append are not there yet
    prefix = meta.seq_lens - steps
    rows = np.repeat(np.arange(cfg.bs), steps)
    pos = (prefix[rows] + np.tile(np.arange(steps), cfg.bs)).astype(np.int64)
    arr = meta.arriving[rows]
    _poison_positions(layer.k_pool, layer.v_pool, meta.block_table, rows[~arr], pos[~arr])
    _poison_positions(layer.k_stage, layer.v_stage, meta.stage_table, rows[arr], pos[arr])
    lens = torch.as_tensor((prefix[None, :] + 1 + np.arange(steps)[:, None]).astype(np.int32),
                           device=device)
    bf = torch.bfloat16
    hq, hkv, d = cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim
    q = torch.empty((steps, cfg.bs, hq, d), dtype=bf, device=device)
    kn = torch.empty((steps, cfg.bs, hkv, d), dtype=bf, device=device)
    vn = torch.empty((steps, cfg.bs, hkv, d), dtype=bf, device=device)
    _fill_normal(q, _torch_gen(cfg.seed, S_DRAFT_Q, 0, device))
    _fill_normal(kn, _torch_gen(cfg.seed, S_DRAFT_K, 0, device))
    _fill_normal(vn, _torch_gen(cfg.seed, S_DRAFT_V, 0, device))
    probs = torch.empty((cfg.bs, steps, vocab), dtype=torch.float32, device=device)
    _softmax_rows(probs.view(-1, vocab), _torch_gen(cfg.seed, S_DRAFT_LOGITS, 0, device), 2.0)
    ug = _torch_gen(cfg.seed, S_DRAFT_U, 0, device)
    u = torch.randint(0, 1 << 24, (steps, cfg.bs), generator=ug, device=device, dtype=torch.int64)
    return DraftData(meta, layer, lens, q, kn, vn, probs, u.to(torch.float32) * (2.0 ** -24))
