"""KV-state preparation from a host arena into double-buffered device banks.

Passage: Algorithm 1 (Prepare(B, w) makes the batch's KV state resident on the
worker before Run); Appendix E.1 (HostKV: persistent pinned host arenas, each
request at a stable extent, Eq. E.1); Appendix E.2 (two device KV banks per
worker: while one serves the current batch, the other is filled for the next,
Eq. E.3: Compute_k || H2D_{k+1}); Appendix E.5 (H2D plans in bounded chunks).

A round's plan copies each arriving request's blocks from its HostKV extent to
the staging ids its stage table names, in a device bank; the bank is then the
staging pool of nsd_gather_verify_attention (or nsd_kv_gather), which moves
the blocks into the paged pool as it first reads them.  The copies run on the
DMA engines (nsd_copy_plan), on a stream of their own.
"""
import numpy as np
import torch

from . import copy_plan, DEFAULT_CHUNK

BLOCK = 16


def h2d_plan(extent, stage_table, arriving, seq_lens, block_bytes):
    """Byte-level copy plan [n][3] (host offset, bank offset, bytes) of one plane:
    block j of arriving request r goes from arena block extent[r] + j to bank block
    stage_table[r][j].  Blocks are listed request by request, so a request whose
    staging ids are consecutive becomes one run after merging."""
    rows = []
    for r in np.nonzero(np.asarray(arriving))[0]:
        n = -(-int(seq_lens[r]) // BLOCK)
        j = np.arange(n, dtype=np.int64)
        src = (int(extent[r]) + j) * block_bytes
        dst = np.asarray(stage_table[r, :n], dtype=np.int64) * block_bytes
        rows.append(np.stack([src, dst, np.full(n, block_bytes, dtype=np.int64)], axis=1))
    if not rows:
        return np.zeros((0, 3), dtype=np.int64)
    return np.concatenate(rows)


class DoubleBank:
    """Two device staging banks filled from pinned host planes on a copy stream.

    prepare(i, ...) fills bank i % 2 once the round that last used that bank has
    finished with it (Eq. E.2 lifecycle: Free -> Filling -> Ready); ready(i) is
    the event a round waits on before reading bank i % 2 (KVReady); done(i, stream)
    marks bank i % 2 free again once the round on `stream` has read it."""

    def __init__(self, k_shape, v_shape, device, copy_stream=None):
        self.k = [torch.empty(k_shape, dtype=torch.bfloat16, device=device) for _ in range(2)]
        self.v = [torch.empty(v_shape, dtype=torch.bfloat16, device=device) for _ in range(2)]
        self.copy_stream = copy_stream or torch.cuda.Stream(device)
        self._free = [None, None]
        self._ready = [None, None]

    def prepare(self, i, host_k, host_v, plan_k, plan_v, chunk_bytes=DEFAULT_CHUNK):
        b = i % 2
        s = self.copy_stream
        if self._free[b] is not None:
            s.wait_event(self._free[b])
        copy_plan(host_k, self.k[b], plan_k, chunk_bytes, stream=s)
        copy_plan(host_v, self.v[b], plan_v, chunk_bytes, stream=s)
        ev = torch.cuda.Event(enable_timing=True)
        ev.record(s)
        self._ready[b] = ev
        return ev

    def ready(self, i):
        return self._ready[i % 2]

    def done(self, i, stream):
        ev = torch.cuda.Event()
        ev.record(stream)
        self._free[i % 2] = ev
        return ev

    def bank(self, i):
        return self.k[i % 2], self.v[i % 2]


def writeback_pairs(block_table, extent, host_len, new_len):
    """(pool block id, arena block id) int32 pairs of the suffix each request writes
    back: the blocks holding its tokens host_len .. new_len - 1 (Section 5:
    incremental writeback of the valid suffix; Appendix E.1 extents)."""
    host_len = np.asarray(host_len, dtype=np.int64)
    new_len = np.asarray(new_len, dtype=np.int64)
    src, dst = [], []
    for r in np.nonzero(new_len > host_len)[0]:
        j = np.arange(host_len[r] // BLOCK, (new_len[r] - 1) // BLOCK + 1)
        src.append(np.asarray(block_table[r, j], dtype=np.int64))
        dst.append(int(extent[r]) + j)
    if not src:
        return np.zeros(0, np.int32), np.zeros(0, np.int32)
    return np.concatenate(src).astype(np.int32), np.concatenate(dst).astype(np.int32)
