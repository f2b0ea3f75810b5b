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

from . import copy_plan, DEFAULT_CHUNK, lib, _check

BLOCK = 16


def h2d_plan(extent, stage_table, arriving, seq_lens, block_bytes):
    """Byte-level copy plan [n][3] (host offset, bank offset, bytes) of one plane:
    block j of arriving request r goes from arena block extent[r] + j to bank block
    stage_table[r][j].  Blocks are listed request by request, so a request whose
    staging ids are consecutive becomes one run after merging (nsd_h2d_plan)."""
    import ctypes
    extent = np.ascontiguousarray(extent, dtype=np.int64)
    st = np.ascontiguousarray(stage_table, dtype=np.int32)
    arr = np.ascontiguousarray(arriving, dtype=np.uint8)
    sl = np.ascontiguousarray(seq_lens, dtype=np.int32)
    bs = len(sl)
    cap = int(np.sum(-(-sl[arr.astype(bool)].astype(np.int64) // BLOCK))) if bs else 0
    out = np.zeros((max(cap, 1), 3), dtype=np.int64)
    n = ctypes.c_int64()
    p = lambda a: a.ctypes.data if a.size else None
    _check("h2d_plan", lib().nsd_h2d_plan(p(extent), p(st), max(1, st.shape[1] if st.ndim == 2 else 1),
                                          p(arr), p(sl), bs, int(block_bytes), out.ctypes.data, cap,
                                          ctypes.byref(n)))
    return out[:n.value].copy()


def writeback_pairs(block_table, extent, host_len, new_len):
    """(pool block id, arena block id) int32 pairs of the suffix each request writes
    back: the blocks holding its tokens host_len .. new_len - 1 (Section 5:
    incremental writeback of the valid suffix; Appendix E.1 extents), by
    nsd_writeback_pairs."""
    import ctypes
    bt = np.ascontiguousarray(block_table, dtype=np.int32)
    extent = np.ascontiguousarray(extent, dtype=np.int64)
    h = np.ascontiguousarray(host_len, dtype=np.int32)
    l = np.ascontiguousarray(new_len, dtype=np.int32)
    bs = len(l)
    grow = l.astype(np.int64) > h
    cap = int(np.sum((l[grow].astype(np.int64) - 1) // BLOCK - h[grow] // BLOCK + 1)) if bs else 0
    src = np.zeros(max(cap, 1), dtype=np.int32)
    dst = np.zeros(max(cap, 1), dtype=np.int32)
    n = ctypes.c_int64()
    p = lambda a: a.ctypes.data if a.size else None
    _check("writeback_pairs", lib().nsd_writeback_pairs(
        p(bt), max(1, bt.shape[1] if bt.ndim == 2 else 1), p(extent), p(h), p(l), bs,
        src.ctypes.data, dst.ctypes.data, cap, ctypes.byref(n)))
    return src[:n.value].copy(), dst[:n.value].copy()


class DoubleBank:
    """Two device staging banks filled from pinned host planes by a DMA stream,
    with the bank lifecycle of Eq. E.2:

        Free -> Filling -> Ready -> Computing -> Exporting -> Free

    prepare(i, ...) fills bank i % 2 (Filling) once that bank is Free again: the
    round that last computed on it has finished and its export has completed.
    With ``window_bytes`` the plan is submitted in bounded groups (Appendix
    E.5) by a DMA thread that waits for each group before submitting the next;
    otherwise every chunk is queued at once.  ready(i) is the KVReady event of
    bank i % 2 (it returns once the submission has been queued, then the event
    marks its completion).  After a round computed on bank i % 2 on `stream`,
    export(i, stream, fn) runs the round's writeback ``fn(d2h_stream)`` on the
    D2H stream once the round is done (Exporting), and the bank becomes Free
    when the export completes; done(i, stream) releases a bank with nothing to
    export.  Background transfers therefore never overwrite a bank an active
    round still reads, and a round's export overlaps the next round's compute
    (Eq. E.3: Compute_{k+1} || D2H_k, Compute_k || H2D_{k+1})."""

    def __init__(self, k_shape, v_shape, device, copy_stream=None, d2h_stream=None):
        self.k = [torch.empty(k_shape, dtype=torch.bfloat16, device=device) for _ in range(2)]
        self.v = [torch.empty(v_shape, dtype=torch.bfloat16, device=device) for _ in range(2)]
        self.copy_stream = copy_stream or torch.cuda.Stream(device)
        self.d2h_stream = d2h_stream or torch.cuda.Stream(device)
        self.device = device
        self._free = [None, None]
        self._ready = [None, None]
        self._thread = [None, None]
        self.state = ["Free", "Free"]

    def _fill(self, b, host_k, host_v, plan_k, plan_v, chunk_bytes, window_bytes):
        s = self.copy_stream
        if self._free[b] is not None:
            s.wait_event(self._free[b])
        copy_plan(host_k, self.k[b], plan_k, chunk_bytes, stream=s, window_bytes=window_bytes)
        copy_plan(host_v, self.v[b], plan_v, chunk_bytes, stream=s, window_bytes=window_bytes)
        ev = torch.cuda.Event(enable_timing=True)
        ev.record(s)
        self._ready[b] = ev

    def prepare(self, i, host_k, host_v, plan_k, plan_v, chunk_bytes=DEFAULT_CHUNK,
                window_bytes=None):
        b = i % 2
        self.wait_submitted(i)
        self.state[b] = "Filling"
        if window_bytes is None:
            self._fill(b, host_k, host_v, plan_k, plan_v, chunk_bytes, None)
            self.state[b] = "Ready"
            return self._ready[b]
        import threading

        def run():
            torch.cuda.set_device(self.device)
            self._fill(b, host_k, host_v, plan_k, plan_v, chunk_bytes, window_bytes)
        self._ready[b] = None
        t = threading.Thread(target=run, daemon=True)
        self._thread[b] = t
        t.start()
        return None

    def wait_submitted(self, i):
        """Block until the DMA thread (if any) has submitted bank i % 2's plan."""
        b = i % 2
        t = self._thread[b]
        if t is not None:
            t.join()
            self._thread[b] = None
            self.state[b] = "Ready"

    def ready(self, i):
        self.wait_submitted(i)
        return self._ready[i % 2]

    def computing(self, i, stream):
        """Make `stream` wait for bank i % 2 to be Ready (KVReady) and mark it Computing."""
        stream.wait_event(self.ready(i))
        self.state[i % 2] = "Computing"

    def export(self, i, stream, fn):
        """Exporting: run fn(d2h_stream) once the round on `stream` is done; the bank is
        Free once it completes.  Returns the completion event."""
        b = i % 2
        done = torch.cuda.Event(enable_timing=True)
        done.record(stream)
        self.d2h_stream.wait_event(done)
        self.state[b] = "Exporting"
        with torch.cuda.stream(self.d2h_stream):
            fn(self.d2h_stream)
        ev = torch.cuda.Event(enable_timing=True)
        ev.record(self.d2h_stream)
        self._free[b] = ev
        return ev

    def done(self, i, stream):
        ev = torch.cuda.Event()
        ev.record(stream)
        self._free[i % 2] = ev
        self.state[i % 2] = "Free"
        return ev

    def bank(self, i):
        return self.k[i % 2], self.v[i % 2]
