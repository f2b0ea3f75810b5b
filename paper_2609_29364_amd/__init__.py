"""Python binding of libnebulasd, the MI355X verification-round library.

Thin argument marshalling over the C ABI declared in ``include/nebulasd.h``:
torch tensors are checked (dtype, device, contiguity, shapes) and passed as
raw device pointers together with torch's current HIP stream.  Every step of
the round runs in the library's HIP kernels; there is no fallback, and a
missing library raises at the first call.
"""
import ctypes
import math
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libnebulasd.so")
BLOCK_SIZE = 16

STATUS_NAMES = {0: "NSD_OK", 1: "NSD_ERR_NULL", 2: "NSD_ERR_SHAPE", 3: "NSD_ERR_UNSUPPORTED",
                4: "NSD_ERR_WORKSPACE", 5: "NSD_ERR_HIP"}


class NsdError(RuntimeError):
    def __init__(self, fn, status, message):
        super().__init__(f"{fn}: {STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


_lib = None
_P, _I32, _I64, _F32, _SZ = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                             ctypes.c_size_t)
_SIGS = {
    "nsd_version": (_I32, []),
    "nsd_last_error": (ctypes.c_char_p, []),
    "nsd_kv_gather": (_I32, [_P, _P, _I64, _P, _P, _I64, _P, _P, _I64, _I32, _I32, _I32, _I32,
                             _I32, _I32, _P]),
    "nsd_verify_attention_workspace_size": (_SZ, [_I32, _I32, _I32, _I32, _I32, _I32]),
    "nsd_verify_attention": (_I32, [_P, _P, _P, _I64, _P, _I32, _P, _P, _I32, _I32, _I32, _I32,
                                    _I32, _I32, _I32, _F32, _P, _P, _SZ, _P]),
    "nsd_gather_verify_attention": (_I32, [_P, _P, _P, _I64, _P, _P, _I64, _P, _P, _I32, _P, _P,
                                           _I32, _I32, _I32, _I32, _I32, _I32, _I32, _F32, _P,
                                           _P, _SZ, _P]),
    "nsd_spec_accept_workspace_size": (_SZ, [_I32, _I32]),
    "nsd_spec_accept": (_I32, [_P, _P, _P, _P, _P, _I32, _I32, _I32, _P, _P, _P, _SZ, _P]),
    "nsd_sample": (_I32, [_P, _I64, _P, _I32, _I32, _P, _I32, _P, _SZ, _P]),
    "nsd_reconstruct": (_I32, [_P, _P, _P, _P, _P, _I32, ctypes.c_double, _I64, _I64, _I32,
                               ctypes.c_double, ctypes.c_double, _P, _P, _P]),
    "nsd_simulate": (_I32, [_P, _P, _I32, _P, _I32, _P, _P, _I64, _P, _I64, _P, _P]),
    "nsd_copy_plan": (_I32, [_P, _I64, _P, _I64, _P, _I64, _I64, _I32, _P]),
    "nsd_copy_plan_windowed": (_I32, [_P, _I64, _P, _I64, _P, _I64, _I64, _I64, _I32, _P]),
    "nsd_h2d_plan": (_I32, [_P, _P, _I32, _P, _P, _I32, _I64, _P, _I64, _P]),
    "nsd_writeback_pairs": (_I32, [_P, _I32, _P, _P, _P, _I32, _P, _P, _I64, _P]),
    "nsd_kv_append": (_I32, [_P, _P, _I64, _P, _P, _P, _I32, _P, _P, _I32, _I32, _I32, _I32, _I32,
                             _P]),
    "nsd_commit_lengths": (_I32, [_P, _P, _P, _P, _I32, _P]),
    "nsd_host_alias": (_I32, [_P, ctypes.POINTER(ctypes.c_void_p)]),
    "nsd_spec_accept_static": (_I32, [_P, _P, _P, _P, _P, _I32, _I32, _I32, _P, _P, _P]),
    "nsd_spec_accept_static_max_bytes": (_SZ, []),
    "nsd_set_attention_waves": (_I32, [_I32]),
    "nsd_attention_waves": (_I32, []),
    "nsd_check_plan": (_I32, [_P, _P, _I32, _P, _P, _I32, _I64, _I64, _I32, _I32, _I64]),
    "nsd_check_pairs": (_I32, [_P, _P, _I64, _I64, _I64]),
}


def lib():
    """The loaded library (torch's HIP runtime is loaded first and shared)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run `python -c \"import "
                               f"__graft_entry__ as g; g.build()\"` at the repository root")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(l, name)
            f.restype, f.argtypes = res, args
        _lib = l
    return _lib


def _check(fn, status):
    if status != 0:
        raise NsdError(fn, status, lib().nsd_last_error().decode())


def _ptr(t):
    return None if t is None else t.data_ptr()


def _dev(t, dtype, name):
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on a GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _stream(t):
    return torch.cuda.current_stream(t.device).cuda_stream


def version():
    v = lib().nsd_version()
    return (v >> 16, v & 0xFFFF)


class attention_waves:
    """Context manager: attention calls (and workspace queries) inside it split
    their work over ``waves`` resident waves (a positive multiple of 4) instead
    of the device's count; ``None`` or 0 keeps the device's count.  The setting
    is process-wide (a test and tuning hook)."""

    def __init__(self, waves):
        self.waves = int(waves or 0)

    def __enter__(self):
        self.old = lib().nsd_attention_waves()
        _check("set_attention_waves", lib().nsd_set_attention_waves(self.waves))
        return self

    def __exit__(self, *exc):
        _check("set_attention_waves", lib().nsd_set_attention_waves(self.old))
        return False


def _host_i32(a, name):
    import numpy as np
    if a is None:
        return None
    if isinstance(a, torch.Tensor):
        a = a.cpu().numpy()
    arr = np.ascontiguousarray(a, dtype=np.int32)
    return arr


def check_plan(block_table, seq_lens, q_indptr, num_blocks, max_q_per_seq, max_seq_len,
               stage_table=None, stage_num_blocks=0, total_q=-1):
    """Validate a round's metadata on the host (nsd_check_plan); raises NsdError
    naming the first violation.  Arrays may be numpy arrays or tensors (copied
    to the host)."""
    bt = _host_i32(block_table, "block_table")
    st = _host_i32(stage_table, "stage_table")
    sl = _host_i32(seq_lens, "seq_lens")
    qi = _host_i32(q_indptr, "q_indptr")
    bs = len(sl)
    if bt.ndim != 2 or bt.shape[0] != bs or len(qi) != bs + 1 or \
            (st is not None and st.shape != bt.shape):
        raise ValueError("block_table / stage_table / q_indptr do not match seq_lens")
    _check("check_plan", lib().nsd_check_plan(
        bt.ctypes.data if bs else None, st.ctypes.data if st is not None and bs else None,
        max(1, bt.shape[1]), sl.ctypes.data if bs else None, qi.ctypes.data, bs,
        int(num_blocks), int(stage_num_blocks), int(max_q_per_seq), int(max_seq_len),
        int(total_q)))


def check_pairs(src_ids, dst_ids, src_num_blocks, dst_num_blocks):
    """Validate a gather plan on the host (nsd_check_pairs); raises NsdError."""
    s = _host_i32(src_ids, "src_ids")
    d = _host_i32(dst_ids, "dst_ids")
    if s.shape != d.shape:
        raise ValueError("src_ids and dst_ids differ in length")
    n = len(s)
    _check("check_pairs", lib().nsd_check_pairs(
        s.ctypes.data if n else None, d.ctypes.data if n else None, n, int(src_num_blocks),
        int(dst_num_blocks)))


def kv_gather(src_k, src_v, dst_k, dst_v, src_ids, dst_ids, layer0=0, n_layers=None):
    """Copy whole KV blocks src -> dst for every pair and layer (in place on dst).

    Planes: K [layers][blocks][Hkv][D/8][16][8], V [layers][blocks][Hkv][D][16] bf16
    (a 5-d tensor is taken as a single layer).  src_ids/dst_ids: int32 [n_pairs].
    """
    planes = [src_k, src_v, dst_k, dst_v]
    if src_k.dim() == 5:
        planes = [t.unsqueeze(0) for t in planes]
    sk, sv, dk, dv = planes
    for t, n in zip(planes, ("src_k", "src_v", "dst_k", "dst_v")):
        _dev(t, torch.bfloat16, n)
    _dev(src_ids, torch.int32, "src_ids")
    _dev(dst_ids, torch.int32, "dst_ids")
    num_layers, _, hkv, dv8, bsz, vec = sk.shape
    d = dv8 * vec
    if (sv.shape != (num_layers, sk.shape[1], hkv, d, bsz) or dk.shape[0] != num_layers
            or dk.shape[2:] != sk.shape[2:] or dv.shape != (num_layers, dk.shape[1], hkv, d, bsz)):
        raise ValueError("inconsistent pool shapes")
    if src_ids.numel() != dst_ids.numel():
        raise ValueError("src_ids and dst_ids differ in length")
    if n_layers is None:
        n_layers = num_layers - layer0
    _check("kv_gather", lib().nsd_kv_gather(
        _ptr(sk), _ptr(sv), sk.shape[1], _ptr(dk), _ptr(dv), dk.shape[1], _ptr(src_ids),
        _ptr(dst_ids), src_ids.numel(), num_layers, layer0, n_layers, hkv, bsz, d, _stream(sk)))
    return dst_k, dst_v


def verify_attention_workspace_size(bs, num_q_heads, num_kv_heads, head_dim, max_q_per_seq,
                                    max_seq_len):
    return int(lib().nsd_verify_attention_workspace_size(bs, num_q_heads, num_kv_heads, head_dim,
                                                         max_q_per_seq, max_seq_len))


def new_workspace(nbytes, device):
    """A verify_attention workspace (no initialisation needed), reusable by later calls on
    its stream."""
    return torch.empty(max(int(nbytes), 16), dtype=torch.uint8, device=device)


def _attn_ws(workspace, need, q):
    """The caller's workspace (checked) or a new one of `need` bytes; (tensor, bytes)."""
    if workspace is None:
        workspace = new_workspace(need, q.device) if need else None
    else:
        _dev(workspace, torch.uint8, "workspace")
        if workspace.device != q.device:
            raise ValueError("workspace must be on q's device")
    return workspace, (0 if workspace is None else workspace.numel())


def verify_attention(q, k_cache, v_cache, block_table, seq_lens, q_indptr, max_q_per_seq,
                     max_seq_len, scale=None, out=None, workspace=None):
    """One layer of verification attention; returns out [total_q][Hq][D] bf16.

    k_cache [blocks][Hkv][D/8][16][8], v_cache [blocks][Hkv][D][16] bf16;
    block_table int32 [bs][max_blocks]; seq_lens int32 [bs]; q_indptr int32 [bs+1].
    max_q_per_seq / max_seq_len are host-side bounds of n_q and L_r.
    """
    _dev(q, torch.bfloat16, "q")
    _dev(k_cache, torch.bfloat16, "k_cache")
    _dev(v_cache, torch.bfloat16, "v_cache")
    for t, n in ((block_table, "block_table"), (seq_lens, "seq_lens"), (q_indptr, "q_indptr")):
        _dev(t, torch.int32, n)
    total_q, hq, d = q.shape
    nb, hkv, dv8, bsz, vec = k_cache.shape
    if dv8 * vec != d or v_cache.shape != (nb, hkv, d, bsz):
        raise ValueError("cache shapes do not match q")
    bs = seq_lens.numel()
    if block_table.dim() != 2 or block_table.shape[0] != bs or q_indptr.numel() != bs + 1:
        raise ValueError("block_table / q_indptr do not match seq_lens")
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if out is None:
        out = torch.empty_like(q)
    else:
        _dev(out, torch.bfloat16, "out")
        if out.shape != q.shape:
            raise ValueError("out must have q's shape")
    need = verify_attention_workspace_size(bs, hq, hkv, d, max_q_per_seq, max_seq_len)
    workspace, ws_bytes = _attn_ws(workspace, need, q)
    _check("verify_attention", lib().nsd_verify_attention(
        _ptr(q), _ptr(k_cache), _ptr(v_cache), nb, _ptr(block_table), block_table.shape[1],
        _ptr(seq_lens), _ptr(q_indptr), bs, hq, hkv, d, bsz, max_q_per_seq, max_seq_len,
        float(scale), _ptr(out), _ptr(workspace), ws_bytes, _stream(q)))
    return out


def gather_verify_attention(q, k_cache, v_cache, k_stage, v_stage, block_table, stage_table,
                            seq_lens, q_indptr, max_q_per_seq, max_seq_len, scale=None, out=None,
                            workspace=None):
    """KV-state preparation fused with one layer of verification attention.

    Arriving requests (stage_table[r][0] >= 0) read their blocks from the
    staging planes and leave them in k_cache/v_cache at block_table[r][b];
    returns out [total_q][Hq][D] bf16.
    """
    for t, n in ((q, "q"), (k_cache, "k_cache"), (v_cache, "v_cache"), (k_stage, "k_stage"),
                 (v_stage, "v_stage")):
        _dev(t, torch.bfloat16, n)
    for t, n in ((block_table, "block_table"), (stage_table, "stage_table"),
                 (seq_lens, "seq_lens"), (q_indptr, "q_indptr")):
        _dev(t, torch.int32, n)
    total_q, hq, d = q.shape
    nb, hkv, dv8, bsz, vec = k_cache.shape
    if dv8 * vec != d or v_cache.shape != (nb, hkv, d, bsz):
        raise ValueError("cache shapes do not match q")
    if k_stage.shape[1:] != k_cache.shape[1:] or v_stage.shape[1:] != v_cache.shape[1:] \
            or k_stage.shape[0] != v_stage.shape[0]:
        raise ValueError("staging planes do not match the caches")
    bs = seq_lens.numel()
    if block_table.dim() != 2 or block_table.shape[0] != bs or q_indptr.numel() != bs + 1 \
            or stage_table.shape != block_table.shape:
        raise ValueError("block_table / stage_table / q_indptr do not match seq_lens")
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if out is None:
        out = torch.empty_like(q)
    else:
        _dev(out, torch.bfloat16, "out")
        if out.shape != q.shape:
            raise ValueError("out must have q's shape")
    need = verify_attention_workspace_size(bs, hq, hkv, d, max_q_per_seq, max_seq_len)
    workspace, ws_bytes = _attn_ws(workspace, need, q)
    _check("gather_verify_attention", lib().nsd_gather_verify_attention(
        _ptr(q), _ptr(k_cache), _ptr(v_cache), nb, _ptr(k_stage), _ptr(v_stage),
        k_stage.shape[0], _ptr(block_table), _ptr(stage_table), block_table.shape[1],
        _ptr(seq_lens), _ptr(q_indptr), bs, hq, hkv, d, bsz, max_q_per_seq, max_seq_len,
        float(scale), _ptr(out), _ptr(workspace), ws_bytes, _stream(q)))
    return out


def accept_workspace_size(rows, vocab):
    """Bytes of workspace spec_accept (rows = bs) or sample (rows = n_rows) needs."""
    return lib().nsd_spec_accept_workspace_size(rows, vocab)


def _accept_ws(workspace, rows, vocab, device):
    need = accept_workspace_size(rows, vocab)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=device)
    _dev(workspace, torch.uint8, "workspace")
    if workspace.device != device:
        raise ValueError("workspace must be on the probabilities' device")
    return workspace, workspace.numel()


def spec_accept(p_target, q_draft, draft_tokens, uniforms, q_indptr, max_k, accepted_len=None,
                out_tokens=None, workspace=None):
    """Acceptance + residual resampling; returns (accepted_len [bs], out_tokens [total_q]) int32.

    workspace: a GPU tensor of at least accept_workspace_size(bs, vocab) bytes
    (allocated per call when None)."""
    _dev(p_target, torch.float32, "p_target")
    _dev(uniforms, torch.float32, "uniforms")
    _dev(q_indptr, torch.int32, "q_indptr")
    if max_k > 0:
        _dev(q_draft, torch.float32, "q_draft")
        _dev(draft_tokens, torch.int32, "draft_tokens")
    total_q, vocab = p_target.shape
    bs = q_indptr.numel() - 1
    if uniforms.numel() != total_q:
        raise ValueError("uniforms must have one entry per target row")
    if max_k > 0 and (q_draft.shape != (total_q - bs, vocab) or draft_tokens.numel() != total_q - bs):
        raise ValueError("q_draft / draft_tokens must have total_q - bs rows")
    if accepted_len is None:
        accepted_len = torch.empty(bs, dtype=torch.int32, device=p_target.device)
    if out_tokens is None:
        out_tokens = torch.empty(total_q, dtype=torch.int32, device=p_target.device)
    _dev(accepted_len, torch.int32, "accepted_len")
    _dev(out_tokens, torch.int32, "out_tokens")
    if accepted_len.numel() != bs or out_tokens.numel() != total_q:
        raise ValueError("accepted_len must have bs entries and out_tokens total_q")
    ws, ws_n = _accept_ws(workspace, bs, vocab, p_target.device)
    _check("spec_accept", lib().nsd_spec_accept(
        _ptr(p_target), _ptr(q_draft) if max_k > 0 else None,
        _ptr(draft_tokens) if max_k > 0 else None, _ptr(uniforms), _ptr(q_indptr), bs, vocab,
        max_k, _ptr(accepted_len), _ptr(out_tokens), _ptr(ws), ws_n, _stream(p_target)))
    return accepted_len, out_tokens


def spec_accept_static(p_target, q_draft, draft_tokens, uniforms, q_indptr, max_k,
                       accepted_len, out_tokens):
    """spec_accept through the entry point that allocates nothing (its scratch is a
    static device array): for callers that cannot allocate, so the outputs are
    the caller's.  Returns (accepted_len, out_tokens)."""
    _dev(p_target, torch.float32, "p_target")
    _dev(uniforms, torch.float32, "uniforms")
    _dev(q_indptr, torch.int32, "q_indptr")
    _dev(accepted_len, torch.int32, "accepted_len")
    _dev(out_tokens, torch.int32, "out_tokens")
    if max_k > 0:
        _dev(q_draft, torch.float32, "q_draft")
        _dev(draft_tokens, torch.int32, "draft_tokens")
    total_q, vocab = p_target.shape
    bs = q_indptr.numel() - 1
    if uniforms.numel() != total_q or out_tokens.numel() != total_q or accepted_len.numel() != bs:
        raise ValueError("uniforms / out_tokens / accepted_len do not match the rows")
    if max_k > 0 and (q_draft.shape != (total_q - bs, vocab) or draft_tokens.numel() != total_q - bs):
        raise ValueError("q_draft / draft_tokens must have total_q - bs rows")
    _check("spec_accept_static", lib().nsd_spec_accept_static(
        _ptr(p_target), _ptr(q_draft) if max_k > 0 else None,
        _ptr(draft_tokens) if max_k > 0 else None, _ptr(uniforms), _ptr(q_indptr), bs, vocab,
        max_k, _ptr(accepted_len), _ptr(out_tokens), _stream(p_target)))
    return accepted_len, out_tokens


def sample(probs, uniforms, out=None, workspace=None):
    """One token per row by inverse CDF (the draft step's x_i ~ q_i).

    probs: fp32 [n][V] on the GPU whose rows may be strided (unit stride within
    a row, row stride a multiple of 4), e.g. step i of request-major draft rows
    ``q_draft.view(bs, K, V)[:, i]``; uniforms: fp32 [n]; out: int32 [n],
    possibly strided (e.g. ``draft_tokens.view(bs, K)[:, i]``); workspace: at
    least accept_workspace_size(n, V) bytes (allocated per call when None).
    Returns out."""
    if probs.dtype != torch.float32 or not probs.is_cuda or probs.dim() != 2:
        raise TypeError("probs must be a 2-d fp32 GPU tensor")
    n, vocab = probs.shape
    if (n > 1 and probs.stride(0) < vocab) or (vocab > 1 and probs.stride(1) != 1):
        raise ValueError("probs rows must be unit-stride and not overlap")
    _dev(uniforms, torch.float32, "uniforms")
    if uniforms.numel() != n:
        raise ValueError("uniforms must have one entry per row")
    if out is None:
        out = torch.empty(n, dtype=torch.int32, device=probs.device)
    if out.dtype != torch.int32 or not out.is_cuda or out.dim() != 1 or out.numel() != n:
        raise ValueError("out must be int32 [n] on the GPU")
    ws, ws_n = _accept_ws(workspace, n, vocab, probs.device)
    _check("sample", lib().nsd_sample(
        _ptr(probs), probs.stride(0) if n > 1 else vocab, _ptr(uniforms), n, vocab, _ptr(out),
        max(1, out.stride(0)), _ptr(ws), ws_n, _stream(probs)))
    return out


COPY_H2D, COPY_D2H = 1, 2
DEFAULT_CHUNK = 32 << 20   # bytes per DMA submission


def copy_plan(src, dst, copies, chunk_bytes=DEFAULT_CHUNK, stream=None, window_bytes=None):
    """Execute a KV copy plan between a pinned host tensor and a device tensor.

    copies: int64 array [n][3] of (source byte offset, destination byte offset,
    bytes).  The direction follows the tensors' devices; the host tensor must be
    pinned.  Runs on ``stream`` (a torch.cuda.Stream) or the current stream.
    With ``window_bytes`` the chunks are submitted in bounded groups and the
    call blocks until the last group is submitted (nsd_copy_plan_windowed)."""
    import numpy as np
    if src.is_cuda == dst.is_cuda:
        raise ValueError("copy_plan moves between a pinned host tensor and a device tensor")
    host, dev = (src, dst) if dst.is_cuda else (dst, src)
    if not host.is_pinned():
        raise ValueError("the host tensor must be pinned (pin_memory=True)")
    if not (src.is_contiguous() and dst.is_contiguous()):
        raise ValueError("src and dst must be contiguous")
    plan = np.ascontiguousarray(np.asarray(copies, dtype=np.int64).reshape(-1, 3))
    st = (stream or torch.cuda.current_stream(dev.device)).cuda_stream
    direction = COPY_H2D if dst.is_cuda else COPY_D2H
    if window_bytes is None:
        _check("copy_plan", lib().nsd_copy_plan(
            _ptr(src), src.numel() * src.element_size(), _ptr(dst),
            dst.numel() * dst.element_size(), plan.ctypes.data if len(plan) else None,
            len(plan), int(chunk_bytes), direction, st))
    else:
        _check("copy_plan_windowed", lib().nsd_copy_plan_windowed(
            _ptr(src), src.numel() * src.element_size(), _ptr(dst),
            dst.numel() * dst.element_size(), plan.ctypes.data if len(plan) else None,
            len(plan), int(chunk_bytes), int(window_bytes), direction, st))


def kv_append(k_pool, v_pool, k_new, v_new, block_table, seq_lens, q_indptr):
    """Write the window rows k_new/v_new [total_q][Hkv][D] into their paged slots (one layer)."""
    for t, n in ((k_pool, "k_pool"), (v_pool, "v_pool"), (k_new, "k_new"), (v_new, "v_new")):
        _dev(t, torch.bfloat16, n)
    for t, n in ((block_table, "block_table"), (seq_lens, "seq_lens"), (q_indptr, "q_indptr")):
        _dev(t, torch.int32, n)
    total_q, hkv, d = k_new.shape
    nb = k_pool.shape[0]
    if v_new.shape != k_new.shape or d % 8 or k_pool.shape != (nb, hkv, d // 8, BLOCK_SIZE, 8) \
            or v_pool.shape != (nb, hkv, d, BLOCK_SIZE):
        raise ValueError("k_new/v_new must be [total_q][Hkv][D] matching the pools")
    bs = seq_lens.numel()
    if block_table.dim() != 2 or block_table.shape[0] != bs or q_indptr.numel() != bs + 1:
        raise ValueError("block_table / q_indptr do not match seq_lens")
    _check("kv_append", lib().nsd_kv_append(
        _ptr(k_pool), _ptr(v_pool), k_pool.shape[0], _ptr(k_new), _ptr(v_new), _ptr(block_table),
        block_table.shape[1], _ptr(seq_lens), _ptr(q_indptr), seq_lens.numel(), total_q, hkv,
        BLOCK_SIZE, d, _stream(k_pool)))


def commit_lengths(seq_lens, q_indptr, accepted_len, out=None):
    """Committed lengths seq_lens - K + accepted_len (int32 [bs])."""
    for t, n in ((seq_lens, "seq_lens"), (q_indptr, "q_indptr"), (accepted_len, "accepted_len")):
        _dev(t, torch.int32, n)
    bs = seq_lens.numel()
    if q_indptr.numel() != bs + 1 or accepted_len.numel() != bs:
        raise ValueError("q_indptr / accepted_len do not match seq_lens")
    if out is None:
        out = torch.empty_like(seq_lens)
    else:
        _dev(out, torch.int32, "out")
        if out.numel() != bs:
            raise ValueError("out must have one entry per request")
    _check("commit_lengths", lib().nsd_commit_lengths(
        _ptr(seq_lens), _ptr(q_indptr), _ptr(accepted_len), _ptr(out), seq_lens.numel(),
        _stream(seq_lens)))
    return out


def host_alias(t):
    """Device address of a pinned host tensor's data."""
    if t.is_cuda or not t.is_pinned():
        raise ValueError("host_alias needs a pinned host tensor")
    p = ctypes.c_void_p()
    _check("host_alias", lib().nsd_host_alias(_ptr(t), ctypes.byref(p)))
    return p.value


def kv_writeback(k_pool, v_pool, host_k, host_v, src_ids, dst_ids):
    """Copy whole pool blocks src_ids[i] into blocks dst_ids[i] of a pinned host arena
    (same block layout), by the gather kernel writing through the arena's device alias."""
    _dev(k_pool, torch.bfloat16, "k_pool")
    _dev(v_pool, torch.bfloat16, "v_pool")
    _dev(src_ids, torch.int32, "src_ids")
    _dev(dst_ids, torch.int32, "dst_ids")
    if host_k.shape[1:] != k_pool.shape[1:] or host_v.shape[1:] != v_pool.shape[1:]:
        raise ValueError("the arena must have the pool's block layout")
    hkv, d = k_pool.shape[1], v_pool.shape[2]
    _check("kv_writeback", lib().nsd_kv_gather(
        _ptr(k_pool), _ptr(v_pool), k_pool.shape[0], host_alias(host_k), host_alias(host_v),
        host_k.shape[0], _ptr(src_ids), _ptr(dst_ids), src_ids.numel(), 1, 0, 1, hkv,
        BLOCK_SIZE, d, _stream(k_pool)))


__all__ = ["lib", "version", "attention_waves", "check_plan", "check_pairs", "kv_gather", "verify_attention", "verify_attention_workspace_size",
           "new_workspace", "gather_verify_attention", "copy_plan", "COPY_H2D", "COPY_D2H",
           "DEFAULT_CHUNK", "kv_append", "commit_lengths", "host_alias", "kv_writeback",
           "spec_accept", "spec_accept_static", "accept_workspace_size", "sample", "NsdError", "BLOCK_SIZE", "LIB_PATH"]
