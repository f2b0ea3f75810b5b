"""Helpers the GPU parity tests share: moving inputs to the device and
comparing GPU results with the oracle under the stated tolerances."""
import numpy as np
import torch

import oracle
from workload.synth import logical_kv

ATTN_ATOL = 2e-2        # bf16 inputs, fp32 accumulation, bf16 output
CDF_BOUNDARY = 1e-6     # a resampled token may differ only this close to a CDF boundary


def i32(a, dev):
    return torch.as_tensor(np.ascontiguousarray(a), dtype=torch.int32, device=dev)


def u16(t):
    return t.view(torch.int16).cpu().numpy()


def attention_ref(meta, layer, r, scale=None):
    cfg = meta.cfg
    k, v = logical_kv(meta, layer, r)
    a, b = int(meta.q_indptr[r]), int(meta.q_indptr[r + 1])
    scale = 1.0 / np.sqrt(cfg.head_dim) if scale is None else scale
    # bf16 bytes to the host first, widened there (a quarter of the transfer)
    return oracle.attention.verify_attention_request(
        layer.q[a:b].cpu().double().numpy(), k.cpu().double().numpy(),
        v.cpu().double().numpy(), scale)


def check_attention(meta, layer, out, requests, scale=None):
    """Max abs error over the listed requests; asserts the tolerance."""
    o = out.float().cpu().numpy() if isinstance(out, torch.Tensor) else out
    worst = 0.0
    for r in requests:
        a, b = int(meta.q_indptr[r]), int(meta.q_indptr[r + 1])
        ref = attention_ref(meta, layer, r, scale)
        got = o[a:b]
        assert np.isfinite(got).all(), f"request {r}: non-finite output"
        err = float(np.abs(got - ref).max())
        worst = max(worst, err)
        assert err <= ATTN_ATOL, f"request {r} (L={meta.seq_lens[r]}): max error {err}"
    return worst


def check_accept(p, q, x, u, q_indptr, acc_gpu, tok_gpu, requests=None):
    """accepted_len bit-exact; tokens exact except at a CDF boundary; never a
    zero-weight token.  Inputs are host numpy arrays."""
    bs = len(q_indptr) - 1
    requests = range(bs) if requests is None else requests
    ref_acc, ref_tok = oracle.accept.spec_accept(p, q, x, u, q_indptr, requests=requests)
    near = 0
    for r in requests:
        a, b = int(q_indptr[r]), int(q_indptr[r + 1])
        k = b - a - 1
        n = int(ref_acc[r])
        assert int(acc_gpu[r]) == n, f"request {r}: accepted {acc_gpu[r]} vs {n}"
        assert list(tok_gpu[a:a + n]) == list(ref_tok[a:a + n])
        assert all(t == -1 for t in tok_gpu[a + n + 1:b])
        w = oracle.accept.residual_weights(p[a:b], q[a - r:a - r + k], n)
        yg, yr = int(tok_gpu[a + n]), int(ref_tok[a + n])
        assert 0 <= yg < len(w) and w[yg] > 0, f"request {r}: emitted token {yg} has no weight"
        if yg != yr:
            c = np.cumsum(w)
            s = c[-1]
            lo, hi = min(yg, yr), max(yg, yr)
            uk = float(u[b - 1])
            assert abs(c[lo] / s - uk) <= CDF_BOUNDARY and abs(c[hi - 1] / s - uk) <= CDF_BOUNDARY, \
                f"request {r}: token {yg} vs {yr} away from a CDF boundary"
            near += 1
    return near


def check_samples(rows, u, got):
    """Inverse-CDF draws against oracle.draft.sample: equal except within
    CDF_BOUNDARY of a CDF boundary; a token of zero weight is never drawn.
    rows: [n][V] host array, u: [n], got: [n] ints.  Returns the number of
    boundary cases."""
    rows = np.asarray(rows)
    ref = oracle.draft.sample(rows, u)
    near = 0
    for i in range(len(rows)):
        g, e = int(got[i]), int(ref[i])
        if e < 0:
            assert g == -1, f"row {i}: drew {g} from a row without mass"
            continue
        w = rows[i].astype(np.float64)
        assert 0 <= g < len(w) and w[g] > 0, f"row {i}: token {g} has no weight"
        if g != e:
            c = np.cumsum(w)
            lo, hi = min(g, e), max(g, e)
            ui = float(u[i])
            assert abs(c[lo] / c[-1] - ui) <= CDF_BOUNDARY and \
                abs(c[hi - 1] / c[-1] - ui) <= CDF_BOUNDARY, \
                f"row {i}: token {g} vs {e} away from a CDF boundary"
            near += 1
    return near
