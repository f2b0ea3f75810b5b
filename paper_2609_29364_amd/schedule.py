"""Binding of the library's host-side scheduler: one worker-triggered batch
reconstruction (Algorithm 1, Eqs. 4-8) and the ideal-migration discrete-event
simulation of the draft and target pools (Appendix H).  Argument marshalling
only; both run in the library's C++ code."""
import ctypes
import math

import numpy as np

from . import lib, _check


class SimConfig(ctypes.Structure):
    _fields_ = [("n_draft", ctypes.c_int32), ("n_target", ctypes.c_int32),
                ("n_requests", ctypes.c_int32), ("rounds", ctypes.c_int32),
                ("b_max", ctypes.c_int32 * 2), ("g", ctypes.c_double * 2),
                ("delta", ctypes.c_double * 2), ("window", ctypes.c_double * 2),
                ("t_stop", ctypes.c_double)]


class SimMetrics(ctypes.Structure):
    _fields_ = [("U", ctypes.c_double), ("S", ctypes.c_double), ("round_rate", ctypes.c_double),
                ("finished", ctypes.c_int64), ("batches", ctypes.c_int64)]


class SimBatch(ctypes.Structure):
    _fields_ = [("stage", ctypes.c_int32), ("worker", ctypes.c_int32), ("size", ctypes.c_int32),
                ("first", ctypes.c_int64), ("start", ctypes.c_double), ("end", ctypes.c_double)]


def _arr(a, dtype):
    return np.ascontiguousarray(np.asarray(a, dtype=dtype))


def reconstruct(ids, e_tilde, k_hat, blocks=None, tokens=None, a_hat=0.0, block_cap=0,
                token_cap=0, b_max=1, g=0.0, delta=0.0):
    """One scheduling opportunity; returns (batch ids in admission order, S(B) or None)."""
    ids, e, k = _arr(ids, np.int32), _arr(e_tilde, np.float64), _arr(k_hat, np.float64)
    n = len(ids)
    if len(e) != n or len(k) != n:
        raise ValueError("ids, e_tilde and k_hat differ in length")
    bl = None if blocks is None else _arr(blocks, np.int64)
    tk = None if tokens is None else _arr(tokens, np.int64)
    for a in (bl, tk):
        if a is not None and len(a) != n:
            raise ValueError("blocks / tokens must have one entry per candidate")
    out = np.zeros(max(1, b_max), dtype=np.int32)
    length, start = ctypes.c_int32(), ctypes.c_double()
    p = lambda a: None if a is None or len(a) == 0 else a.ctypes.data
    _check("reconstruct", lib().nsd_reconstruct(
        p(ids), p(e), p(k), p(bl), p(tk), n, float(a_hat), int(block_cap), int(token_cap),
        int(b_max), float(g), float(delta), out.ctypes.data, ctypes.byref(length),
        ctypes.byref(start)))
    n_b = length.value
    return [int(x) for x in out[:n_b]], (start.value if n_b else None)


def _table(phi):
    t = np.ascontiguousarray(np.asarray(phi, dtype=np.float64).reshape(3, -1))
    return t, t.shape[1]


def simulate(n_draft, n_target, n_requests, rounds, phi_d, phi_t, b_max_d, b_max_t, g_d, g_t,
             delta_d, delta_t, window, t_stop=math.inf, trace=True):
    """Run the simulation; phi_* = (sizes, times, sm).  Returns (metrics dict,
    trace [(stage, worker, start, end, members)] or None)."""
    cfg = SimConfig(n_draft, n_target, n_requests, rounds, (b_max_d, b_max_t), (g_d, g_t),
                    (delta_d, delta_t), tuple(window), t_stop)
    td, nd = _table(phi_d)
    tt, nt = _table(phi_t)
    m = SimMetrics()
    n_tr, n_mem = ctypes.c_int64(), ctypes.c_int64()
    tr_buf = mem_buf = None
    cap_t = cap_m = 0
    if trace:
        # first pass sizes the trace, second records it
        st = lib().nsd_simulate(ctypes.addressof(cfg), td.ctypes.data, nd, tt.ctypes.data, nt,
                                ctypes.addressof(m), None, 0, None, 0, ctypes.byref(n_tr),
                                ctypes.byref(n_mem))
        _check("simulate", st)
        cap_t, cap_m = n_tr.value, n_mem.value
        tr_buf = (SimBatch * max(1, cap_t))()
        mem_buf = np.zeros(max(1, cap_m), dtype=np.int32)
    _check("simulate", lib().nsd_simulate(
        ctypes.addressof(cfg), td.ctypes.data, nd, tt.ctypes.data, nt, ctypes.addressof(m),
        None if tr_buf is None else ctypes.addressof(tr_buf), cap_t,
        None if mem_buf is None else mem_buf.ctypes.data, cap_m, ctypes.byref(n_tr),
        ctypes.byref(n_mem)))
    metrics = {"U": m.U, "S": m.S, "round_rate": m.round_rate, "finished": m.finished,
               "batches": m.batches}
    if not trace:
        return metrics, None
    out = [(b.stage, b.worker, b.start, b.end, [int(x) for x in mem_buf[b.first:b.first + b.size]])
           for b in tr_buf[:n_tr.value]]
    return metrics, out
