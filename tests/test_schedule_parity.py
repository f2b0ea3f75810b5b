"""The library's host scheduler (C++, through the C ABI) against
oracle.schedule: identical batches and start times for single opportunities,
identical traces and metrics for whole simulations.  No GPU is involved."""
import math

import numpy as np
import pytest

import oracle.schedule as ref
from paper_2609_29364_amd import schedule as sch
from paper_2609_29364_amd import NsdError


@pytest.mark.parametrize("seed", range(60))
def test_reconstruct_matches_oracle(seed):
    g = np.random.default_rng(100 + seed)
    n = int(g.integers(0, 200))
    ids = [int(x) for x in g.permutation(5000)[:n]]
    # coarse grids make ties in d^ and S({r}) common, so the id tie-break matters
    e = list(g.integers(0, 12, n) * 0.5)
    k = list(g.integers(0, 12, n) * 0.5)
    if n > 3:
        e[0], k[1] = math.inf, -math.inf
    blocks = [int(x) for x in g.integers(0, 40, n)]
    tokens = [int(x) for x in g.integers(0, 9, n)]
    a_hat = float(g.integers(0, 10) * 0.5)
    gs = float(g.integers(0, 6) * 0.5)
    delta = math.inf if seed % 7 == 0 else float(g.integers(0, 6) * 0.25)
    b_max = int(g.integers(1, 64))
    bcap, tcap = int(g.integers(0, 800)), int(g.integers(0, 200))
    want = ref.reconstruct(ids, e, k, blocks, tokens, a_hat, bcap, tcap, b_max, gs, delta)
    got = sch.reconstruct(ids, e, k, blocks, tokens, a_hat, bcap, tcap, b_max, gs, delta)
    assert got == want


def _tables(g, sizes):
    t = np.sort(g.uniform(0.2, 3.0, len(sizes))).round(3)
    sm = g.uniform(0.05, 1.0, len(sizes)).round(3)
    return (list(sizes), list(t), list(sm))


@pytest.mark.parametrize("seed", range(25))
def test_simulation_matches_oracle(seed):
    g = np.random.default_rng(200 + seed)
    nd, nt = int(g.integers(1, 4)), int(g.integers(1, 6))
    r, rounds = int(g.integers(0, 120)), int(g.integers(0, 6))
    phi_d = _tables(g, [1, 16, 64, 512])
    phi_t = _tables(g, [1, 4, 24, 32])
    args = (nd, nt, r, rounds, phi_d, phi_t, int(g.integers(1, 80)), int(g.integers(1, 33)),
            float(g.integers(0, 4) * 0.5), float(g.integers(0, 4) * 0.5),
            float(g.integers(0, 4) * 0.25), math.inf if seed % 5 == 0 else float(g.uniform(0, 1)),
            (float(g.uniform(0, 2)), float(g.uniform(3, 8))))
    stop = math.inf if seed % 3 else 4.0
    want_m, want_t = ref.simulate(*args, t_stop=stop)
    got_m, got_t = sch.simulate(*args, t_stop=stop)
    assert got_t == want_t
    assert got_m == want_m


def test_metrics_only_run_and_small_trace_buffers():
    phi = ([1, 64], [1.0, 2.0], [0.3, 0.9])
    args = (2, 3, 50, 3, phi, phi, 16, 8, 0.5, 0.5, 0.5, 0.5, (1.0, 5.0))
    m_full, tr = sch.simulate(*args)
    m_only, none = sch.simulate(*args, trace=False)
    assert none is None and m_only == m_full and m_full["batches"] == len(tr)
    # too small a trace buffer: the metrics are still computed, the call reports the sizes
    from paper_2609_29364_amd import lib
    import ctypes
    cfg = sch.SimConfig(2, 3, 50, 3, (16, 8), (0.5, 0.5), (0.5, 0.5), (1.0, 5.0), math.inf)
    t = np.ascontiguousarray(np.asarray(phi, dtype=np.float64))
    m = sch.SimMetrics()
    buf = (sch.SimBatch * 2)()
    mem = np.zeros(4, dtype=np.int32)
    nt_, nm_ = ctypes.c_int64(), ctypes.c_int64()
    st = lib().nsd_simulate(ctypes.addressof(cfg), t.ctypes.data, 2, t.ctypes.data, 2,
                            ctypes.addressof(m), ctypes.addressof(buf), 2, mem.ctypes.data, 4,
                            ctypes.byref(nt_), ctypes.byref(nm_))
    assert st == 4 and nt_.value == len(tr) and nm_.value == sum(len(x[4]) for x in tr)
    assert m.U == m_full["U"] and m.batches == m_full["batches"]


def test_argument_checks():
    with pytest.raises(NsdError):
        sch.reconstruct([0], [math.nan], [0.0], b_max=2)
    with pytest.raises(NsdError):
        sch.reconstruct([0], [0.0], [0.0], b_max=0)
    with pytest.raises(NsdError):
        sch.reconstruct([0], [0.0], [0.0], b_max=1, g=-1.0)
    assert sch.reconstruct([], [], [], b_max=3) == ([], None)
    good = ([1, 8], [1.0, 2.0], [0.5, 0.5])
    for bad in (([8, 1], [1.0, 2.0], [0.5, 0.5]), ([1, 8], [0.0, 2.0], [0.5, 0.5]),
                ([1, 8], [1.0, math.nan], [0.5, 0.5])):
        with pytest.raises(NsdError):
            sch.simulate(1, 1, 4, 1, bad, good, 4, 4, 0.0, 0.0, 0.0, 0.0, (0.0, 1.0))
    with pytest.raises(NsdError):
        sch.simulate(0, 1, 4, 1, good, good, 4, 4, 0.0, 0.0, 0.0, 0.0, (0.0, 1.0))
    with pytest.raises(NsdError):
        sch.simulate(1, 1, 4, 1, good, good, 4, 4, 0.0, 0.0, 0.0, 0.0, (1.0, 1.0))


def test_large_simulation_runs_to_completion():
    # a 38-GPU pool (6 draft + 32 target workers), 4096 requests, 32 rounds
    sizes_d, sizes_t = [1, 64, 256, 512], [1, 8, 24, 32]
    phi_d = (sizes_d, [16.0, 16.5, 17.5, 18.0], [0.09, 0.5, 0.8, 0.87])
    phi_t = (sizes_t, [20.0, 22.0, 27.0, 28.8], [0.74, 0.8, 0.86, 0.875])
    m, _ = sch.simulate(6, 32, 4096, 32, phi_d, phi_t, 512, 32, 10.0, 10.0, 20.0, 20.0,
                        (1000.0, 2500.0), trace=False)
    assert m["finished"] == 4096 and 0 < m["U"] <= 1 and 0 < m["S"] <= 1
