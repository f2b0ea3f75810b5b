"""Pins for oracle.schedule: a hand-worked reconstruction, the admission
conditions recomputed over the whole batch, greedy rejections, capacity and
degenerate cases; simulator closed forms (one cohort in lockstep, two cohorts
keeping both workers busy) and invariants of every trace."""
import math

import numpy as np
import pytest

from oracle.schedule import INF, interp, reconstruct, simulate


def test_interp_closed_forms():
    b, v = [1, 4, 8], [2.0, 5.0, 13.0]
    assert interp(b, v, 1) == 2.0 and interp(b, v, 4) == 5.0 and interp(b, v, 8) == 13.0
    assert interp(b, v, 2) == 3.0 and interp(b, v, 6) == 9.0
    assert interp(b, v, 0) == 2.0 and interp(b, v, 100) == 13.0


def _worked(b_max, delta):
    # a^ = 5, g = 2; (id, e~, k^)
    ids = [0, 1, 2, 3, 4]
    e = [4.0, 6.0, 1.0, 5.5, 0.0]
    k = [3.0, 0.0, 9.0, 0.0, 0.0]
    z = [0] * 5
    return reconstruct(ids, e, k, z, z, 5.0, 0, 0, b_max, 2.0, delta)


def test_worked_example():
    # S({r}) = 5, 6, 9, 5.5, 5 and d^ = S... : with Delta = 1, d^ = 7, 9, 10, 8.5, 6,
    # rank 4, 0, 3, 1, 2
    assert _worked(3, 1.0) == ([4, 0, 3], 5.5)
    # r1 joins with S(B) = 6 = min d^ (equality admits); r2 would need S = 9 > 6
    assert _worked(5, 1.0) == ([4, 0, 3, 1], 6.0)
    # Delta = 0.4: d^ = 6.4, 8.4, 9.4, 7.9, 5.4; r3 would start the batch at 5.5 > 5.4
    assert _worked(5, 0.4) == ([4, 0], 5.0)


def _admissible(batch, pos, e, k, a_hat, g, delta, b_max, blocks, tokens, bcap, tcap):
    if not batch:
        return True
    idx = [pos[r] for r in batch]
    s_b = max([a_hat] + [e[i] for i in idx] + [k[i] for i in idx])
    d = min(max(e[i] + g, max(a_hat, e[i], k[i])) + delta for i in idx)
    return (len(batch) <= b_max and sum(blocks[i] for i in idx) <= bcap
            and sum(tokens[i] for i in idx) <= tcap and s_b <= d)


@pytest.mark.parametrize("seed", range(40))
def test_batches_are_admissible_and_rejections_justified(seed):
    g = np.random.default_rng(seed)
    n = int(g.integers(1, 30))
    ids = list(g.permutation(1000)[:n])
    e = list(g.uniform(0, 10, n).round(2))
    k = list(g.uniform(0, 10, n).round(2))
    blocks = list(g.integers(1, 50, n))
    tokens = list(g.integers(1, 9, n))
    a_hat = float(g.uniform(0, 10))
    gs, delta = float(g.uniform(0, 3)), float(g.uniform(0, 3))
    b_max = int(g.integers(1, 12))
    bcap, tcap = int(g.integers(20, 400)), int(g.integers(5, 60))
    batch, s_b = reconstruct(ids, e, k, blocks, tokens, a_hat, bcap, tcap, b_max, gs, delta)
    pos = {r: i for i, r in enumerate(ids)}
    assert len(set(batch)) == len(batch)
    assert _admissible(batch, pos, e, k, a_hat, gs, delta, b_max, blocks, tokens, bcap, tcap)
    if batch:
        idx = [pos[r] for r in batch]
        assert s_b == max([a_hat] + [e[i] for i in idx] + [k[i] for i in idx])
    # replay the scan over the ranked first-B_max list: every rejected candidate
    # breaks Eq. 8 against the batch admitted before it
    fits = [i for i in range(n) if blocks[i] <= bcap and tokens[i] <= tcap]
    key = lambda i: (max(e[i] + gs, max(a_hat, e[i], k[i])) + delta,
                     max(a_hat, e[i], k[i]), ids[i])
    ranked = sorted(fits, key=key)[:b_max]
    prefix = []
    for i in ranked:
        if ids[i] in batch:
            assert _admissible(prefix + [ids[i]], pos, e, k, a_hat, gs, delta, b_max, blocks,
                               tokens, bcap, tcap)
            prefix.append(ids[i])
        else:
            assert not _admissible(prefix + [ids[i]], pos, e, k, a_hat, gs, delta, b_max,
                                   blocks, tokens, bcap, tcap)
    assert prefix == batch


def test_unbounded_slack_takes_the_first_b_max():
    ids = list(range(10))
    e = [9.0, 1.0, 5.0, 2.0, 8.0, 3.0, 7.0, 4.0, 6.0, 0.0]
    z = [0] * 10
    batch, s_b = reconstruct(ids, e, [0.0] * 10, z, z, 0.0, 0, 0, 4, 0.0, INF)
    assert batch == [9, 1, 3, 5] and s_b == 3.0       # ranked by singleton start, then id
    same = reconstruct([7, 3, 5], [1.0] * 3, [1.0] * 3, [0] * 3, [0] * 3, 0.0, 0, 0, 2, 0.5, 0.0)
    assert same == ([3, 5], 1.0)


def test_capacity_fit():
    ids = [0, 1, 2, 3]
    z = [0.0] * 4
    blocks = [120, 60, 50, 30]      # request 0 never fits a 100-block bank
    batch, _ = reconstruct(ids, z, z, blocks, [1] * 4, 0.0, 100, 100, 4, 1.0, 1.0)
    assert batch == [1, 3]          # 1 + 2 would need 110 blocks; 3 still fits
    batch, _ = reconstruct(ids, z, z, [1] * 4, [3, 3, 3, 3], 0.0, 100, 7, 4, 1.0, 1.0)
    assert batch == [0, 1]          # token budget 7 holds two requests of 3
    assert reconstruct([], [], [], [], [], 0.0, 1, 1, 4, 1.0, 1.0) == ([], None)


CONST = lambda t, sm: ([1, 4096], [t, t], [sm, sm])


@pytest.mark.parametrize("a,b,sd,st,r", [(1.0, 1.0, 0.5, 0.5, 8), (0.25, 0.75, 0.3, 0.9, 5),
                                         (2.0, 0.5, 0.6, 0.2, 1)])
def test_one_cohort_in_lockstep(a, b, sd, st, r):
    # every request fits one batch: draft and target alternate, period a + b
    rounds = 6
    w = (a + b, 4 * (a + b))
    m, trace = simulate(1, 1, r, rounds, CONST(a, sd), CONST(b, st), 512, 512, 0.0, 0.0, 0.0,
                        0.0, w)
    assert m["finished"] == r and m["batches"] == 2 * rounds
    span = w[1] - w[0]
    assert math.isclose(m["U"], 3 * (a * sd + b * st) / (2 * span))
    assert math.isclose(m["S"], 1.0)
    assert math.isclose(m["round_rate"], r / (a + b))


def test_two_cohorts_keep_both_workers_busy():
    # 2 B_max requests, equal stage times: while one cohort drafts the other verifies
    bm, a = 4, 1.0
    m, trace = simulate(1, 1, 2 * bm, 8, CONST(a, 0.5), CONST(a, 0.8), bm, bm, 0.0, 0.0, 10.0,
                        10.0, (2.0, 6.0))
    assert math.isclose(m["U"], (0.5 + 0.8) / 2)
    assert math.isclose(m["S"], 1.0)
    assert math.isclose(m["round_rate"], bm / a)
    # the second draft batch was planned on the standby slot and starts as the first ends
    assert trace[1][0] == 0 and trace[1][2] == a


@pytest.mark.parametrize("seed", range(12))
def test_trace_invariants(seed):
    g = np.random.default_rng(seed)
    nd, nt = int(g.integers(1, 4)), int(g.integers(1, 5))
    r, rounds = int(g.integers(1, 60)), int(g.integers(1, 5))
    sizes = [1, 8, 32, 128]
    phi_d = (sizes, list(np.sort(g.uniform(0.5, 2.0, 4)).round(3)), list(g.uniform(0, 1, 4)))
    phi_t = (sizes, list(np.sort(g.uniform(0.5, 3.0, 4)).round(3)), list(g.uniform(0, 1, 4)))
    bmd, bmt = int(g.integers(1, 40)), int(g.integers(1, 20))
    m, trace = simulate(nd, nt, r, rounds, phi_d, phi_t, bmd, bmt, float(g.uniform(0, 2)),
                        float(g.uniform(0, 2)), float(g.uniform(0, 2)), float(g.uniform(0, 2)),
                        (0.0, 10.0))
    assert m["finished"] == r
    per_req = {i: [] for i in range(r)}
    busy = {}
    for s, w, a, b, members in trace:
        assert 1 <= len(members) <= (bmd if s == 0 else bmt)
        assert math.isclose(b - a, interp(*(phi_d if s == 0 else phi_t)[:2], len(members)))
        busy.setdefault((s, w), []).append((a, b))
        for q in members:
            per_req[q].append((s, a, b))
    for spans in busy.values():                      # a worker runs one batch at a time
        spans.sort()
        assert all(spans[i][1] <= spans[i + 1][0] for i in range(len(spans) - 1))
    for q, stages in per_req.items():                # D, T, D, T, ... each after its predecessor
        stages.sort(key=lambda x: x[1])
        assert [s for s, _, _ in stages] == [0, 1] * rounds
        assert all(stages[i][2] <= stages[i + 1][1] for i in range(len(stages) - 1))
    assert 0.0 <= m["U"] <= 1.0 and 0.0 <= m["S"] <= 1.0


def test_scaling_pools_and_requests_together_keeps_the_operating_point():
    # Appendix H: with the draft-target ratio and the requests per worker fixed, the
    # idealized simulator keeps U and S and scales the round rate with the pool
    phi_d = ([1, 512, 1024], [0.064, 0.072, 0.1544], [0.091, 0.868, 0.951])
    phi_t = ([1, 32, 64, 128], [0.0288, 0.0288, 0.0463, 0.0828], [0.741, 0.875, 0.932, 0.957])
    base, _ = simulate(1, 4, 150, 6, phi_d, phi_t, 64, 16, 0.0, 0.0, 0.03, 0.03, (0.1, 0.4))
    for k in (2, 3):
        m, _ = simulate(k, 4 * k, 150 * k, 6, phi_d, phi_t, 64, 16, 0.0, 0.0, 0.03, 0.03,
                        (0.1, 0.4))
        assert math.isclose(m["U"], base["U"], rel_tol=1e-12)
        assert math.isclose(m["S"], base["S"], rel_tol=1e-12)
        assert math.isclose(m["round_rate"], k * base["round_rate"], rel_tol=1e-12)
