"""Oracle for worker-triggered batch reconstruction and the profiling-driven
discrete-event simulator -- TEST INFRASTRUCTURE (imported only by the test
suite and the benchmark's CPU baseline).

Batch reconstruction (Section 4, Algorithm 1, Eqs. 4-8; Appendix F.2):
for a scheduling opportunity of worker w at stage s, every eligible request r
has an available predecessor completion time e~_r (observed, or predicted as
t_start + phi(z) for a running predecessor batch, Eq. 4) and a KV-ready time
k^_r(w).  The worker is available at a^_w.

* singleton start  S({r}) = max(a^_w, e~_r, k^_r)                   (Eq. 6)
* admission bound  d^_r = max(e~_r + g_s, S({r})) + Delta_s          (Eq. 7)
* batch start      S(B) = max(a^_w, max_r e~_r, max_r k^_r)          (Eqs. 5, 6)
* admissible      |B| <= B_max, Fit(B, w), S(B) <= min_{r in B} d^_r  (Eq. 8)

Fit: the batch's KV blocks and tokens stay within the bank's capacities, and
each request fits on its own (Appendix F.2).  Candidates are ranked, the first
B_max form F, and F is scanned once in rank order, adding each request that
keeps the batch admissible (Algorithm 1).

Ranking reading (the paper names its criteria -- service urgency via the
waiting time, temporal compatibility, the singleton start as a feasibility
baseline -- but no formula): ascending admission bound d^_r (earliest
deadline; an earlier predecessor completion means a longer wait, which gives
the aging), then ascending singleton start, then request id.

Simulator (Appendix H): requests start at t = 0 after prefill with an anchor
token and run a fixed number of speculative rounds, each a draft stage then a
target stage (Eq. 1).  Stage times and SM activity come from profiled tables
interpolated linearly across batch sizes.  Migration is ideal (KV ready at
planning time).  Each worker has a compute slot and one standby preparation
slot: whenever a worker holds no prepared batch it is a planning
opportunity (workers in index order, draft workers first); requests whose
predecessor batch is still running take part with its predicted end.  A
prepared batch starts once every member's predecessor output is published
and the worker is idle (InputReady, KVReady, WorkerReady).  All transitions at
one virtual time are applied before planning.  Metrics over the window
[w0, w1] (Eqs. H.1, H.2): U = sum tau_j s_j / (G Delta), S = sum tau_j b_j /
(R Delta), and the request-round rate = request-level target rounds completed
in the window (ends in (w0, w1]) / Delta.
"""
import math

INF = math.inf


def interp(table_b, table_v, b):
    """Linear interpolation of a profiled table over batch sizes (sizes
    ascending); constant beyond the ends."""
    if b <= table_b[0]:
        return float(table_v[0])
    for i in range(1, len(table_b)):
        if b <= table_b[i]:
            b0, b1 = table_b[i - 1], table_b[i]
            v0, v1 = table_v[i - 1], table_v[i]
            return v0 + (v1 - v0) * ((b - b0) / (b1 - b0))
    return float(table_v[-1])


def reconstruct(ids, e_tilde, k_hat, blocks, tokens, a_hat, block_cap, token_cap, b_max,
                g, delta):
    """One scheduling opportunity.  Per-candidate lists (same length): request
    ids, e~_r, k^_r, KV blocks, tokens.  Returns (batch ids in admission order,
    S(B) or None if empty)."""
    cands = []
    for i in range(len(ids)):
        if blocks[i] > block_cap or tokens[i] > token_cap:
            continue                                    # does not fit on its own
        s1 = max(a_hat, e_tilde[i], k_hat[i])
        d = max(e_tilde[i] + g, s1) + delta
        cands.append((d, s1, ids[i], i))
    cands.sort()
    first = cands[:b_max]
    batch = []
    s_b, d_min, used_b, used_t = a_hat, INF, 0, 0
    for d, _, rid, i in first:
        s_new = max(s_b, e_tilde[i], k_hat[i])
        d_new = min(d_min, d)
        if used_b + blocks[i] <= block_cap and used_t + tokens[i] <= token_cap and s_new <= d_new:
            batch.append(rid)
            s_b, d_min = s_new, d_new
            used_b += blocks[i]
            used_t += tokens[i]
    return batch, (s_b if batch else None)


def simulate(n_draft, n_target, n_requests, rounds, phi_d, phi_t, b_max_d, b_max_t, g_d, g_t,
             delta_d, delta_t, window, t_stop=INF):
    """Discrete-event simulation.  phi_d, phi_t: (sizes, times, sm) tables.
    Returns (metrics dict, batch trace [(stage, worker, start, end, members)]).

    Per request and stage: how many instances have been planned, and the state
    of the latest one: prepared (frozen, not started), running (its end
    predicted from its start, Eq. 4) or done (end observed).  A request needs
    a draft stage when both counts are equal (and rounds remain), a target
    stage otherwise; it is a candidate once the latest instance of the other
    stage is running or done (the prefill's anchor counts as a done target
    stage at t = 0)."""
    D, T = 0, 1
    NONE, PREPARED, RUNNING, DONE = 0, 1, 2, 3
    phis = (phi_d, phi_t)
    b_max = (b_max_d, b_max_t)
    gs = (g_d, g_t)
    deltas = (delta_d, delta_t)
    workers = [D] * n_draft + [T] * n_target
    index = list(range(n_draft)) + list(range(n_target))
    nw = len(workers)
    planned = [[0] * n_requests, [0] * n_requests]
    state = [[NONE] * n_requests, [DONE] * n_requests]
    end = [[0.0] * n_requests, [0.0] * n_requests]
    run_end = [None] * nw
    running = [None] * nw
    prepared = [None] * nw
    trace = []
    finished = 0
    t = 0.0

    def need(r):
        if planned[D][r] == planned[T][r]:
            return D if planned[D][r] < rounds else None
        return T

    while True:
        # 1. completions at time t (every transition at t before any planning)
        for w in range(nw):
            if run_end[w] is not None and run_end[w] == t:
                s = workers[w]
                for r in running[w]:
                    state[s][r] = DONE
                    if s == T and planned[T][r] == rounds:
                        finished += 1
                run_end[w], running[w] = None, None
        # 2. planning opportunities and 3. progress, until nothing changes at t
        changed = True
        while changed:
            changed = False
            for w in range(nw):
                if prepared[w] is not None:
                    continue
                s = workers[w]
                p = 1 - s
                ids, et, kh = [], [], []
                for r in range(n_requests):
                    if need(r) == s and state[p][r] in (RUNNING, DONE):
                        ids.append(r)
                        et.append(end[p][r])
                        kh.append(t)                      # ideal migration
                a_hat = run_end[w] if run_end[w] is not None else t
                zeros = [0] * len(ids)
                batch, _ = reconstruct(ids, et, kh, zeros, zeros, a_hat, 0, 0, b_max[s], gs[s],
                                       deltas[s])
                if batch:
                    prepared[w] = batch
                    for r in batch:
                        planned[s][r] += 1
                        state[s][r] = PREPARED
                    changed = True
            for w in range(nw):
                if prepared[w] is None or run_end[w] is not None:
                    continue
                s = workers[w]
                # InputReady: every member's predecessor output is published
                if all(state[1 - s][r] == DONE for r in prepared[w]):
                    members = prepared[w]
                    e = t + interp(phis[s][0], phis[s][1], len(members))
                    run_end[w], running[w], prepared[w] = e, members, None
                    trace.append((s, index[w], t, e, list(members)))
                    for r in members:
                        state[s][r] = RUNNING
                        end[s][r] = e
                    changed = True
        ends = [e for e in run_end if e is not None]
        if not ends:
            break
        t = min(ends)
        if t > t_stop:
            break
    w0, w1 = window
    span = w1 - w0
    u_num = s_num = 0.0
    rounds_in = 0
    for s, _, a, b, members in trace:
        tau = max(0.0, min(b, w1) - max(a, w0))
        u_num += tau * interp(phis[s][0], phis[s][2], len(members))
        s_num += tau * len(members)
        if s == T and w0 < b <= w1:
            rounds_in += len(members)
    metrics = {"U": u_num / (nw * span), "S": s_num / (n_requests * span),
               "round_rate": rounds_in / span, "finished": finished, "batches": len(trace)}
    return metrics, trace
