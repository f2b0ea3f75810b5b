// Worker-triggered batch reconstruction and the profiling-driven
// discrete-event simulator (host code).
//
// Reconstruction, for a scheduling opportunity of worker w at stage s
// (Section 4, Algorithm 1, Eqs. 4-8; Appendix F.2): every candidate r has an
// available predecessor completion time e~_r (observed, or predicted from a
// running predecessor batch, Eq. 4) and a KV-ready time k^_r; the worker is
// available at a^_w.  Singleton start S({r}) = max(a^_w, e~_r, k^_r) (Eq. 6),
// admission bound d^_r = max(e~_r + g_s, S({r})) + Delta_s (Eq. 7); a batch is
// admissible when |B| <= B_max, its KV blocks and tokens fit the bank, and
// S(B) = max(a^_w, max e~, max k^) <= min d^ over B (Eqs. 5, 6, 8).
// Candidates that do not fit on their own are dropped, the rest ranked by
// (d^_r, S({r}), id), and the first B_max are scanned once in that order,
// each joining if the batch stays admissible.  Selecting the first B_max is a
// partial selection (nth_element), so an opportunity over C candidates costs
// O(C + B_max log B_max).
//
// Simulator (Appendix H): requests start after prefill at t = 0 and run a
// fixed number of rounds, each a draft then a target stage (Eq. 1).  Stage
// times and SM activity are profiled tables interpolated linearly over batch
// sizes; migration is ideal (KV ready at planning time).  Each worker has a
// compute slot and one standby preparation slot.  At every virtual time all
// completions are applied first; then, until nothing changes, every worker
// without a prepared batch (in index order, draft workers first) takes a
// planning opportunity over the requests whose next stage is its stage and
// whose latest predecessor stage is running (predicted end) or done, and every
// idle worker whose prepared batch has all predecessor outputs published
// starts it.  Candidates are kept per stage and updated only when a request is
// prepared (leaves) or its predecessor starts (joins), so an opportunity never
// scans finished or waiting requests.  Metrics are accumulated over the
// window as batches are created (Eqs. H.1, H.2).
#include <algorithm>
#include <cmath>
#include <vector>

#include "nsd_internal.h"

// Results are defined by the written order of operations: no fused multiply-add.
#pragma STDC FP_CONTRACT OFF

namespace {

struct Cand {
  double d, s1;
  int32_t id;
  int32_t i;
};

inline bool rank_less(const Cand& a, const Cand& b) {
  if (a.d != b.d) return a.d < b.d;
  if (a.s1 != b.s1) return a.s1 < b.s1;
  return a.id < b.id;
}

// One opportunity; returns the batch length, writes ids into batch[0..b_max)
// and S(B) into *start (a_hat when empty).  cand is scratch of n entries.
int32_t reconstruct_core(const int32_t* ids, const double* e, const double* k,
                         const int64_t* blocks, const int64_t* tokens, int32_t n, double a_hat,
                         int64_t block_cap, int64_t token_cap, int32_t b_max, double g,
                         double delta, int32_t* batch, double* start, std::vector<Cand>& cand) {
  cand.clear();
  for (int32_t i = 0; i < n; ++i) {
    const int64_t bl = blocks ? blocks[i] : 0, tk = tokens ? tokens[i] : 0;
    if (bl > block_cap || tk > token_cap) continue;
    const double s1 = std::max(std::max(a_hat, e[i]), k[i]);
    const double d = std::max(e[i] + g, s1) + delta;
    cand.push_back({d, s1, ids[i], i});
  }
  const size_t f = std::min(cand.size(), (size_t)b_max);
  if (f < cand.size()) std::nth_element(cand.begin(), cand.begin() + f, cand.end(), rank_less);
  std::sort(cand.begin(), cand.begin() + f, rank_less);
  int32_t len = 0;
  double s_b = a_hat, d_min = INFINITY;
  int64_t used_b = 0, used_t = 0;
  for (size_t j = 0; j < f; ++j) {
    const int32_t i = cand[j].i;
    const int64_t bl = blocks ? blocks[i] : 0, tk = tokens ? tokens[i] : 0;
    const double s_new = std::max(std::max(s_b, e[i]), k[i]);
    const double d_new = std::min(d_min, cand[j].d);
    if (used_b + bl <= block_cap && used_t + tk <= token_cap && s_new <= d_new) {
      batch[len++] = cand[j].id;
      s_b = s_new;
      d_min = d_new;
      used_b += bl;
      used_t += tk;
    }
  }
  *start = s_b;
  return len;
}

struct Table {
  const double *b, *t, *sm;
  int32_t n;
  double at(const double* v, double x) const {
    if (x <= b[0]) return v[0];
    for (int32_t i = 1; i < n; ++i) {
      if (x <= b[i]) {
        const double b0 = b[i - 1], b1 = b[i], v0 = v[i - 1], v1 = v[i];
        return v0 + (v1 - v0) * ((x - b0) / (b1 - b0));
      }
    }
    return v[n - 1];
  }
};

nsd_status check_table(const double* p, int32_t n, const char* name) {
  using namespace nsd;
  if (!p) return fail(NSD_ERR_NULL, "simulate: %s table is NULL", name);
  if (n < 1) return fail(NSD_ERR_SHAPE, "simulate: %s table is empty", name);
  for (int32_t i = 0; i < n; ++i) {
    if (!std::isfinite(p[i]) || !std::isfinite(p[n + i]) || !std::isfinite(p[2 * n + i]) ||
        p[n + i] <= 0.0 || (i > 0 && !(p[i] > p[i - 1])))
      return fail(NSD_ERR_SHAPE, "simulate: %s table needs ascending finite sizes and positive "
                  "finite times (entry %d)", name, i);
  }
  return NSD_OK;
}

// Per-stage candidate set with O(1) insert and remove.
struct CandSet {
  std::vector<int32_t> items, pos;
  explicit CandSet(int32_t n) : pos(n, -1) {}
  void add(int32_t r) {
    if (pos[r] >= 0) return;
    pos[r] = (int32_t)items.size();
    items.push_back(r);
  }
  void remove(int32_t r) {
    const int32_t p = pos[r];
    if (p < 0) return;
    const int32_t last = items.back();
    items[p] = last;
    pos[last] = p;
    items.pop_back();
    pos[r] = -1;
  }
};

}  // namespace

extern "C" nsd_status nsd_reconstruct(const int32_t* ids, const double* e_tilde,
                                      const double* k_hat, const int64_t* blocks,
                                      const int64_t* tokens, int32_t n, double a_hat,
                                      int64_t block_cap, int64_t token_cap, int32_t b_max,
                                      double g, double delta, int32_t* batch, int32_t* batch_len,
                                      double* batch_start) {
  using namespace nsd;
  const char* fn = "reconstruct";
  if (n < 0 || b_max < 1) return fail(NSD_ERR_SHAPE, "%s: n < 0 or b_max < 1", fn);
  if (!batch || !batch_len || !batch_start || (n > 0 && (!ids || !e_tilde || !k_hat)))
    return fail(NSD_ERR_NULL, "%s: NULL pointer argument", fn);
  if (std::isnan(a_hat) || std::isnan(g) || std::isnan(delta) || g < 0 || delta < 0)
    return fail(NSD_ERR_SHAPE, "%s: a_hat, g, delta must be numbers, g and delta >= 0", fn);
  for (int32_t i = 0; i < n; ++i)
    if (std::isnan(e_tilde[i]) || std::isnan(k_hat[i]))
      return fail(NSD_ERR_SHAPE, "%s: candidate %d has a NaN time", fn, i);
  std::vector<Cand> cand;
  cand.reserve(n);
  double s = 0;
  const int32_t len = reconstruct_core(ids, e_tilde, k_hat, blocks, tokens, n, a_hat, block_cap,
                                       token_cap, b_max, g, delta, batch, &s, cand);
  *batch_len = len;
  *batch_start = len ? s : NAN;
  return NSD_OK;
}

extern "C" nsd_status nsd_simulate(const nsd_sim_config* cfg, const double* phi_d,
                                   int32_t n_phi_d, const double* phi_t, int32_t n_phi_t,
                                   nsd_sim_metrics* metrics, nsd_sim_batch* trace,
                                   int64_t trace_cap, int32_t* members, int64_t members_cap,
                                   int64_t* n_trace, int64_t* n_members) {
  using namespace nsd;
  const char* fn = "simulate";
  if (!cfg || !metrics) return fail(NSD_ERR_NULL, "%s: NULL pointer argument", fn);
  const int32_t nd = cfg->n_draft, nt = cfg->n_target, R = cfg->n_requests;
  if (nd < 1 || nt < 1 || R < 0 || cfg->rounds < 0 || cfg->b_max[0] < 1 || cfg->b_max[1] < 1)
    return fail(NSD_ERR_SHAPE, "%s: needs >= 1 worker per pool, b_max >= 1, n_requests and "
                "rounds >= 0", fn);
  for (int s = 0; s < 2; ++s)
    if (!(cfg->g[s] >= 0) || !(cfg->delta[s] >= 0))
      return fail(NSD_ERR_SHAPE, "%s: g and delta must be >= 0", fn);
  if (!(cfg->window[1] > cfg->window[0]) || !std::isfinite(cfg->window[0]) ||
      !std::isfinite(cfg->window[1]) || std::isnan(cfg->t_stop))
    return fail(NSD_ERR_SHAPE, "%s: the window needs w0 < w1, both finite", fn);
  if ((trace_cap > 0 && !trace) || (members_cap > 0 && !members))
    return fail(NSD_ERR_NULL, "%s: trace capacity given without a buffer", fn);
  nsd_status st = check_table(phi_d, n_phi_d, "draft");
  if (st != NSD_OK) return st;
  if ((st = check_table(phi_t, n_phi_t, "target")) != NSD_OK) return st;
  const Table tab[2] = {{phi_d, phi_d + n_phi_d, phi_d + 2 * n_phi_d, n_phi_d},
                        {phi_t, phi_t + n_phi_t, phi_t + 2 * n_phi_t, n_phi_t}};

  enum { NONE = 0, PREPARED = 1, RUNNING = 2, DONE = 3 };
  const int32_t nw = nd + nt;
  const int32_t rounds = cfg->rounds;
  std::vector<int32_t> planned[2] = {std::vector<int32_t>(R, 0), std::vector<int32_t>(R, 0)};
  std::vector<uint8_t> state[2] = {std::vector<uint8_t>(R, NONE), std::vector<uint8_t>(R, DONE)};
  std::vector<double> end[2] = {std::vector<double>(R, 0.0), std::vector<double>(R, 0.0)};
  std::vector<double> run_end(nw, NAN);
  std::vector<std::vector<int32_t>> running(nw), prepared(nw);
  std::vector<uint8_t> has_run(nw, 0), has_prep(nw, 0);
  CandSet cands[2] = {CandSet(R), CandSet(R)};
  for (int32_t r = 0; r < R && rounds > 0; ++r) cands[0].add(r);   // anchors published at t = 0

  std::vector<Cand> scratch;
  std::vector<int32_t> ids, batch;
  std::vector<double> et, kh;
  const double w0 = cfg->window[0], w1 = cfg->window[1], span = w1 - w0;
  double u_num = 0.0, s_num = 0.0;
  int64_t rounds_in = 0, finished = 0, n_batches = 0, n_mem = 0;
  double t = 0.0;
  auto need = [&](int32_t r) -> int {
    if (planned[0][r] == planned[1][r]) return planned[0][r] < rounds ? 0 : -1;
    return 1;
  };

  for (;;) {
    // completions at t
    for (int32_t w = 0; w < nw; ++w) {
      if (!has_run[w] || run_end[w] != t) continue;
      const int s = w < nd ? 0 : 1;
      for (int32_t r : running[w]) {
        state[s][r] = DONE;
        if (s == 1 && planned[1][r] == rounds) ++finished;
      }
      has_run[w] = 0;
      running[w].clear();
    }
    bool changed = true;
    while (changed) {
      changed = false;
      for (int32_t w = 0; w < nw; ++w) {            // planning opportunities
        if (has_prep[w]) continue;
        const int s = w < nd ? 0 : 1, p = 1 - s;
        const std::vector<int32_t>& pool = cands[s].items;
        const int32_t n = (int32_t)pool.size();
        if (n == 0) continue;
        ids.assign(pool.begin(), pool.end());
        et.resize(n);
        kh.assign(n, t);                             // ideal migration
        for (int32_t i = 0; i < n; ++i) et[i] = end[p][ids[i]];
        batch.resize(cfg->b_max[s]);
        const double a_hat = has_run[w] ? run_end[w] : t;
        double sb;
        const int32_t len = reconstruct_core(ids.data(), et.data(), kh.data(), nullptr, nullptr,
                                             n, a_hat, 0, 0, cfg->b_max[s], cfg->g[s],
                                             cfg->delta[s], batch.data(), &sb, scratch);
        if (len == 0) continue;
        prepared[w].assign(batch.begin(), batch.begin() + len);
        has_prep[w] = 1;
        for (int32_t r : prepared[w]) {
          ++planned[s][r];
          state[s][r] = PREPARED;
          cands[s].remove(r);
        }
        changed = true;
      }
      for (int32_t w = 0; w < nw; ++w) {            // progress: InputReady and WorkerReady
        if (!has_prep[w] || has_run[w]) continue;
        const int s = w < nd ? 0 : 1;
        bool ready = true;
        for (int32_t r : prepared[w]) ready = ready && state[1 - s][r] == DONE;
        if (!ready) continue;
        const int32_t b = (int32_t)prepared[w].size();
        const double e = t + tab[s].at(tab[s].t, (double)b);
        running[w].swap(prepared[w]);
        prepared[w].clear();
        has_prep[w] = 0;
        has_run[w] = 1;
        run_end[w] = e;
        for (int32_t r : running[w]) {
          state[s][r] = RUNNING;
          end[s][r] = e;
          if (need(r) == 1 - s) cands[1 - s].add(r);   // its successor can now be planned
        }
        // metrics and trace, in creation order
        const double tau = std::max(0.0, std::min(e, w1) - std::max(t, w0));
        u_num += tau * tab[s].at(tab[s].sm, (double)b);
        s_num += tau * (double)b;
        if (s == 1 && w0 < e && e <= w1) rounds_in += b;
        if (n_batches < trace_cap && n_mem + b <= members_cap) {
          trace[n_batches] = {s, s == 0 ? w : w - nd, b, n_mem, t, e};
          std::copy(running[w].begin(), running[w].end(), members + n_mem);
        } else if (trace_cap > 0) {
          trace_cap = -trace_cap;                      // out of room: stop recording
        }
        ++n_batches;
        n_mem += b;
        changed = true;
      }
    }
    double next = INFINITY;
    for (int32_t w = 0; w < nw; ++w)
      if (has_run[w]) next = std::min(next, run_end[w]);
    if (next == INFINITY) break;
    t = next;
    if (t > cfg->t_stop) break;
  }
  metrics->U = u_num / ((double)nw * span);
  metrics->S = R > 0 ? s_num / ((double)R * span) : 0.0;
  metrics->round_rate = (double)rounds_in / span;
  metrics->finished = finished;
  metrics->batches = n_batches;
  if (n_trace) *n_trace = n_batches;
  if (n_members) *n_members = n_mem;
  if (trace_cap < 0)
    return fail(NSD_ERR_WORKSPACE, "%s: the trace needs %lld batches and %lld members", fn,
                (long long)n_batches, (long long)n_mem);
  return NSD_OK;
}
