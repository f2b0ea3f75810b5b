// Verification attention: every request's anchor + K proposal queries attend,
// causally, to its paged KV cache (Section 1: one target forward verifies all
// proposals; Appendix G.2/H: anchor plus depth-d proposals; Section 3: paged,
// append-dominant cache that already holds the window).
//
// Design (gfx950, wave64, bf16 MFMA 16x16x32):
// * The (Hq/Hkv) query heads x n_q queries that share KV head g form the M rows
//   of one wave's tile products, so each K/V byte is read from HBM once for the
//   whole group.
// * S^T = K Q^T: the K plane's [D/8][16][8] run layout puts, for MFMA k-step
//   kk, the 16 slots x 8 dims that lane group (lane/16) needs in one 256-byte
//   run: K operands are loaded straight from HBM into registers, 16 bytes per
//   lane, 1 KiB contiguous per wave instruction.  The accumulator gives each
//   lane 4 tokens of one query row (row = lane%16), so the row max needs two
//   cross-lane steps and the row sum none until the end.
// * O^T = V^T P^T: the V plane's [D][16] layout makes V^T rows contiguous, so
//   V operands also load straight into registers (8 bytes per lane, 512 B
//   contiguous per instruction), and P^T is exactly the S^T accumulator
//   layout (converted to bf16), with no data exchange between lanes.  O^T
//   accumulates per lane for one query row, so the online-softmax rescale is
//   lane-local.  No LDS round trip is needed for either operand.
// * K/V are streamed once, so they are loaded non-temporally.
// * Load balance (stream-K): the spans of all (request, KV head) items are cut
//   into as many equal contiguous ranges as the device keeps waves resident,
//   whatever the spread of context lengths.  Items cut by a range boundary
//   leave partials that a small second kernel merges in wave order
//   (deterministic, no atomics); all other items are written directly.
// * Masked tokens (past a query's position, past L_r, or in a block whose id
//   is out of range) are removed by selection: scores become -inf and V
//   elements past L_r are zeroed, so NaN-filled unused slots never leak.
#include "nsd_internal.h"

#include <math.h>
#include <stdlib.h>

#include <algorithm>

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

constexpr int kBlock = 16;   // token slots per KV block
constexpr int kSpan = 32;    // tokens per main-loop step
constexpr int kMaxRows = 64; // (Hq/Hkv) * max_q_per_seq limit
constexpr int kMaxBatch = 8192;   // the span prefix of the batch lives in LDS

struct Params {
  const uint16_t* q;
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  const int32_t* block_table;
  const int32_t* seq_lens;
  const int32_t* q_indptr;
  uint16_t* out;
  float* part_o;     // [2 * num_waves][MT*16][D]: head/tail partial O per wave
  float2* part_ml;   // [2 * num_waves][MT*16]: (running max, sum)
  uint32_t* prefix;    // [bs+1]: exclusive prefix of per-request span counts
  uint32_t* counters;  // [1]: next dynamic chunk to claim (zero between dispatches)
  int64_t num_blocks;
  int32_t bs;
  int32_t max_blocks_per_seq;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t group;
  int32_t max_q;
  int32_t max_seq_len;
  int32_t num_waves;
  float scale_log2;  // softmax scale * log2(e)
};

template <int D>
struct KOps {
  u32x4 k[2][D / 32];   // K operands of a span's two blocks
};

template <int D>
struct VOps {
  u32x2 v[2][D / 16];   // V^T operand halves of a span's two blocks
};

struct SpanRef {
  int64_t hb0, hb1;     // element offsets of the two blocks' (block, KV head) tiles
  int32_t t;            // first token of the span
  bool bad0, bad1;      // block id out of range
};

__device__ inline float wave_max_groups(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  return fmaxf(x, __shfl_xor(x, 32));
}

__device__ inline float wave_sum_groups(float x) {
  x += __shfl_xor(x, 16);
  return x + __shfl_xor(x, 32);
}

__device__ inline uint32_t keep_mask(int n_valid_elems) {
  // mask for one 32-bit word holding two bf16 (element 0 in the low half)
  return n_valid_elems <= 0 ? 0u : (n_valid_elems == 1 ? 0x0000ffffu : 0xffffffffu);
}

// The span of the request starting at token t (blocks t/16 and t/16 + 1).
// Block ids are wave-uniform, so they are fetched with scalar loads, which
// keep the vector-memory counter free for the K/V stream.
template <int D>
__device__ inline SpanRef span_ref(const Params& p, const int32_t* __restrict__ bt, int t, int L,
                                   int g) {
  SpanRef s;
  s.t = t;
  const int b0 = t / kBlock;
  const bool has1 = t + kBlock < L;
  int32_t id0 = bt[b0];
  int32_t id1 = has1 ? bt[b0 + 1] : id0;
  s.bad0 = id0 < 0 || id0 >= p.num_blocks;
  if (s.bad0) id0 = 0;
  const bool bad1 = id1 < 0 || id1 >= p.num_blocks;
  s.bad1 = has1 && bad1;
  if (!has1 || bad1) id1 = id0;
  s.hb0 = ((int64_t)id0 * p.num_kv_heads + g) * (D * kBlock);
  s.hb1 = ((int64_t)id1 * p.num_kv_heads + g) * (D * kBlock);
  return s;
}

template <int D>
__device__ inline void load_k(KOps<D>& o, const uint16_t* kc, const SpanRef& s, int lane) {
  const int row = lane & 15, grp = lane >> 4;
  const uint16_t* k0 = kc + s.hb0;
  const uint16_t* k1 = kc + s.hb1;
#pragma unroll
  for (int kk = 0; kk < D / 32; ++kk) {
    const int off = ((kk * 4 + grp) * kBlock + row) * 8;
    o.k[0][kk] = __builtin_nontemporal_load((const u32x4*)(k0 + off));
    o.k[1][kk] = __builtin_nontemporal_load((const u32x4*)(k1 + off));
  }
}

template <int D>
__device__ inline void load_v(VOps<D>& o, const uint16_t* vc, const SpanRef& s, int lane) {
  const int row = lane & 15, grp = lane >> 4;
  const uint16_t* v0 = vc + s.hb0;
  const uint16_t* v1 = vc + s.hb1;
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const int off = (dt * 16 + row) * kBlock + grp * 4;
    o.v[0][dt] = __builtin_nontemporal_load((const u32x2*)(v0 + off));
    o.v[1][dt] = __builtin_nontemporal_load((const u32x2*)(v1 + off));
  }
}

// S^T[token][row] of the span's two blocks.  Q operands come from this
// wave's LDS copy, stored in operand order: one 16-byte run per lane per
// (row tile, k-step), so every read is conflict-free.
template <int D, int MT>
__device__ inline void span_scores(const KOps<D>& k, const u32x4* qlds, int lane,
                                   f32x4 (&st)[2][MT]) {
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    f32x4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = c0;
#pragma unroll
    for (int kk = 0; kk < D / 32; ++kk) {
      const bf16x8 qo = __builtin_bit_cast(bf16x8, qlds[(mt * (D / 32) + kk) * 64 + lane]);
      c0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, k.k[0][kk]), qo,
                                                   c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, k.k[1][kk]), qo,
                                                   c1, 0, 0, 0);
    }
    st[0][mt] = c0;
    st[1][mt] = c1;
  }
}

// Online-softmax update from one span's scores; returns P^T operands (bf16).
template <int D, int MT>
__device__ inline void span_softmax(const f32x4 (&st)[2][MT], const SpanRef& s,
                                    f32x4 (&acc)[MT][D / 16], float (&m_run)[MT],
                                    float (&l_run)[MT], const int (&pos)[MT], int win,
                                    float scale_log2, int lane, bf16x8 (&pop)[MT]) {
  const int grp = lane >> 4;
  const bool need_mask = (s.t + kSpan > win) || s.bad0 || s.bad1;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    float x[2][4];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int i = 0; i < 4; ++i) x[h][i] = st[h][mt][i] * scale_log2;
    if (need_mask) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const bool bad = h ? s.bad1 : s.bad0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = s.t + h * kBlock + grp * 4 + i;
          x[h][i] = (t <= pos[mt] && !bad) ? x[h][i] : -INFINITY;
        }
      }
    }
    float mx = x[0][0];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int i = 0; i < 4; ++i) mx = fmaxf(mx, x[h][i]);
    mx = wave_max_groups(mx);
    const float m_new = fmaxf(m_run[mt], mx);
    const bool none = m_new == -INFINITY;
    const float alpha = none ? 1.f : __builtin_amdgcn_exp2f(m_run[mt] - m_new);
    const float msub = none ? 0.f : m_new;
    float pr[2][4];
    float psum = 0.f;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pr[h][i] = __builtin_amdgcn_exp2f(x[h][i] - msub);
        psum += pr[h][i];
      }
    l_run[mt] = l_run[mt] * alpha + psum;
    m_run[mt] = m_new;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) acc[mt][dt] *= alpha;
    pop[mt] = bf16x8{(__bf16)pr[0][0], (__bf16)pr[0][1], (__bf16)pr[0][2], (__bf16)pr[0][3],
                     (__bf16)pr[1][0], (__bf16)pr[1][1], (__bf16)pr[1][2], (__bf16)pr[1][3]};
  }
}

// O^T += V^T P^T; V elements of tokens >= L (or of bad blocks) are zeroed.
template <int D, int MT>
__device__ inline void span_pv(const VOps<D>& v, const SpanRef& s, int L,
                               const bf16x8 (&pop)[MT], f32x4 (&acc)[MT][D / 16], int lane) {
  const int grp = lane >> 4;
  uint32_t keep[4] = {0xffffffffu, 0xffffffffu, 0xffffffffu, 0xffffffffu};
  if (s.t + kSpan > L || s.bad0 || s.bad1) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const bool bad = h ? s.bad1 : s.bad0;
      const int nv = bad ? 0 : min(4, max(0, L - (s.t + h * kBlock + grp * 4)));
      keep[2 * h] = keep_mask(nv);
      keep[2 * h + 1] = keep_mask(nv - 2);
    }
  }
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const u32x4 w = {v.v[0][dt].x & keep[0], v.v[0][dt].y & keep[1], v.v[1][dt].x & keep[2],
                     v.v[1][dt].y & keep[3]};
    const bf16x8 vop = __builtin_bit_cast(bf16x8, w);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
      acc[mt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pop[mt], acc[mt][dt], 0, 0, 0);
  }
}

__device__ inline int clamp_len(const Params& p, const int32_t* __restrict__ seq_lens, int r) {
  const int L = seq_lens[r];
  return max(0, min(L, min(p.max_seq_len, p.max_blocks_per_seq * kBlock)));
}

// Spans of one (request, KV head) item; an empty context still owns one span
// so that its rows are written (as zeros).
__device__ inline int spans_of(int L) { return max(1, (L + kSpan - 1) / kSpan); }

// Values every lane of a wave agrees on, marked so for the compiler (uniform
// values live in scalar registers and their loads become scalar loads).
__device__ inline int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ inline int64_t uniform64(int64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ inline int64_t wave_sum_i64(int64_t x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

__device__ inline int64_t wave_incl_scan_i64(int64_t x, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  return x;
}

constexpr int kStaticPct = 100;  // share of spans split evenly over the waves up front
constexpr int kChunkSpans = 8;   // spans per dynamically claimed chunk

// The global sequence of T spans (ordered by request, then KV head, then
// position) is cut into ranges: W static ranges covering the first Ts spans
// evenly, one per wave, then C dynamic chunks of kChunkSpans spans that waves
// claim from a counter once their static range is done.  Waves on slower
// paths to memory (the XCDs differ) thereby end together.  Every kernel
// derives the same ranges from T and W.
struct Ranges {
  int64_t T, Ts, W, C;
  __device__ Ranges(int64_t total, int64_t waves) : T(total), W(waves) {
    Ts = total * kStaticPct / 100;
    C = (total - Ts + kChunkSpans - 1) / kChunkSpans;
  }
  __device__ int64_t begin(int64_t rid) const {
    return rid < W ? rid * Ts / W : Ts + (rid - W) * kChunkSpans;
  }
  __device__ int64_t end(int64_t rid) const {
    return rid < W ? (rid + 1) * Ts / W : min(T, Ts + (rid - W + 1) * kChunkSpans);
  }
  // range holding span s
  __device__ int64_t of(int64_t s) const {
    return s < Ts ? ((s + 1) * W - 1) / Ts : W + (s - Ts) / kChunkSpans;
  }
};

// Request whose spans [hkv*pre[r], hkv*pre[r+1]) contain global span s.
__device__ inline int find_request(const uint32_t* pre, int bs, int hkv, int64_t s) {
  int lo = 0, hi = bs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if ((int64_t)hkv * pre[mid] <= s) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// One span: S from K, online softmax, PV from V; with LOADS the registers
// each phase has consumed are refilled at once with the span `nr`.
template <int D, int MT, bool LOADS>
__device__ inline void span_step(KOps<D>& kr, VOps<D>& vr, const SpanRef& sr, const SpanRef& nr,
                                 const u32x4* qlds, const Params& p, f32x4 (&acc)[MT][D / 16],
                                 float (&m_run)[MT], float (&l_run)[MT], const int (&pos)[MT],
                                 int win, int L, int lane) {
  f32x4 st[2][MT];
  span_scores<D, MT>(kr, qlds, lane, st);
  if constexpr (LOADS) load_k<D>(kr, p.k_cache, nr, lane);
  bf16x8 pop[MT];
  span_softmax<D, MT>(st, sr, acc, m_run, l_run, pos, win, p.scale_log2, lane, pop);
  span_pv<D, MT>(vr, sr, L, pop, acc, lane);
  if constexpr (LOADS) load_v<D>(vr, p.v_cache, nr, lane);
}

// One range [s, s1) of global spans, range id rid: online softmax over every
// (request, KV head) item the range touches.  An item wholly inside the range
// is finished and written; an item cut by a range boundary leaves a partial
// (running max, sum, unnormalised O) in the range's head slot (the item began
// in an earlier range) or tail slot (it continues in a later one).
template <int D, int MT, int DEPTH>
__device__ void process_range(const Params& p, const int32_t* __restrict__ block_table,
                              const int32_t* __restrict__ seq_lens,
                              const int32_t* __restrict__ q_indptr, const uint32_t* pre,
                              u32x4* qlds, int64_t rid, int64_t s, int64_t s1, int lane) {
  const int grp = lane >> 4;
  const int hkv = p.num_kv_heads;
  int r = uniform(find_request(pre, p.bs, hkv, s));
  int64_t pr = pre[r];
  while (s < s1) {
    __builtin_amdgcn_wave_barrier();
    const int L = clamp_len(p, seq_lens, r);
    const int n = spans_of(L);
    const int qo = q_indptr[r];
    const int nq = max(0, min(q_indptr[r + 1] - qo, p.max_q));
    const int64_t off = s - hkv * pr;
    const int g = (int)(off / n);
    const int j0 = (int)(off - (int64_t)g * n);
    const int j1 = (int)min((int64_t)n, j0 + (s1 - s));
    const int rows = p.group * nq;
    const int win = L - nq;

    int pos[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = mt * 16 + (lane & 15);
      if (m < rows) {
        const int j = m / p.group;
        const int h = g * p.group + m % p.group;
        const uint16_t* src = p.q + ((int64_t)(qo + j) * p.num_q_heads + h) * D;
#pragma unroll
        for (int kk = 0; kk < D / 32; ++kk)
          qlds[(mt * (D / 32) + kk) * 64 + lane] = *(const u32x4*)(src + kk * 32 + grp * 8);
        pos[mt] = win + j;
      } else {
#pragma unroll
        for (int kk = 0; kk < D / 32; ++kk)
          qlds[(mt * (D / 32) + kk) * 64 + lane] = u32x4{0, 0, 0, 0};
        pos[mt] = L - 1;
      }
    }
    __builtin_amdgcn_wave_barrier();
    f32x4 acc[MT][D / 16];
    float m_run[MT], l_run[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      m_run[mt] = -INFINITY;
      l_run[mt] = 0.f;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) acc[mt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // Software pipeline over spans.  With DEPTH = 1, K(j+1) is requested as
    // soon as S(j) has consumed K(j) and V(j+1) as soon as PV(j) has consumed
    // V(j); with DEPTH = 2 (when registers allow only one wave per SIMD anyway)
    // two buffers alternate and spans j+1 and j+2 are in flight during span j.
    // Loads inside the loops are unconditional (tails are peeled): a
    // conditional load would force a full drain of the load counter per span.
    const int32_t* __restrict__ bt = block_table + (int64_t)r * p.max_blocks_per_seq;
#define NSD_STEP(LOADS, KR, VR, SR, NR)                                                         \
  span_step<D, MT, LOADS>(KR, VR, SR, NR, qlds, p, acc, m_run, l_run, pos, win, L, lane)
    if constexpr (DEPTH == 1) {
      SpanRef cur = span_ref<D>(p, bt, j0 * kSpan, L, g);
      KOps<D> kreg;
      VOps<D> vreg;
      load_k<D>(kreg, p.k_cache, cur, lane);
      load_v<D>(vreg, p.v_cache, cur, lane);
      for (int j = j0; j + 1 < j1; ++j) {
        const SpanRef nxt = span_ref<D>(p, bt, (j + 1) * kSpan, L, g);
        NSD_STEP(true, kreg, vreg, cur, nxt);
        cur = nxt;
      }
      NSD_STEP(false, kreg, vreg, cur, cur);
    } else {
      SpanRef ra = span_ref<D>(p, bt, j0 * kSpan, L, g);
      SpanRef rb = ra;
      KOps<D> ka, kb;
      VOps<D> va, vb;
      load_k<D>(ka, p.k_cache, ra, lane);
      load_v<D>(va, p.v_cache, ra, lane);
      if (j0 + 1 < j1) {
        rb = span_ref<D>(p, bt, (j0 + 1) * kSpan, L, g);
        load_k<D>(kb, p.k_cache, rb, lane);
        load_v<D>(vb, p.v_cache, rb, lane);
      }
      int j = j0;
      for (; j + 3 < j1; j += 2) {
        const SpanRef na = span_ref<D>(p, bt, (j + 2) * kSpan, L, g);
        NSD_STEP(true, ka, va, ra, na);
        const SpanRef nb = span_ref<D>(p, bt, (j + 3) * kSpan, L, g);
        NSD_STEP(true, kb, vb, rb, nb);
        ra = na;
        rb = nb;
      }
      const int rem = j1 - j;
      if (rem == 3) {
        const SpanRef na = span_ref<D>(p, bt, (j + 2) * kSpan, L, g);
        NSD_STEP(true, ka, va, ra, na);
        NSD_STEP(false, kb, vb, rb, rb);
        NSD_STEP(false, ka, va, na, na);
      } else if (rem == 2) {
        NSD_STEP(false, ka, va, ra, ra);
        NSD_STEP(false, kb, vb, rb, rb);
      } else {
        NSD_STEP(false, ka, va, ra, ra);
      }
    }
#undef NSD_STEP
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) l_run[mt] = wave_sum_groups(l_run[mt]);

    if (j0 == 0 && j1 == n) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = mt * 16 + (lane & 15);
        if (m >= rows) continue;
        const int j = m / p.group;
        const int h = g * p.group + m % p.group;
        const float inv = l_run[mt] > 0.f ? 1.f / l_run[mt] : 0.f;
        uint16_t* dst = p.out + ((int64_t)(qo + j) * p.num_q_heads + h) * D + grp * 4;
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt) {
          const bf16x2 lo = {(__bf16)(acc[mt][dt][0] * inv), (__bf16)(acc[mt][dt][1] * inv)};
          const bf16x2 hi = {(__bf16)(acc[mt][dt][2] * inv), (__bf16)(acc[mt][dt][3] * inv)};
          *(u32x2*)(dst + dt * 16) = u32x2{__builtin_bit_cast(uint32_t, lo),
                                           __builtin_bit_cast(uint32_t, hi)};
        }
      }
    } else {
      const int64_t slot = 2 * rid + (j0 > 0 ? 0 : 1);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = mt * 16 + (lane & 15);
        if (m >= rows) continue;
        float* dst = p.part_o + (slot * (MT * 16) + m) * D + grp * 4;
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt) *(f32x4*)(dst + dt * 16) = acc[mt][dt];
        if (grp == 0) p.part_ml[slot * (MT * 16) + m] = make_float2(m_run[mt], l_run[mt]);
      }
    }
    s += j1 - j0;
    if (j1 == n && g == hkv - 1) {
      pr += n;
      ++r;
    }
  }
}

// One dispatch of W waves (W / 4 workgroups of 4 independent waves).
template <int D, int MT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(D * MT <= 128 ? 2 : 1)))
void verify_attention_kernel(Params p, const int32_t* __restrict__ block_table,
                             const int32_t* __restrict__ seq_lens,
                             const int32_t* __restrict__ q_indptr) {
  extern __shared__ uint32_t s_pre[];        // [bs + 1]: exclusive prefix of per-request spans
  __shared__ uint32_t s_wsum[4];
  __shared__ u32x4 s_q[4][MT * (D / 32) * 64];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = uniform(tid >> 6);

  // prefix of per-request span counts (every workgroup keeps its own copy)
  uint32_t carry = 0;
  for (int base = 0; base < p.bs; base += 256) {
    const int r = base + tid;
    const uint32_t n = r < p.bs ? spans_of(clamp_len(p, seq_lens, r)) : 0;
    uint32_t incl = n;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(incl, o);
      if (lane >= o) incl += y;
    }
    if (lane == 63) s_wsum[wave] = incl;
    __syncthreads();
    uint32_t before = carry;
    for (int i = 0; i < wave; ++i) before += s_wsum[i];
    if (r < p.bs) {
      s_pre[r] = before + incl - n;
      if (blockIdx.x == 0) p.prefix[r] = before + incl - n;
    }
    carry += s_wsum[0] + s_wsum[1] + s_wsum[2] + s_wsum[3];
    __syncthreads();
  }
  if (tid == 0) {
    s_pre[p.bs] = carry;
    if (blockIdx.x == 0) p.prefix[p.bs] = carry;
  }
  __syncthreads();

  const Ranges R((int64_t)p.num_kv_heads * carry, p.num_waves);
  const int64_t w = (int64_t)blockIdx.x * 4 + wave;
  u32x4* qlds = s_q[wave];
  int64_t rid = w;
  while (true) {
    const int64_t b = uniform64(R.begin(rid)), e = uniform64(R.end(rid));
    if (b < e)
      process_range<D, MT, 1>(p, block_table, seq_lens, q_indptr, s_pre,
                                                     qlds, rid, b, e, lane);
    uint32_t c = 0;
    if (lane == 0)
      c = __hip_atomic_fetch_add(p.counters, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    c = uniform(__shfl(c, 0));
    if (c >= R.C) break;
    rid = R.W + c;
  }
}

// Merge the partials of every item that a range boundary cut, in range order
// (deterministic, no atomics).
template <int D, int MT>
__global__ __launch_bounds__(256) void combine_kernel(Params p) {
  const int g = blockIdx.x;
  const int r = blockIdx.y;
  // the attention dispatch has finished: rewind its chunk counter for the next one
  if (g == 0 && r == 0 && threadIdx.x == 0) *p.counters = 0;
  const int hkv = p.num_kv_heads;
  const Ranges R((int64_t)hkv * p.prefix[p.bs], p.num_waves);
  const int L = clamp_len(p, p.seq_lens, r);
  const int n = spans_of(L);
  const int qo = p.q_indptr[r];
  const int nq = max(0, min(p.q_indptr[r + 1] - qo, p.max_q));
  const int64_t a = (int64_t)p.prefix[r] * hkv + (int64_t)g * n;
  const int64_t ra = R.of(a);
  const int64_t rb = R.of(a + n - 1);
  if (ra == rb || nq == 0) return;
  const int rows = p.group * nq;
  constexpr int kVec = D / 4;
  for (int idx = threadIdx.x; idx < rows * kVec; idx += blockDim.x) {
    const int m = idx / kVec;
    const int d = (idx % kVec) * 4;
    float mx = -INFINITY;
    for (int64_t q = ra; q <= rb; ++q) {
      if (R.begin(q) >= R.end(q)) continue;
      const int64_t slot = 2 * q + (q == ra ? 1 : 0);
      mx = fmaxf(mx, p.part_ml[slot * (MT * 16) + m].x);
    }
    f32x4 num = {0.f, 0.f, 0.f, 0.f};
    float den = 0.f;
    for (int64_t q = ra; q <= rb; ++q) {
      if (R.begin(q) >= R.end(q)) continue;
      const int64_t slot = 2 * q + (q == ra ? 1 : 0);
      const float2 ml = p.part_ml[slot * (MT * 16) + m];
      const float wt = (ml.x == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(ml.x - mx);
      const f32x4 o = *(const f32x4*)(p.part_o + (slot * (MT * 16) + m) * D + d);
      num += wt * o;
      den += wt * ml.y;
    }
    const float inv = den > 0.f ? 1.f / den : 0.f;
    const int j = m / p.group;
    const int h = g * p.group + m % p.group;
    uint16_t* dst = p.out + ((int64_t)(qo + j) * p.num_q_heads + h) * D + d;
    const bf16x2 lo = {(__bf16)(num[0] * inv), (__bf16)(num[1] * inv)};
    const bf16x2 hi = {(__bf16)(num[2] * inv), (__bf16)(num[3] * inv)};
    *(u32x2*)dst = u32x2{__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
  }
}

template <int D, int MT>
const void* kernel_ptr() {
  return (const void*)&verify_attention_kernel<D, MT>;
}

const void* kernel_for(int d, int mt) {
  if (d == 64) {
    switch (mt) {
      case 1: return kernel_ptr<64, 1>();
      case 2: return kernel_ptr<64, 2>();
      case 3: return kernel_ptr<64, 3>();
      default: return kernel_ptr<64, 4>();
    }
  }
  switch (mt) {
    case 1: return kernel_ptr<128, 1>();
    case 2: return kernel_ptr<128, 2>();
    case 3: return kernel_ptr<128, 3>();
    default: return kernel_ptr<128, 4>();
  }
}

struct Plan {
  int mt;            // 16-row tiles
  int num_waves;     // W: resident waves of the launch
  int64_t max_chunks;
  size_t lds_bytes;  // dynamic LDS: the span prefix
  size_t counter_bytes, prefix_bytes, part_o_bytes, part_ml_bytes, ws_bytes;
};

// Waves the device keeps resident for this kernel (CUs x waves per CU), or
// NSD_ATTN_WAVES when set (a multiple of 4, for tests and tuning).
int resident_waves(int d, int mt) {
  const char* env = getenv("NSD_ATTN_WAVES");
  if (env) {
    const int v = atoi(env);
    if (v >= 4 && v % 4 == 0) return v;
  }
  int dev = 0, cus = 0, blocks = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, kernel_for(d, mt), 256, 0) !=
          hipSuccess ||
      cus <= 0 || blocks <= 0) {
    (void)hipGetLastError();
    cus = 256;
    blocks = 2;
  }
  return cus * blocks * 4;
}

bool make_plan(int bs, int hq, int hkv, int d, int max_q, int max_seq_len, Plan* pl) {
  if (bs < 0 || bs > kMaxBatch || hq < 1 || hkv < 1 || hq % hkv || (d != 64 && d != 128) ||
      max_q < 1 || max_seq_len < 0)
    return false;
  const int rows = (hq / hkv) * max_q;
  if (rows > kMaxRows) return false;
  pl->mt = (rows + 15) / 16;
  pl->num_waves = resident_waves(d, pl->mt);
  // upper bound of the dynamic chunks: at most 1 + (100-kStaticPct)% of the spans
  const int64_t max_spans = (int64_t)hkv * bs * std::max(1, (max_seq_len + kSpan - 1) / kSpan);
  pl->max_chunks = (max_spans - max_spans * kStaticPct / 100 + kChunkSpans - 1) / kChunkSpans + 1;
  const size_t slots = 2 * ((size_t)pl->num_waves + (size_t)pl->max_chunks) * pl->mt * 16;
  pl->lds_bytes = ((size_t)bs + 1) * sizeof(uint32_t);
  pl->counter_bytes = 256;
  pl->prefix_bytes = (((size_t)bs + 1) * sizeof(uint32_t) + 255) / 256 * 256;
  pl->part_o_bytes = slots * d * sizeof(float);
  pl->part_ml_bytes = slots * sizeof(float2);
  pl->ws_bytes = pl->counter_bytes + pl->prefix_bytes + pl->part_o_bytes + pl->part_ml_bytes;
  return true;
}

template <int D, int MT>
void launch(const Params& p, int bs, hipStream_t stream) {
  hipLaunchKernelGGL((verify_attention_kernel<D, MT>), dim3(p.num_waves / 4), dim3(256),
                     ((size_t)bs + 1) * sizeof(uint32_t), stream, p, p.block_table, p.seq_lens,
                     p.q_indptr);
  hipLaunchKernelGGL((combine_kernel<D, MT>), dim3(p.num_kv_heads, bs), dim3(256), 0, stream, p);
}

template <int D>
void launch_d(const Params& p, int mt, int bs, hipStream_t stream) {
  switch (mt) {
    case 1: launch<D, 1>(p, bs, stream); break;
    case 2: launch<D, 2>(p, bs, stream); break;
    case 3: launch<D, 3>(p, bs, stream); break;
    default: launch<D, 4>(p, bs, stream); break;
  }
}

}  // namespace

extern "C" size_t nsd_verify_attention_workspace_size(int32_t bs, int32_t num_q_heads,
                                                      int32_t num_kv_heads, int32_t head_dim,
                                                      int32_t max_q_per_seq,
                                                      int32_t max_seq_len) {
  Plan pl;
  if (!make_plan(bs, num_q_heads, num_kv_heads, head_dim, max_q_per_seq, max_seq_len, &pl))
    return 0;
  return pl.ws_bytes;
}

extern "C" nsd_status nsd_verify_attention(const void* q, const void* k_cache,
                                           const void* v_cache, int64_t num_blocks,
                                           const int32_t* block_table,
                                           int32_t max_blocks_per_seq, const int32_t* seq_lens,
                                           const int32_t* q_indptr, int32_t bs,
                                           int32_t num_q_heads, int32_t num_kv_heads,
                                           int32_t head_dim, int32_t block_size,
                                           int32_t max_q_per_seq, int32_t max_seq_len,
                                           float scale, void* out, void* workspace,
                                           size_t workspace_bytes, void* stream) {
  using namespace nsd;
  if (bs < 0 || bs > kMaxBatch)
    return fail(NSD_ERR_SHAPE, "verify_attention: bs must be in [0, %d]", kMaxBatch);
  if (block_size != NSD_BLOCK_SIZE)
    return fail(NSD_ERR_UNSUPPORTED, "verify_attention: block_size must be 16 (got %d)", block_size);
  if (head_dim != 64 && head_dim != 128)
    return fail(NSD_ERR_UNSUPPORTED, "verify_attention: head_dim must be 64 or 128 (got %d)",
                head_dim);
  if (num_q_heads < 1 || num_kv_heads < 1 || num_q_heads % num_kv_heads)
    return fail(NSD_ERR_SHAPE, "verify_attention: num_q_heads (%d) must be a positive multiple "
                "of num_kv_heads (%d)", num_q_heads, num_kv_heads);
  if (max_q_per_seq < 1) return fail(NSD_ERR_SHAPE, "verify_attention: max_q_per_seq < 1");
  if ((num_q_heads / num_kv_heads) * max_q_per_seq > kMaxRows)
    return fail(NSD_ERR_UNSUPPORTED, "verify_attention: (Hq/Hkv)*max_q_per_seq = %d exceeds %d",
                (num_q_heads / num_kv_heads) * max_q_per_seq, kMaxRows);
  if (max_seq_len < 1 || max_blocks_per_seq < 1 || num_blocks < 1)
    return fail(NSD_ERR_SHAPE, "verify_attention: max_seq_len, max_blocks_per_seq and "
                "num_blocks must be >= 1");
  if (!(scale == scale) || isinf(scale))
    return fail(NSD_ERR_SHAPE, "verify_attention: scale must be finite");
  if (bs == 0) return NSD_OK;
  if (!q || !k_cache || !v_cache || !block_table || !seq_lens || !q_indptr || !out)
    return fail(NSD_ERR_NULL, "verify_attention: NULL pointer argument");
  Plan pl;
  make_plan(bs, num_q_heads, num_kv_heads, head_dim, max_q_per_seq, max_seq_len, &pl);
  if (!workspace || workspace_bytes < pl.ws_bytes)
    return fail(NSD_ERR_WORKSPACE, "verify_attention: workspace of %zu bytes needed, %zu given",
                pl.ws_bytes, workspace ? workspace_bytes : (size_t)0);

  int dev = 0, lds_max = 0;
  hipFuncAttributes fa;
  if (hipGetDevice(&dev) == hipSuccess &&
      hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) ==
          hipSuccess &&
      hipFuncGetAttributes(&fa, kernel_for(head_dim, pl.mt)) == hipSuccess &&
      fa.sharedSizeBytes + pl.lds_bytes > (size_t)lds_max)
    return fail(NSD_ERR_UNSUPPORTED, "verify_attention: bs=%d needs %zu bytes of LDS, %d available",
                bs, fa.sharedSizeBytes + pl.lds_bytes, lds_max);
  (void)hipGetLastError();

  Params p;
  p.q = (const uint16_t*)q;
  p.k_cache = (const uint16_t*)k_cache;
  p.v_cache = (const uint16_t*)v_cache;
  p.block_table = block_table;
  p.seq_lens = seq_lens;
  p.q_indptr = q_indptr;
  p.out = (uint16_t*)out;
  p.counters = (uint32_t*)workspace;
  p.prefix = (uint32_t*)((char*)workspace + pl.counter_bytes);
  p.part_o = (float*)((char*)workspace + pl.counter_bytes + pl.prefix_bytes);
  p.part_ml = (float2*)((char*)workspace + pl.counter_bytes + pl.prefix_bytes + pl.part_o_bytes);
  p.num_blocks = num_blocks;
  p.bs = bs;
  p.max_blocks_per_seq = max_blocks_per_seq;
  p.num_q_heads = num_q_heads;
  p.num_kv_heads = num_kv_heads;
  p.group = num_q_heads / num_kv_heads;
  p.max_q = max_q_per_seq;
  p.max_seq_len = max_seq_len;
  p.num_waves = pl.num_waves;
  p.scale_log2 = scale * 1.4426950408889634f;

  clear_stale_error();
  if (head_dim == 64)
    launch_d<64>(p, pl.mt, bs, (hipStream_t)stream);
  else
    launch_d<128>(p, pl.mt, bs, (hipStream_t)stream);
  return check_launch("verify_attention");
}
