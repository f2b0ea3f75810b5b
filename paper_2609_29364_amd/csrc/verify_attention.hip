// Verification attention: every request's anchor + K proposal queries attend,
// causally, to its paged KV cache (Section 1: one target forward verifies all
// proposals; Appendix G.2/H: anchor plus depth-d proposals; Section 3: paged,
// append-dominant cache that already holds the window).  Optionally fused with
// the KV-state preparation of arriving requests (Prepare, Algorithm 1;
// Appendix E.1): their K/V tiles are read from the staging pool, used, and
// stored into the worker pool in the same pass.
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
//   lane-local.  No LDS round trip is needed for either operand; Q operands
//   sit in LDS in operand order.
// * K/V are streamed once, so they are loaded non-temporally.  The registers
//   loaded for one span are exactly the tile bytes, so the fused variant
//   stores them back unchanged into the worker pool.
// * Software pipeline: within an item K(j+1) is requested as soon as S(j)
//   consumed K(j) and V(j+1) as soon as PV(j) consumed V(j); across items the
//   next item's first span is requested during the current item's last span
//   and its Q is fetched one item ahead, so a wave never drains its loads at
//   an item boundary.  Block ids are wave-uniform scalar loads; every vector
//   load inside a loop is unconditional (a conditional load makes the
//   compiler wait for all outstanding loads at the join).
// * Load balance (stream-K): the spans of all (request, KV head) items are cut
//   into as many equal contiguous ranges as the device keeps waves resident,
//   whatever the spread of context lengths.  Items cut by a range boundary
//   leave partials that a small second kernel merges in range order
//   (deterministic, no atomics in the arithmetic); all other items are
//   written directly.
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

constexpr int kBlock = 16;        // token slots per KV block
constexpr int kSpan = 32;         // tokens per main-loop step
constexpr int kMaxRows = 64;      // (Hq/Hkv) * max_q_per_seq limit
constexpr int kMaxBatch = 8192;   // the span prefix of the batch lives in LDS

struct Params {
  const uint16_t* q;
  const uint16_t* k_cache;   // worker pool (read for resident requests)
  const uint16_t* v_cache;
  uint16_t* k_dst;           // worker pool, written by the fused variant
  uint16_t* v_dst;
  const uint16_t* k_stage;   // staging pool (fused variant)
  const uint16_t* v_stage;
  const int32_t* block_table;
  const int32_t* stage_table;
  const int32_t* seq_lens;
  const int32_t* q_indptr;
  uint16_t* out;
  float* part_o;       // [2 * ranges][MT*16][D]: head/tail partial O per range
  float2* part_ml;     // [2 * ranges][MT*16]: (running max, sum)
  uint32_t* prefix;    // [bs+1]: exclusive prefix of per-request span counts
  uint32_t* counters;  // [1]: next dynamic chunk to claim (zero between dispatches)
  uint16_t* trash;     // one K tile + one V tile that absorb stores to invalid ids
  int64_t num_blocks;
  int64_t stage_blocks;
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

template <int MT, int D>
struct QOps {
  u32x4 q[MT][D / 32];  // Q operands of one item (fetched one item ahead)
};

// Values every lane of a wave agrees on, marked so for the compiler (uniform
// values live in scalar registers and their loads become scalar loads).
__device__ inline int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ inline int64_t uniform64(int64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

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

__device__ inline int clamp_len(const Params& p, const int32_t* __restrict__ seq_lens, int r) {
  const int L = seq_lens[r];
  return max(0, min(L, min(p.max_seq_len, p.max_blocks_per_seq * kBlock)));
}

// Spans of one (request, KV head) item; an empty context still owns one span
// so that its rows are written (as zeros).
__device__ inline int spans_of(int L) { return max(1, (L + kSpan - 1) / kSpan); }

// One (request r, KV head g) item restricted to spans [j0, j1) of a range.
struct Item {
  int r, g, L, n, qo, nq, rows, win, j0, j1;
  int64_t pr;        // exclusive span prefix of request r (per KV head)
  bool arriving;     // fused variant: K/V come from the staging pool
};

template <bool FUSE>
__device__ inline Item make_item(const Params& p, const int32_t* __restrict__ seq_lens,
                                 const int32_t* __restrict__ q_indptr,
                                 const int32_t* __restrict__ stage_table, int r, int64_t pr,
                                 int64_t s, int64_t s1) {
  Item it;
  it.r = r;
  it.pr = pr;
  it.L = clamp_len(p, seq_lens, r);
  it.n = spans_of(it.L);
  it.qo = q_indptr[r];
  it.nq = max(0, min(q_indptr[r + 1] - it.qo, p.max_q));
  const int64_t off = s - (int64_t)p.num_kv_heads * pr;
  it.g = (int)(off / it.n);
  it.j0 = (int)(off - (int64_t)it.g * it.n);
  it.j1 = (int)min((int64_t)it.n, it.j0 + (s1 - s));
  it.rows = p.group * it.nq;
  it.win = it.L - it.nq;
  it.arriving = FUSE && p.stage_blocks > 0 &&
                stage_table[(int64_t)r * p.max_blocks_per_seq] >= 0;
  return it;
}

struct SpanRef {
  const uint16_t* k_src;  // planes the span is read from (pool or staging)
  const uint16_t* v_src;
  int64_t hs0, hs1;       // element offsets of the two source tiles
  int64_t hd0, hd1;       // element offsets of the two destination tiles (fused)
  int32_t t;              // first token of the span
  bool bad0, bad1;        // block id out of range: tokens invisible
  bool has1;              // the span's second block exists
};

// Span j of item it.  Block ids are wave-uniform, so they are fetched with
// scalar loads, which keep the vector-memory counter free for the K/V stream.
template <int D, bool FUSE>
__device__ inline SpanRef span_ref(const Params& p, const int32_t* __restrict__ block_table,
                                   const int32_t* __restrict__ stage_table, const Item& it,
                                   int j) {
  SpanRef s;
  s.t = j * kSpan;
  const int b0 = s.t / kBlock;
  s.has1 = s.t + kBlock < it.L;
  const int64_t row = (int64_t)it.r * p.max_blocks_per_seq;
  const int64_t tile = (int64_t)D * kBlock;
  int32_t id0 = block_table[row + b0];
  int32_t id1 = s.has1 ? block_table[row + b0 + 1] : id0;
  const bool pbad0 = id0 < 0 || id0 >= p.num_blocks;
  const bool pbad1 = id1 < 0 || id1 >= p.num_blocks;
  if (FUSE && it.arriving) {
    int32_t sid0 = stage_table[row + b0];
    int32_t sid1 = s.has1 ? stage_table[row + b0 + 1] : sid0;
    s.bad0 = sid0 < 0 || sid0 >= p.stage_blocks;
    const bool sbad1 = sid1 < 0 || sid1 >= p.stage_blocks;
    s.bad1 = s.has1 && sbad1;
    if (s.bad0) sid0 = 0;
    if (!s.has1 || sbad1) sid1 = sid0;
    s.k_src = p.k_stage;
    s.v_src = p.v_stage;
    s.hs0 = ((int64_t)sid0 * p.num_kv_heads + it.g) * tile;
    s.hs1 = ((int64_t)sid1 * p.num_kv_heads + it.g) * tile;
    // destinations outside the pool are redirected to the trash tile
    s.hd0 = pbad0 ? -1 : ((int64_t)id0 * p.num_kv_heads + it.g) * tile;
    s.hd1 = (pbad1 || !s.has1) ? -1 : ((int64_t)id1 * p.num_kv_heads + it.g) * tile;
  } else {
    s.bad0 = pbad0;
    s.bad1 = s.has1 && pbad1;
    if (pbad0) id0 = 0;
    if (!s.has1 || pbad1) id1 = id0;
    s.k_src = p.k_cache;
    s.v_src = p.v_cache;
    s.hs0 = ((int64_t)id0 * p.num_kv_heads + it.g) * tile;
    s.hs1 = ((int64_t)id1 * p.num_kv_heads + it.g) * tile;
    s.hd0 = s.hd1 = -1;
  }
  return s;
}

template <int D>
__device__ inline void load_k(KOps<D>& o, const SpanRef& s, int lane) {
  const int row = lane & 15, grp = lane >> 4;
  const uint16_t* k0 = s.k_src + s.hs0;
  const uint16_t* k1 = s.k_src + s.hs1;
#pragma unroll
  for (int kk = 0; kk < D / 32; ++kk) {
    const int off = ((kk * 4 + grp) * kBlock + row) * 8;
    o.k[0][kk] = __builtin_nontemporal_load((const u32x4*)(k0 + off));
    o.k[1][kk] = __builtin_nontemporal_load((const u32x4*)(k1 + off));
  }
}

template <int D>
__device__ inline void load_v(VOps<D>& o, const SpanRef& s, int lane) {
  const int row = lane & 15, grp = lane >> 4;
  const uint16_t* v0 = s.v_src + s.hs0;
  const uint16_t* v1 = s.v_src + s.hs1;
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const int off = (dt * 16 + row) * kBlock + grp * 4;
    o.v[0][dt] = __builtin_nontemporal_load((const u32x2*)(v0 + off));
    o.v[1][dt] = __builtin_nontemporal_load((const u32x2*)(v1 + off));
  }
}

// Fused variant: the loaded tiles go back out unchanged to the worker pool
// (same offsets inside the tile as they were read from).
template <int D>
__device__ inline void store_k(const KOps<D>& o, const Params& p, const SpanRef& s, bool second,
                               int lane) {
  const int row = lane & 15, grp = lane >> 4;
  uint16_t* k0 = s.hd0 >= 0 ? p.k_dst + s.hd0 : p.trash;
  uint16_t* k1 = s.hd1 >= 0 ? p.k_dst + s.hd1 : p.trash;
#pragma unroll
  for (int kk = 0; kk < D / 32; ++kk) {
    const int off = ((kk * 4 + grp) * kBlock + row) * 8;
    __builtin_nontemporal_store(o.k[0][kk], (u32x4*)(k0 + off));
    if (second) __builtin_nontemporal_store(o.k[1][kk], (u32x4*)(k1 + off));
  }
}

template <int D>
__device__ inline void store_v(const VOps<D>& o, const Params& p, const SpanRef& s, bool second,
                               int lane) {
  const int row = lane & 15, grp = lane >> 4;
  uint16_t* v0 = s.hd0 >= 0 ? p.v_dst + s.hd0 : p.trash + D * kBlock;
  uint16_t* v1 = s.hd1 >= 0 ? p.v_dst + s.hd1 : p.trash + D * kBlock;
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const int off = (dt * 16 + row) * kBlock + grp * 4;
    __builtin_nontemporal_store(o.v[0][dt], (u32x2*)(v0 + off));
    if (second) __builtin_nontemporal_store(o.v[1][dt], (u32x2*)(v1 + off));
  }
}

// Q operands of item it for this lane's rows (garbage past the item's rows,
// zeroed when staged).  Addresses are clamped into the Q tensor so the loads
// are unconditional.
template <int D, int MT>
__device__ inline void load_q(QOps<MT, D>& o, const Params& p, const Item& it, int total_q,
                              int lane) {
  const int grp = lane >> 4;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = mt * 16 + (lane & 15);
    const int mm = min(m, max(it.rows - 1, 0));
    const int j = mm / p.group;
    const int h = it.g * p.group + mm % p.group;
    const int qrow = min(it.qo + j, total_q - 1);
    const uint16_t* src = p.q + ((int64_t)qrow * p.num_q_heads + h) * D;
#pragma unroll
    for (int kk = 0; kk < D / 32; ++kk) o.q[mt][kk] = *(const u32x4*)(src + kk * 32 + grp * 8);
  }
}

template <int D, int MT>
__device__ inline void stage_q(u32x4* qlds, const QOps<MT, D>& o, const Item& it, int lane) {
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const bool valid = mt * 16 + (lane & 15) < it.rows;
#pragma unroll
    for (int kk = 0; kk < D / 32; ++kk)
      qlds[(mt * (D / 32) + kk) * 64 + lane] = valid ? o.q[mt][kk] : u32x4{0, 0, 0, 0};
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

// Running softmax state of one item.
template <int D, int MT>
struct Acc {
  f32x4 o[MT][D / 16];
  float m[MT], l[MT];
  int pos[MT];
};

// Online-softmax update from one span's scores; returns P^T operands (bf16).
template <int D, int MT>
__device__ inline void span_softmax(const f32x4 (&st)[2][MT], const SpanRef& s, Acc<D, MT>& a,
                                    int win, float scale_log2, int lane, bf16x8 (&pop)[MT]) {
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
          x[h][i] = (t <= a.pos[mt] && !bad) ? x[h][i] : -INFINITY;
        }
      }
    }
    float mx = x[0][0];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int i = 0; i < 4; ++i) mx = fmaxf(mx, x[h][i]);
    mx = wave_max_groups(mx);
    const float m_new = fmaxf(a.m[mt], mx);
    const bool none = m_new == -INFINITY;
    const float alpha = none ? 1.f : __builtin_amdgcn_exp2f(a.m[mt] - m_new);
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
    a.l[mt] = a.l[mt] * alpha + psum;
    a.m[mt] = m_new;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) a.o[mt][dt] *= alpha;
    pop[mt] = bf16x8{(__bf16)pr[0][0], (__bf16)pr[0][1], (__bf16)pr[0][2], (__bf16)pr[0][3],
                     (__bf16)pr[1][0], (__bf16)pr[1][1], (__bf16)pr[1][2], (__bf16)pr[1][3]};
  }
}

// O^T += V^T P^T; V elements of tokens >= L (or of bad blocks) are zeroed.
template <int D, int MT>
__device__ inline void span_pv(const VOps<D>& v, const SpanRef& s, int L, const bf16x8 (&pop)[MT],
                               Acc<D, MT>& a, int lane) {
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
      a.o[mt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pop[mt], a.o[mt][dt], 0, 0, 0);
  }
}

// One span: S from K, online softmax, PV from V.  The registers each phase
// has consumed are refilled at once with span `nr`; with STORE (fused
// variant, arriving item) the loaded tiles are first written to the pool
// (SECOND: the span's second block exists).
template <int D, int MT, bool STORE, bool SECOND>
__device__ inline void span_step(KOps<D>& kr, VOps<D>& vr, const SpanRef& sr, const SpanRef& nr,
                                 const u32x4* qlds, const Params& p, Acc<D, MT>& a, int win,
                                 int L, int lane) {
  f32x4 st[2][MT];
  span_scores<D, MT>(kr, qlds, lane, st);
  if constexpr (STORE) store_k<D>(kr, p, sr, SECOND, lane);
  load_k<D>(kr, nr, lane);
  bf16x8 pop[MT];
  span_softmax<D, MT>(st, sr, a, win, p.scale_log2, lane, pop);
  span_pv<D, MT>(vr, sr, L, pop, a, lane);
  if constexpr (STORE) store_v<D>(vr, p, sr, SECOND, lane);
  load_v<D>(vr, nr, lane);
}

template <int D, int MT>
__device__ inline void init_acc(Acc<D, MT>& a, const Params& p, const Item& it, int lane) {
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    a.m[mt] = -INFINITY;
    a.l[mt] = 0.f;
    const int m = mt * 16 + (lane & 15);
    a.pos[mt] = m < it.rows ? it.win + m / p.group : it.L - 1;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) a.o[mt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
}

// Finish item it: a whole item is normalised and written to the output; an
// item cut by a range boundary leaves its partial in the range's head slot
// (the item began in an earlier range) or tail slot (it continues later).
template <int D, int MT>
__device__ inline void finish_item(const Params& p, Acc<D, MT>& a, const Item& it, int64_t rid,
                                   int lane) {
  const int grp = lane >> 4;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) a.l[mt] = wave_sum_groups(a.l[mt]);
  if (it.j0 == 0 && it.j1 == it.n) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = mt * 16 + (lane & 15);
      if (m >= it.rows) continue;
      const int j = m / p.group;
      const int h = it.g * p.group + m % p.group;
      const float inv = a.l[mt] > 0.f ? 1.f / a.l[mt] : 0.f;
      uint16_t* dst = p.out + ((int64_t)(it.qo + j) * p.num_q_heads + h) * D + grp * 4;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const bf16x2 lo = {(__bf16)(a.o[mt][dt][0] * inv), (__bf16)(a.o[mt][dt][1] * inv)};
        const bf16x2 hi = {(__bf16)(a.o[mt][dt][2] * inv), (__bf16)(a.o[mt][dt][3] * inv)};
        *(u32x2*)(dst + dt * 16) = u32x2{__builtin_bit_cast(uint32_t, lo),
                                         __builtin_bit_cast(uint32_t, hi)};
      }
    }
  } else {
    const int64_t slot = 2 * rid + (it.j0 > 0 ? 0 : 1);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = mt * 16 + (lane & 15);
      float* dst = p.part_o + (slot * (MT * 16) + m) * D + grp * 4;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) *(f32x4*)(dst + dt * 16) = a.o[mt][dt];
      if (grp == 0) p.part_ml[slot * (MT * 16) + m] = make_float2(a.m[mt], a.l[mt]);
    }
  }
}

constexpr int kStaticPct = 100;  // share of spans split evenly over the waves up front
constexpr int kChunkSpans = 8;   // spans per dynamically claimed chunk

// The global sequence of T spans (ordered by request, then KV head, then
// position) is cut into ranges: W static ranges covering the first Ts spans
// evenly, one per wave, then C dynamic chunks of kChunkSpans spans that waves
// claim from a counter once their static range is done.  Every kernel derives
// the same ranges from T and W.
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

// Spans [j0, j1) of one item.  The loads of the item's first span were issued
// by the caller; during its last span the first span of `next` is requested
// (when the range ends inside `it`, `next` is `it` and the loads are spare).
template <int D, int MT, bool FUSE, bool ARR>
__device__ inline void run_item(const Params& p, const int32_t* __restrict__ block_table,
                                const int32_t* __restrict__ stage_table, const Item& it,
                                const Item& next, KOps<D>& kreg, VOps<D>& vreg, SpanRef& cur,
                                const u32x4* qlds, Acc<D, MT>& a, int lane) {
  for (int j = it.j0; j + 1 < it.j1; ++j) {
    const SpanRef nxt = span_ref<D, FUSE>(p, block_table, stage_table, it, j + 1);
    span_step<D, MT, ARR, true>(kreg, vreg, cur, nxt, qlds, p, a, it.win, it.L, lane);
    cur = nxt;
  }
  const SpanRef nxt = span_ref<D, FUSE>(p, block_table, stage_table, next, next.j0);
  if (!ARR || cur.has1)
    span_step<D, MT, ARR, true>(kreg, vreg, cur, nxt, qlds, p, a, it.win, it.L, lane);
  else
    span_step<D, MT, ARR, false>(kreg, vreg, cur, nxt, qlds, p, a, it.win, it.L, lane);
  cur = nxt;
}

// One range [s, s1) of global spans, range id rid: online softmax over every
// (request, KV head) item the range touches.
template <int D, int MT, bool FUSE>
__device__ void process_range(const Params& p, const int32_t* __restrict__ block_table,
                              const int32_t* __restrict__ stage_table,
                              const int32_t* __restrict__ seq_lens,
                              const int32_t* __restrict__ q_indptr, const uint32_t* pre,
                              u32x4* qbuf0, u32x4* qbuf1, int total_q, int64_t rid, int64_t s,
                              int64_t s1, int lane) {
  const int hkv = p.num_kv_heads;
  const int r0 = uniform(find_request(pre, p.bs, hkv, s));
  Item it = make_item<FUSE>(p, seq_lens, q_indptr, stage_table, r0, uniform64(pre[r0]), s, s1);
  Item next = it;
  int64_t s_next = s + (it.j1 - it.j0);
  if (s_next < s1) {
    const bool nr = it.g == hkv - 1;
    next = make_item<FUSE>(p, seq_lens, q_indptr, stage_table, nr ? it.r + 1 : it.r,
                           nr ? it.pr + it.n : it.pr, s_next, s1);
  }

  // Q of the next item is fetched one item ahead into registers when the
  // tile leaves room for them (PREQ); larger tiles fetch it at the switch.
  constexpr bool PREQ = D * MT <= 256;
  QOps<MT, D> qr;
  load_q<D, MT>(qr, p, it, total_q, lane);
  SpanRef cur = span_ref<D, FUSE>(p, block_table, stage_table, it, it.j0);
  KOps<D> kreg;
  VOps<D> vreg;
  load_k<D>(kreg, cur, lane);
  load_v<D>(vreg, cur, lane);
  stage_q<D, MT>(qbuf0, qr, it, lane);
  if constexpr (PREQ) load_q<D, MT>(qr, p, next, total_q, lane);
  __builtin_amdgcn_wave_barrier();
  u32x4* qcur = qbuf0;
  u32x4* qnext = qbuf1;
  while (true) {
    Acc<D, MT> a;
    init_acc<D, MT>(a, p, it, lane);
    if (FUSE && it.arriving)
      run_item<D, MT, FUSE, true>(p, block_table, stage_table, it, next, kreg, vreg, cur, qcur,
                                  a, lane);
    else
      run_item<D, MT, FUSE, false>(p, block_table, stage_table, it, next, kreg, vreg, cur, qcur,
                                   a, lane);
    finish_item<D, MT>(p, a, it, rid, lane);
    if (s_next >= s1) break;
    // switch to the next item
    if constexpr (!PREQ) load_q<D, MT>(qr, p, next, total_q, lane);
    stage_q<D, MT>(qnext, qr, next, lane);
    __builtin_amdgcn_wave_barrier();
    u32x4* t = qcur;
    qcur = qnext;
    qnext = t;
    it = next;
    s_next += it.j1 - it.j0;
    if (s_next < s1) {
      const bool nr = it.g == hkv - 1;
      next = make_item<FUSE>(p, seq_lens, q_indptr, stage_table, nr ? it.r + 1 : it.r,
                             nr ? it.pr + it.n : it.pr, s_next, s1);
    }
    if constexpr (PREQ) load_q<D, MT>(qr, p, next, total_q, lane);
  }
}

// One dispatch of W waves (W / 4 workgroups of 4 independent waves).
template <int D, int MT, bool FUSE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(D * MT <= 128 ? 2 : 1)))
void verify_attention_kernel(Params p, const int32_t* __restrict__ block_table,
                             const int32_t* __restrict__ stage_table,
                             const int32_t* __restrict__ seq_lens,
                             const int32_t* __restrict__ q_indptr) {
  extern __shared__ uint32_t s_pre[];        // [bs + 1]: exclusive prefix of per-request spans
  __shared__ uint32_t s_wsum[4];
  constexpr int kQBufs = D * MT <= 256 ? 2 : 1;   // one-item-ahead Q needs two buffers
  __shared__ u32x4 s_q[4][kQBufs][MT * (D / 32) * 64];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = uniform(tid >> 6);
  const int total_q = uniform(q_indptr[p.bs]);

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
  if (total_q <= 0) return;   // no query rows: nothing to attend

  const Ranges R((int64_t)p.num_kv_heads * carry, p.num_waves);
  const int64_t w = (int64_t)blockIdx.x * 4 + wave;
  int64_t rid = w;
  while (true) {
    const int64_t b = uniform64(R.begin(rid)), e = uniform64(R.end(rid));
    if (b < e)
      process_range<D, MT, FUSE>(p, block_table, stage_table, seq_lens, q_indptr, s_pre,
                                 s_q[wave][0], s_q[wave][kQBufs - 1], total_q, rid, b, e, lane);
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

template <int D, int MT, bool FUSE>
const void* kernel_ptr() {
  return (const void*)&verify_attention_kernel<D, MT, FUSE>;
}

template <bool FUSE>
const void* kernel_for(int d, int mt) {
  if (d == 64) {
    switch (mt) {
      case 1: return kernel_ptr<64, 1, FUSE>();
      case 2: return kernel_ptr<64, 2, FUSE>();
      case 3: return kernel_ptr<64, 3, FUSE>();
      default: return kernel_ptr<64, 4, FUSE>();
    }
  }
  switch (mt) {
    case 1: return kernel_ptr<128, 1, FUSE>();
    case 2: return kernel_ptr<128, 2, FUSE>();
    case 3: return kernel_ptr<128, 3, FUSE>();
    default: return kernel_ptr<128, 4, FUSE>();
  }
}

struct Plan {
  int mt;            // 16-row tiles
  int num_waves;     // W: resident waves of the launch
  int64_t max_chunks;
  size_t lds_bytes;  // dynamic LDS: the span prefix
  size_t counter_bytes, prefix_bytes, trash_bytes, part_o_bytes, part_ml_bytes, ws_bytes;
};

// Waves the device keeps resident for this kernel (CUs x waves per CU), or
// NSD_ATTN_WAVES when set (a multiple of 4, for tests and tuning).
int resident_waves(int d, int mt, bool fuse) {
  const char* env = getenv("NSD_ATTN_WAVES");
  if (env) {
    const int v = atoi(env);
    if (v >= 4 && v % 4 == 0) return v;
  }
  int dev = 0, cus = 0, blocks = 0;
  const void* k = fuse ? kernel_for<true>(d, mt) : kernel_for<false>(d, mt);
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k, 256, 0) != hipSuccess ||
      cus <= 0 || blocks <= 0) {
    (void)hipGetLastError();
    cus = 256;
    blocks = 2;
  }
  return cus * blocks * 4;
}

bool make_plan(int bs, int hq, int hkv, int d, int max_q, int max_seq_len, bool fuse,
               Plan* pl) {
  if (bs < 0 || bs > kMaxBatch || hq < 1 || hkv < 1 || hq % hkv || (d != 64 && d != 128) ||
      max_q < 1 || max_seq_len < 0)
    return false;
  const int rows = (hq / hkv) * max_q;
  if (rows > kMaxRows) return false;
  pl->mt = (rows + 15) / 16;
  pl->num_waves = resident_waves(d, pl->mt, fuse);
  // upper bound of the dynamic chunks: at most 1 + (100-kStaticPct)% of the spans
  const int64_t max_spans = (int64_t)hkv * bs * std::max(1, (max_seq_len + kSpan - 1) / kSpan);
  pl->max_chunks = (max_spans - max_spans * kStaticPct / 100 + kChunkSpans - 1) / kChunkSpans + 1;
  const size_t slots = 2 * ((size_t)pl->num_waves + (size_t)pl->max_chunks) * pl->mt * 16;
  pl->lds_bytes = ((size_t)bs + 1) * sizeof(uint32_t);
  pl->counter_bytes = 256;
  pl->prefix_bytes = (((size_t)bs + 1) * sizeof(uint32_t) + 255) / 256 * 256;
  pl->trash_bytes = (size_t)2 * d * kBlock * 2;
  pl->part_o_bytes = slots * d * sizeof(float);
  pl->part_ml_bytes = slots * sizeof(float2);
  pl->ws_bytes = pl->counter_bytes + pl->prefix_bytes + pl->trash_bytes + pl->part_o_bytes +
                 pl->part_ml_bytes;
  return true;
}

template <int D, int MT, bool FUSE>
void launch(const Params& p, int bs, hipStream_t stream) {
  hipLaunchKernelGGL((verify_attention_kernel<D, MT, FUSE>), dim3(p.num_waves / 4), dim3(256),
                     ((size_t)bs + 1) * sizeof(uint32_t), stream, p, p.block_table,
                     p.stage_table, p.seq_lens, p.q_indptr);
  hipLaunchKernelGGL((combine_kernel<D, MT>), dim3(p.num_kv_heads, bs), dim3(256), 0, stream, p);
}

template <int D, bool FUSE>
void launch_d(const Params& p, int mt, int bs, hipStream_t stream) {
  switch (mt) {
    case 1: launch<D, 1, FUSE>(p, bs, stream); break;
    case 2: launch<D, 2, FUSE>(p, bs, stream); break;
    case 3: launch<D, 3, FUSE>(p, bs, stream); break;
    default: launch<D, 4, FUSE>(p, bs, stream); break;
  }
}

// Shared by both entry points: validation, workspace carving, launch.
nsd_status run(const char* fn, bool fuse, const void* q, const void* k_cache,
               const void* v_cache, void* k_dst, void* v_dst, int64_t num_blocks,
               const void* k_stage, const void* v_stage, int64_t stage_blocks,
               const int32_t* block_table, const int32_t* stage_table,
               int32_t max_blocks_per_seq, const int32_t* seq_lens, const int32_t* q_indptr,
               int32_t bs, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
               int32_t block_size, int32_t max_q_per_seq, int32_t max_seq_len, float scale,
               void* out, void* workspace, size_t workspace_bytes, void* stream) {
  using namespace nsd;
  if (bs < 0 || bs > kMaxBatch)
    return fail(NSD_ERR_SHAPE, "%s: bs must be in [0, %d]", fn, kMaxBatch);
  if (block_size != NSD_BLOCK_SIZE)
    return fail(NSD_ERR_UNSUPPORTED, "%s: block_size must be 16 (got %d)", fn, block_size);
  if (head_dim != 64 && head_dim != 128)
    return fail(NSD_ERR_UNSUPPORTED, "%s: head_dim must be 64 or 128 (got %d)", fn, head_dim);
  if (num_q_heads < 1 || num_kv_heads < 1 || num_q_heads % num_kv_heads)
    return fail(NSD_ERR_SHAPE, "%s: num_q_heads (%d) must be a positive multiple of "
                "num_kv_heads (%d)", fn, num_q_heads, num_kv_heads);
  if (max_q_per_seq < 1) return fail(NSD_ERR_SHAPE, "%s: max_q_per_seq < 1", fn);
  if ((num_q_heads / num_kv_heads) * max_q_per_seq > kMaxRows)
    return fail(NSD_ERR_UNSUPPORTED, "%s: (Hq/Hkv)*max_q_per_seq = %d exceeds %d", fn,
                (num_q_heads / num_kv_heads) * max_q_per_seq, kMaxRows);
  if (max_seq_len < 1 || max_blocks_per_seq < 1 || num_blocks < 1)
    return fail(NSD_ERR_SHAPE, "%s: max_seq_len, max_blocks_per_seq and num_blocks must be "
                ">= 1", fn);
  if (fuse && stage_blocks < 0) return fail(NSD_ERR_SHAPE, "%s: stage_num_blocks < 0", fn);
  if (!(scale == scale) || isinf(scale)) return fail(NSD_ERR_SHAPE, "%s: scale must be finite", fn);
  if (bs == 0) return NSD_OK;
  if (!q || !k_cache || !v_cache || !block_table || !seq_lens || !q_indptr || !out ||
      (fuse && (!k_dst || !v_dst || !stage_table || (stage_blocks > 0 && (!k_stage || !v_stage)))))
    return fail(NSD_ERR_NULL, "%s: NULL pointer argument", fn);
  Plan pl;
  make_plan(bs, num_q_heads, num_kv_heads, head_dim, max_q_per_seq, max_seq_len, fuse, &pl);
  if (!workspace || workspace_bytes < pl.ws_bytes)
    return fail(NSD_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn,
                pl.ws_bytes, workspace ? workspace_bytes : (size_t)0);
  int dev = 0, lds_max = 0;
  hipFuncAttributes fa;
  const void* kfn = fuse ? kernel_for<true>(head_dim, pl.mt) : kernel_for<false>(head_dim, pl.mt);
  if (hipGetDevice(&dev) == hipSuccess &&
      hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) ==
          hipSuccess &&
      hipFuncGetAttributes(&fa, kfn) == hipSuccess &&
      fa.sharedSizeBytes + pl.lds_bytes > (size_t)lds_max)
    return fail(NSD_ERR_UNSUPPORTED, "%s: bs=%d needs %zu bytes of LDS, %d available", fn, bs,
                fa.sharedSizeBytes + pl.lds_bytes, lds_max);
  (void)hipGetLastError();

  Params p;
  p.q = (const uint16_t*)q;
  p.k_cache = (const uint16_t*)k_cache;
  p.v_cache = (const uint16_t*)v_cache;
  p.k_dst = (uint16_t*)k_dst;
  p.v_dst = (uint16_t*)v_dst;
  p.k_stage = (const uint16_t*)k_stage;
  p.v_stage = (const uint16_t*)v_stage;
  p.block_table = block_table;
  p.stage_table = stage_table;
  p.seq_lens = seq_lens;
  p.q_indptr = q_indptr;
  p.out = (uint16_t*)out;
  char* ws = (char*)workspace;
  p.counters = (uint32_t*)ws;
  p.prefix = (uint32_t*)(ws + pl.counter_bytes);
  p.trash = (uint16_t*)(ws + pl.counter_bytes + pl.prefix_bytes);
  p.part_o = (float*)(ws + pl.counter_bytes + pl.prefix_bytes + pl.trash_bytes);
  p.part_ml = (float2*)(ws + pl.counter_bytes + pl.prefix_bytes + pl.trash_bytes +
                        pl.part_o_bytes);
  p.num_blocks = num_blocks;
  p.stage_blocks = fuse ? stage_blocks : 0;
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
  if (fuse) {
    if (head_dim == 64) launch_d<64, true>(p, pl.mt, bs, (hipStream_t)stream);
    else launch_d<128, true>(p, pl.mt, bs, (hipStream_t)stream);
  } else {
    if (head_dim == 64) launch_d<64, false>(p, pl.mt, bs, (hipStream_t)stream);
    else launch_d<128, false>(p, pl.mt, bs, (hipStream_t)stream);
  }
  return check_launch(fn);
}

}  // namespace

extern "C" size_t nsd_verify_attention_workspace_size(int32_t bs, int32_t num_q_heads,
                                                      int32_t num_kv_heads, int32_t head_dim,
                                                      int32_t max_q_per_seq,
                                                      int32_t max_seq_len) {
  Plan pl, pf;
  if (!make_plan(bs, num_q_heads, num_kv_heads, head_dim, max_q_per_seq, max_seq_len, false,
                 &pl) ||
      !make_plan(bs, num_q_heads, num_kv_heads, head_dim, max_q_per_seq, max_seq_len, true, &pf))
    return 0;
  return std::max(pl.ws_bytes, pf.ws_bytes);
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
  return run("verify_attention", false, q, k_cache, v_cache, nullptr, nullptr, num_blocks,
             nullptr, nullptr, 0, block_table, nullptr, max_blocks_per_seq, seq_lens, q_indptr,
             bs, num_q_heads, num_kv_heads, head_dim, block_size, max_q_per_seq, max_seq_len,
             scale, out, workspace, workspace_bytes, stream);
}

extern "C" nsd_status nsd_gather_verify_attention(
    const void* q, void* k_cache, void* v_cache, int64_t num_blocks, const void* k_stage,
    const void* v_stage, int64_t stage_num_blocks, const int32_t* block_table,
    const int32_t* stage_table, int32_t max_blocks_per_seq, const int32_t* seq_lens,
    const int32_t* q_indptr, int32_t bs, int32_t num_q_heads, int32_t num_kv_heads,
    int32_t head_dim, int32_t block_size, int32_t max_q_per_seq, int32_t max_seq_len,
    float scale, void* out, void* workspace, size_t workspace_bytes, void* stream) {
  return run("gather_verify_attention", true, q, k_cache, v_cache, k_cache, v_cache, num_blocks,
             k_stage, v_stage, stage_num_blocks, block_table, stage_table, max_blocks_per_seq,
             seq_lens, q_indptr, bs, num_q_heads, num_kv_heads, head_dim, block_size,
             max_q_per_seq, max_seq_len, scale, out, workspace, workspace_bytes, stream);
}
