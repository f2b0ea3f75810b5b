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
//   lane-local.  No LDS round trip is needed for either operand; an item's Q
//   operands stay in registers.
// * K/V are streamed once, so they are loaded non-temporally.  The registers
//   loaded for one span are exactly the tile bytes, so the fused variant
//   stores them back unchanged into the worker pool.
// * A main-loop step covers NB blocks (NB * 16 tokens).  A wave's throughput
//   is bounded by the K/V bytes it keeps in flight over the HBM latency, so
//   tiles whose registers allow it take four blocks (32 KiB of K and V per
//   step for head_dim 128) and run one wave per SIMD.
// * Software pipeline: within an item K(j+1) is requested as soon as S(j)
//   consumed K(j) and V(j+1) as soon as PV(j) consumed V(j); across items the
//   next item's first span is requested during the current item's last span
//   (without fusion, together with its Q), so a wave never drains its K/V
//   loads at an item boundary.  Block ids are wave-uniform scalar loads;
//   every vector load inside a loop is unconditional (a conditional load
//   makes the compiler wait for all outstanding loads at the join).
// * Load balance (stream-K): the spans of all (request, KV head) items are cut
//   into as many equal contiguous ranges as the device keeps waves resident,
//   whatever the spread of context lengths.  The fused variant cuts the
//   resident and the arriving requests' spans separately and every wave takes
//   one range of each, resident first, so that all waves write the staged
//   tiles in the same phase of the launch (writes gathered in time cost HBM
//   less than writes spread through the read stream).  The resident segment
//   only reads, so it streams the separate attention's deeper spans; the
//   arriving segment's spans are sized for the tile that also stores.  The split is static:
//   the workspace needs no initialisation and no wave waits on another.
//   Items cut by a range boundary leave partials that a small second kernel
//   merges in range order (deterministic, no atomics in the arithmetic); all
//   other items are written directly.
// * No stores while the K/V stream runs: stores retire through the same
//   in-order vector-memory counter as the loads, and a store's
//   acknowledgement comes late under a full read stream, so every later load
//   wait would also wait for it.  A finished item's output rows (or its
//   partial) go to the wave's LDS buffer, which is written out, in whole
//   rows, when it is full and when the wave's work ends.  (The fused
//   variant's own tile stores are the preparation itself and stay in line.)
// * Masked tokens (past a query's position, past L_r, or in a block whose id
//   is out of range) are removed by selection: scores become -inf and V
//   elements past L_r are zeroed, so NaN-filled unused slots never leak.
#include "nsd_internal.h"

#include <math.h>

#include <algorithm>
#include <atomic>
#include <mutex>

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

constexpr int kBlock = 16;        // token slots per KV block
constexpr int kMaxRows = 64;      // (Hq/Hkv) * max_q_per_seq limit
constexpr int kMaxBatch = 8192;   // the span prefix of the batch lives in LDS
constexpr int kSpare = -1;        // span index of loads that are never used

// Blocks per main-loop step for a (head_dim, row tiles) tile, reading only
// (store = false: the separate attention and the fused pass's resident
// segment) or also writing the tiles back (the fused pass's arriving
// segment): four where the registers of two extra K/V tiles fit beside the
// accumulators.  The writing tile also holds its store path: with four blocks
// and more than one 16-row tile at head_dim 128 it ran out of registers and
// reloaded a spilled lane offset before every span's loads (waiting for all
// of them), so it takes two.  The two segments of the fused pass are split
// into ranges separately, so each takes its own span size.
__host__ __device__ constexpr int span_blocks(int d, int mt, bool store) {
  return (store && d * mt > 128) ? 2 : (d * mt <= 256 ? 4 : 2);
}

// Waves per SIMD an instantiation is compiled for, and the most its launch
// keeps resident: one.  The larger tiles take the whole register file; the
// single-tile attention without fusion (the decode shape) fits twice, but two
// waves per SIMD measured no faster (decode attention on the draft_decode
// shape 489 against 461-470 us: the second wave's K/V stream adds bytes in
// flight past what HBM rewards).
__host__ __device__ constexpr int waves_per_simd(int, int, bool) { return 1; }

// The item a range cuts at its end and that began in that range (the one the
// merge kernel's workgroup for the range finishes), with what the merge needs
// to find its parts: written by the range's wave when its work ends.
struct CutRec {
  int64_t base;     // span position of the item's first span
  int32_t n;        // the item's spans; -1: the range leaves nothing to merge
  int32_t r, g, qo, nq, pad;
};

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
  uint16_t* part_o;    // [4 * waves][MT*16][D]: head/tail partial per range, O / sum in bf16
  float2* part_ml;     // [4 * waves][MT*16]: (running max, sum)
  struct CutRec* cut_rec;  // [2 * waves]: the item each range cuts at its end, for the merge
  uint32_t* prefix;    // [bs+1]: exclusive span prefix over the work order's positions
  uint32_t* pos_of;    // [bs+1]: position of each request; [bs]: resident requests;
                       // then [2]: spans of the two segments (per KV head)
  int32_t num_blocks;    // blocks in the worker pool (tiles fit 32-bit indexes)
  int32_t stage_blocks;  // blocks in the staging pool (0 without fusion)
  int32_t bs;
  int32_t max_blocks_per_seq;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t group;
  int32_t max_q;
  int32_t max_seq_len;
  int32_t num_waves;
  int32_t out_off;         // dynamic LDS: byte offset of the output buffers
  int32_t out_cap;         // bytes of each wave's output buffer
  int32_t w_even;          // relative range length of waves on even XCDs
  int32_t w_odd, w_odd_b;  // ... on odd XCDs, resident / arriving segment
  float scale_log2;  // softmax scale * log2(e)
};

template <int D, int NB>
struct KOps {
  u32x4 k[NB][D / 32];  // K operands of a span's NB blocks
};

template <int D, int NB>
struct VOps {
  u32x2 v[NB][D / 16];  // V^T operand halves of a span's NB blocks
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

// Reductions over the four 16-lane rows of a wave (lanes l, l^16, l^32 and
// l^48 hold the same query row): two cross-row register swaps, no LDS.
// Swapping a register with a copy of itself leaves, in every lane, its own
// value and its row partner's in the two registers.  The instruction is
// written out because the compiler's builtin for it merges the two results;
// the nops cover the VALU-write to cross-lane-read hazard on both sides.  The
// sum pairs (l, l^32) first, so every lane of a row adds the same two halves.
struct Pair {
  float a, b;
};

__device__ inline Pair swap32(float x) {
  Pair r = {x, x};
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(r.a), "+v"(r.b));
  return r;
}

__device__ inline Pair swap16(float x) {
  Pair r = {x, x};
  asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1\n\ts_nop 1" : "+v"(r.a), "+v"(r.b));
  return r;
}

__device__ inline float wave_max_groups(float x) {
  const Pair a = swap32(x);
  const Pair b = swap16(fmaxf(a.a, a.b));
  return fmaxf(b.a, b.b);
}

__device__ inline float wave_sum_groups(float x) {
  const Pair a = swap32(x);
  const Pair b = swap16(a.a + a.b);
  return b.a + b.b;
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
template <int NB>
__device__ inline int spans_of(int L) {
  return max(1, (L + NB * kBlock - 1) / (NB * kBlock));
}

__device__ inline bool is_arriving(const Params& p, const int32_t* __restrict__ stage_table,
                                   int r) {
  return p.stage_blocks > 0 && stage_table[(int64_t)r * p.max_blocks_per_seq] >= 0;
}

// Spans of an item (n spans from span position base) that lie in [b, e).
__device__ inline void spans_in(int64_t base, int n, int64_t b, int64_t e, int& j0, int& j1) {
  j0 = (int)max((int64_t)0, min((int64_t)n, b - base));
  j1 = (int)max((int64_t)0, min((int64_t)n, e - base));
}

// Request at position i of the work order: the fused variant orders the
// batch resident requests first, then arriving ones; otherwise position i is
// request i.
template <bool FUSE>
__device__ inline int request_at(const uint16_t* order, int i) {
  return FUSE ? (int)order[i] : i;
}

// Query rows of request r: [qo, qo + nq) from q_indptr, clamped into the
// rows [0, total_q) that total_q = q_indptr[bs] gives q and out, and nq to at
// most max_q.  A well-formed q_indptr (non-decreasing, q_indptr[0] = 0) is
// unchanged by the clamps; any other contents still address rows of q and
// out only.
__device__ inline void q_rows(const int32_t* __restrict__ q_indptr, int r, int total_q,
                              int max_q, int& qo, int& nq) {
  qo = min(max(q_indptr[r], 0), total_q);
  nq = max(0, min(min(q_indptr[r + 1] - qo, max_q), total_q - qo));
}

// One (request r, KV head g) item restricted to the spans [j0, j1) whose
// start lies in a range.
struct Item {
  int pos, r, g, L, n, qo, nq, rows, win, j0, j1;
  int64_t pr;        // exclusive span prefix of position pos (per KV head)
  int64_t base;      // span position of the item's first span
  bool arriving;     // fused variant: K/V come from the staging pool
};

template <int NB, bool ARR>
__device__ inline Item make_item(const Params& p, const int32_t* __restrict__ seq_lens,
                                 const int32_t* __restrict__ q_indptr,
                                 const int32_t* __restrict__ stage_table, int pos, int r,
                                 int g, int64_t pr, int64_t s, int64_t s1, int total_q) {
  Item it;
  it.pos = pos;
  it.r = r;
  it.g = g;
  it.pr = pr;
  it.L = clamp_len(p, seq_lens, r);
  it.n = spans_of<NB>(it.L);
  it.arriving = ARR;
  it.base = (int64_t)p.num_kv_heads * pr + (int64_t)g * it.n;
  spans_in(it.base, it.n, s, s1, it.j0, it.j1);
  q_rows(q_indptr, r, total_q, p.max_q, it.qo, it.nq);
  it.rows = p.group * it.nq;
  it.win = it.L - it.nq;
  return it;
}

// The item after `it` in (position, KV head) order; `it` is not the last
// item of the order.  ORD: positions map to requests through the work order.
template <int NB, bool ORD, bool ARR>
__device__ inline Item next_item(const Params& p, const int32_t* __restrict__ seq_lens,
                                 const int32_t* __restrict__ q_indptr,
                                 const int32_t* __restrict__ stage_table, const uint16_t* order,
                                 const Item& it, int64_t s, int64_t s1, int total_q) {
  const bool nr = it.g == p.num_kv_heads - 1;
  const int pos = nr ? it.pos + 1 : it.pos;
  return make_item<NB, ARR>(p, seq_lens, q_indptr, stage_table, pos,
                            nr ? uniform(request_at<ORD>(order, pos)) : it.r, nr ? 0 : it.g + 1,
                            nr ? it.pr + it.n : it.pr, s, s1, total_q);
}

// Raw block-table entries of one span (scalar loads, checked later).
template <int NB>
struct SpanIds {
  int32_t src[NB];   // ids the tiles are read from (worker pool, or staging if arriving)
  int32_t dst[NB];   // worker-pool ids the fused variant writes
};

template <int NB>
struct SpanRef {
  const uint16_t* k_src;  // planes the span is read from (pool or staging)
  const uint16_t* v_src;
  int32_t ts[NB];         // source tiles (block * num_kv_heads + head)
  int32_t td[NB];         // destination tiles (fused); -1: not written
  int32_t t;              // first token of the span
  uint32_t bad;           // bit b: block b's id is out of range (its tokens are invisible)
};

// Table entries of span j of item it.  Block ids are wave-uniform, so they
// are fetched with scalar loads, which keep the vector-memory counter free
// for the K/V stream; the indexes are clamped into the row, so the loads are
// unconditional.
template <int NB, bool ARR>
__device__ inline SpanIds<NB> load_ids(const Params& p, const int32_t* __restrict__ block_table,
                                       const int32_t* __restrict__ stage_table, const Item& it,
                                       int j) {
  SpanIds<NB> ids;
  const int64_t row = (int64_t)it.r * p.max_blocks_per_seq;
  const int last = p.max_blocks_per_seq - 1;
  const int32_t* __restrict__ src = ARR ? stage_table : block_table;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int e = min(j * NB + b, last);
    ids.src[b] = src[row + e];
    ids.dst[b] = ARR ? block_table[row + e] : -1;
  }
  return ids;
}

// Span j of item it from its table entries.  Blocks past the context reuse
// block 0's tile (their tokens are masked) and are not written by the fused
// variant, nor are arriving blocks with an invalid staging or destination id.
template <int NB, bool ARR>
__device__ inline SpanRef<NB> make_ref(const Params& p, const Item& it, int j,
                                       const SpanIds<NB>& ids) {
  SpanRef<NB> s;
  // kSpare: loads that are never used read block 0's tile, nothing is stored
  const bool spare = j == kSpare;
  s.t = spare ? 0 : j * NB * kBlock;
  s.bad = 0;
  const int nb = max(1, min(NB, (it.L - s.t + kBlock - 1) / kBlock));
  const bool arr = ARR;
  s.k_src = arr ? p.k_stage : p.k_cache;
  s.v_src = arr ? p.v_stage : p.v_cache;
  const int32_t src_blocks = arr ? p.stage_blocks : p.num_blocks;
  int32_t ts0 = 0;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int32_t sid = spare ? 0 : ids.src[b];
    const bool here = b < nb;
    const bool sbad = sid < 0 || sid >= src_blocks;
    if (here && sbad) s.bad |= 1u << b;
    const int32_t ts = (sbad ? 0 : sid) * p.num_kv_heads + it.g;
    if (b == 0) ts0 = ts;
    s.ts[b] = (here && !sbad) ? ts : ts0;
    const int32_t did = ids.dst[b];
    const bool dbad = did < 0 || did >= p.num_blocks;
    s.td[b] = (arr && here && !sbad && !dbad && !spare) ? did * p.num_kv_heads + it.g : -1;
  }
  return s;
}

template <int D, int NB>
__device__ inline void load_k(KOps<D, NB>& o, const SpanRef<NB>& s, int lane) {
  const int row = lane & 15, grp = lane >> 4;
#pragma unroll
  for (int kk = 0; kk < D / 32; ++kk) {
    const int off = ((kk * 4 + grp) * kBlock + row) * 8;
#pragma unroll
    for (int b = 0; b < NB; ++b)
      o.k[b][kk] = __builtin_nontemporal_load(
          (const u32x4*)(s.k_src + (int64_t)s.ts[b] * (D * kBlock) + off));
  }
}

template <int D, int NB>
__device__ inline void load_v(VOps<D, NB>& o, const SpanRef<NB>& s, int lane) {
  const int row = lane & 15, grp = lane >> 4;
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const int off = (dt * 16 + row) * kBlock + grp * 4;
#pragma unroll
    for (int b = 0; b < NB; ++b)
      o.v[b][dt] = __builtin_nontemporal_load(
          (const u32x2*)(s.v_src + (int64_t)s.ts[b] * (D * kBlock) + off));
  }
}

// Fused variant: the loaded tiles go back out unchanged to the worker pool
// (same offsets inside the tile as they were read from).
template <int D, int NB>
__device__ inline void store_k(const KOps<D, NB>& o, const Params& p, const SpanRef<NB>& s,
                               int lane) {
  const int row = lane & 15, grp = lane >> 4;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    if (s.td[b] < 0) continue;   // block past the context, or an invalid id
    uint16_t* dst = p.k_dst + (int64_t)s.td[b] * (D * kBlock);
#pragma unroll
    for (int kk = 0; kk < D / 32; ++kk) {
      const int off = ((kk * 4 + grp) * kBlock + row) * 8;
      __builtin_nontemporal_store(o.k[b][kk], (u32x4*)(dst + off));
    }
  }
}

template <int D, int NB>
__device__ inline void store_v(const VOps<D, NB>& o, const Params& p, const SpanRef<NB>& s,
                               int lane) {
  const int row = lane & 15, grp = lane >> 4;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    if (s.td[b] < 0) continue;
    uint16_t* dst = p.v_dst + (int64_t)s.td[b] * (D * kBlock);
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
      const int off = (dt * 16 + row) * kBlock + grp * 4;
      __builtin_nontemporal_store(o.v[b][dt], (u32x2*)(dst + off));
    }
  }
}

// Q operands of item it for this lane's rows.  Rows past the item's rows load
// its last row again (addresses clamped into the Q tensor, so the loads are
// unconditional): the tile products never mix rows (a row's scores, softmax
// and output column depend on that row's Q alone), and such rows are never
// stored, so they need no masking.
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

// S^T[token][row] of the span's NB blocks; the item's Q operands stay in
// registers.
template <int D, int MT, int NB>
__device__ inline void span_scores(const KOps<D, NB>& k, const QOps<MT, D>& q,
                                   f32x4 (&st)[NB][MT]) {
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    f32x4 c[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) c[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < D / 32; ++kk) {
      const bf16x8 qo = __builtin_bit_cast(bf16x8, q.q[mt][kk]);
#pragma unroll
      for (int b = 0; b < NB; ++b)
        c[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, k.k[b][kk]),
                                                       qo, c[b], 0, 0, 0);
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) st[b][mt] = c[b];
  }
}

// Running softmax state of one item.
template <int D, int MT>
struct Acc {
  f32x4 o[MT][D / 16];
  float m[MT], l[MT];
  int pos[MT];
};

// Online-softmax update from one span's scores; returns the P^T operands
// (bf16), one per pair of blocks: a 32-token k-step whose lane holds 4 tokens
// of each block of the pair, as the S^T accumulators left them.
template <int D, int MT, int NB>
__device__ inline void span_softmax(const f32x4 (&st)[NB][MT], const SpanRef<NB>& s,
                                    Acc<D, MT>& a, int win, float scale_log2, int lane,
                                    bf16x8 (&pop)[NB / 2][MT]) {
  const int grp = lane >> 4;
  const bool need_mask = (s.t + NB * kBlock > win) || s.bad;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    float x[NB][4];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) x[b][i] = st[b][mt][i] * scale_log2;
    if (need_mask) {
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const bool bad = (s.bad >> b) & 1u;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = s.t + b * kBlock + grp * 4 + i;
          x[b][i] = (t <= a.pos[mt] && !bad) ? x[b][i] : -INFINITY;
        }
      }
    }
    float mx = x[0][0];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) mx = fmaxf(mx, x[b][i]);
    mx = wave_max_groups(mx);
    const float m_new = fmaxf(a.m[mt], mx);
    const bool none = m_new == -INFINITY;
    const float alpha = none ? 1.f : __builtin_amdgcn_exp2f(a.m[mt] - m_new);
    const float msub = none ? 0.f : m_new;
    float pr[NB][4];
    float psum = 0.f;
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pr[b][i] = __builtin_amdgcn_exp2f(x[b][i] - msub);
        psum += pr[b][i];
      }
    a.l[mt] = a.l[mt] * alpha + psum;
    a.m[mt] = m_new;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) a.o[mt][dt] *= alpha;
#pragma unroll
    for (int kp = 0; kp < NB / 2; ++kp) {
      const float(&u)[4] = pr[2 * kp];
      const float(&w)[4] = pr[2 * kp + 1];
      pop[kp][mt] = bf16x8{(__bf16)u[0], (__bf16)u[1], (__bf16)u[2], (__bf16)u[3],
                           (__bf16)w[0], (__bf16)w[1], (__bf16)w[2], (__bf16)w[3]};
    }
  }
}

// O^T += V^T P^T; V elements of tokens >= L (or of bad blocks) are zeroed.
template <int D, int MT, int NB>
__device__ inline void span_pv(const VOps<D, NB>& v, const SpanRef<NB>& s, int L,
                               const bf16x8 (&pop)[NB / 2][MT], Acc<D, MT>& a, int lane) {
  const int grp = lane >> 4;
  uint32_t keep[NB][2];
#pragma unroll
  for (int b = 0; b < NB; ++b) keep[b][0] = keep[b][1] = 0xffffffffu;
  if (s.t + NB * kBlock > L || s.bad) {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const bool bad = (s.bad >> b) & 1u;
      const int nv = bad ? 0 : min(4, max(0, L - (s.t + b * kBlock + grp * 4)));
      keep[b][0] = keep_mask(nv);
      keep[b][1] = keep_mask(nv - 2);
    }
  }
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
#pragma unroll
    for (int kp = 0; kp < NB / 2; ++kp) {
      const u32x2 v0 = v.v[2 * kp][dt], v1 = v.v[2 * kp + 1][dt];
      const u32x4 w = {v0.x & keep[2 * kp][0], v0.y & keep[2 * kp][1],
                       v1.x & keep[2 * kp + 1][0], v1.y & keep[2 * kp + 1][1]};
      const bf16x8 vop = __builtin_bit_cast(bf16x8, w);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        a.o[mt][dt] =
            __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pop[kp][mt], a.o[mt][dt], 0, 0, 0);
    }
  }
}

// One span: S from K, online softmax, PV from V.  The registers each phase
// has consumed are refilled at once with span nj of item nit (whose table
// entries were requested before this step, so their latency hides behind the
// score products); with STORE (fused variant, arriving item) the loaded tiles
// are first written to the pool.  With NEXTQ (the item's last span; nit is
// the next item) the Q registers, free once the scores are formed, are
// refilled with nit's Q before its first K/V loads are issued: the loads
// complete in order, so waiting for that K also covers Q, and the switch to
// the next item waits for nothing.
template <int D, int MT, int NB, bool ARR, bool STORE, bool NEXTQ>
__device__ inline void span_step(KOps<D, NB>& kr, VOps<D, NB>& vr, SpanRef<NB>& cur,
                                 const Item& nit, int nj, const SpanIds<NB>& nids,
                                 QOps<MT, D>& q, const Params& p, Acc<D, MT>& a, int win, int L,
                                 int total_q, int lane) {
  f32x4 st[NB][MT];
  span_scores<D, MT, NB>(kr, q, st);
  if constexpr (STORE) store_k<D, NB>(kr, p, cur, lane);
  // keep the next span's address arithmetic (and the wait for its table
  // entries) behind the score products
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (NEXTQ) load_q<D, MT>(q, p, nit, total_q, lane);
  const SpanRef<NB> nr = make_ref<NB, ARR>(p, nit, nj, nids);
  load_k<D, NB>(kr, nr, lane);
  bf16x8 pop[NB / 2][MT];
  span_softmax<D, MT, NB>(st, cur, a, win, p.scale_log2, lane, pop);
  span_pv<D, MT, NB>(vr, cur, L, pop, a, lane);
  if constexpr (STORE) store_v<D, NB>(vr, p, cur, lane);
  load_v<D, NB>(vr, nr, lane);
  cur = nr;
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

// Results leave the wave through LDS.  Stores share the in-order
// vector-memory counter with the K/V loads, so a store issued while loads
// stream makes every later load wait also wait for the store, whose
// acknowledgement, under a full read stream, comes late: storing each item's
// rows when it finishes cost 12 % of the pass.  Instead each finished 16-row
// tile is appended to the wave's LDS buffer (a 16-byte header, then the rows,
// padded by 16 bytes so the 16 rows of a column fall in different banks) and
// the buffer is written out when it is full and when the wave's work ends.
struct OutBuf {
  char* base;   // this wave's LDS buffer
  int cap;      // its bytes
  int used;     // bytes holding records (wave-uniform)
};

constexpr int kOutO = 1;   // record of normalised bf16 output rows
constexpr int kOutP = 2;   // record of partial rows (normalised, bf16) and their fp32 max, sum

// Bytes of one record (16-byte aligned): header, rows, and for partials each
// row's (max, sum).
template <int D>
__host__ __device__ constexpr int out_record_bytes(int kind, int nrows) {
  return (kind == kOutO ? 16 + nrows * (D * 2 + 16)
                        : 16 + nrows * (D * 2 + 16) + nrows * 8 + 15) / 16 * 16;
}

// Ordering of the wave's LDS writes before its reads of other lanes' data,
// and of those reads before the buffer is written again: a compiler memory
// barrier and a wait for the wave's LDS operations.
__device__ inline void lds_fence() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Write out every record of the buffer: each row with whole 16-byte chunks,
// the lanes of a row contiguous.
template <int D, int MT>
__device__ inline void out_flush(const Params& p, OutBuf& ob, int lane) {
  lds_fence();
  int off = 0;
  while (off < ob.used) {
    // header: kind, (KV head << 16) | rows, first row, qo (output) or slot (partial)
    const int4 h = *(const int4*)(ob.base + off);
    const int kind = uniform(h.x), nrows = uniform(h.y), m0 = uniform(h.z), key = uniform(h.w);
    const char* rows = ob.base + off + 16;
    if (kind == kOutO) {
      const int qo = key;
      const int gg = nrows >> 16, nr = nrows & 0xffff;
      constexpr int RS = D * 2 + 16, CPR = D / 8, RPI = 64 / CPR;
      const int c = lane % CPR, rr = lane / CPR;
      for (int r0 = 0; r0 < nr; r0 += RPI) {
        const int r = r0 + rr;
        if (r < nr) {
          const u32x4 v = *(const u32x4*)(rows + r * RS + c * 16);
          const int m = m0 + r;
          const int j = m / p.group, hh = gg * p.group + m % p.group;
          *(u32x4*)(p.out + ((int64_t)(qo + j) * p.num_q_heads + hh) * D + c * 8) = v;
        }
      }
      off += out_record_bytes<D>(kOutO, nr);
    } else {
      const int64_t slot = key;
      const int nr = nrows & 0xffff;
      constexpr int RS = D * 2 + 16, CPR = D / 8, RPI = 64 / CPR;
      const int c = lane % CPR, rr = lane / CPR;
      for (int r0 = 0; r0 < nr; r0 += RPI) {
        const int r = r0 + rr;
        if (r < nr)
          *(u32x4*)(p.part_o + (slot * (MT * 16) + m0 + r) * D + c * 8) =
              *(const u32x4*)(rows + r * RS + c * 16);
      }
      if (lane < nr)
        p.part_ml[slot * (MT * 16) + m0 + lane] = *(const float2*)(rows + nr * RS + lane * 8);
      off += out_record_bytes<D>(kOutP, nr);
    }
  }
  ob.used = 0;
  lds_fence();
}

// Finish item it: a whole item is normalised and becomes output rows; an
// item cut by a range boundary leaves its partial in the range's head slot
// (the item began in an earlier range) or tail slot (it continues later).
// Both go to the wave's LDS buffer, one record per 16-row tile.
template <int D, int MT>
__device__ inline void finish_item(const Params& p, Acc<D, MT>& a, const Item& it, int64_t rid,
                                   int lane, OutBuf& ob) {
  const int grp = lane >> 4, row = lane & 15;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) a.l[mt] = wave_sum_groups(a.l[mt]);
  const bool whole = it.j0 == 0 && it.j1 == it.n;
  const int slot = (int)(2 * rid + (it.j0 > 0 ? 0 : 1));
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    if (mt * 16 >= it.rows) break;
    const int nr = min(16, it.rows - mt * 16);
    const int kind = whole ? kOutO : kOutP;
    const int need = out_record_bytes<D>(kind, nr);
    if (ob.used + need > ob.cap) out_flush<D, MT>(p, ob, lane);
    char* rec = ob.base + ob.used;
    if (lane == 0)
      *(int4*)rec = whole ? int4{kOutO, (it.g << 16) | nr, mt * 16, it.qo}
                          : int4{kOutP, nr, mt * 16, slot};
    char* rows = rec + 16;
    if (row < nr) {
      // output rows, or a partial's rows over its own tokens (O / sum), in
      // bf16; a partial also keeps the running max and sum that weight it in
      // the merge
      const float inv = a.l[mt] > 0.f ? 1.f / a.l[mt] : 0.f;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const bf16x2 lo = {(__bf16)(a.o[mt][dt][0] * inv), (__bf16)(a.o[mt][dt][1] * inv)};
        const bf16x2 hi = {(__bf16)(a.o[mt][dt][2] * inv), (__bf16)(a.o[mt][dt][3] * inv)};
        *(u32x2*)(rows + row * (D * 2 + 16) + (dt * 16 + grp * 4) * 2) =
            u32x2{__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
      }
      if (!whole && grp == 0)
        *(float2*)(rows + nr * (D * 2 + 16) + row * 8) = make_float2(a.m[mt], a.l[mt]);
    }
    ob.used += need;
  }
}

// A segment's sequence of T spans (in work-order position, KV head, span
// order) is cut into W contiguous ranges, one per resident wave, sized by the
// wave's speed: workgroups are dealt to
// the eight XCDs in turn, and waves on odd XCDs stream HBM measurably slower
// than those on even ones, so their ranges are shorter in the ratio
// w_odd : w_even.  Every kernel derives the same ranges from T, W and the
// weights.
struct Ranges {
  int64_t T, W, we, wo, total;
  __device__ Ranges(int64_t t, int64_t waves, int w_even, int w_odd)
      : T(t), W(waves), we(w_even), wo(w_odd) {
    total = weight_before(W);
  }
  // summed weight of ranges [0, q): range q is wave q % 4 of workgroup q / 4
  __device__ int64_t weight_before(int64_t q) const {
    const int64_t k = q % 8;
    return (q / 8) * 4 * (we + wo) + (k < 4 ? k * we : 4 * we + (k - 4) * wo);
  }
  __device__ int64_t begin(int64_t rid) const { return T * weight_before(rid) / total; }
  __device__ int64_t end(int64_t rid) const { return T * weight_before(rid + 1) / total; }
  // range holding span s: the last q with begin(q) <= s, i.e. the last q
  // with weight_before(q) <= G = floor(((s + 1) * total - 1) / T), found by
  // inverting the piecewise-linear weight_before
  __device__ int64_t of(int64_t s) const {
    const int64_t G = ((s + 1) * total - 1) / T;
    const int64_t blk = 4 * (we + wo);
    const int64_t full = G / blk;
    const int64_t rem = G - full * blk;
    const int64_t k = rem < 4 * we ? rem / we : 4 + min((int64_t)3, (rem - 4 * we) / wo);
    return min(W - 1, full * 8 + k);
  }
};

// Waves a launch of W waves uses for a batch of B blocks (per KV head, over
// the segments' spans: ta spans of the reading tile's blocks, tb of the
// writing tile's), a multiple of 4, at least kMinWaves, at most W.  A small batch
// spread over every resident wave cuts each item into one-span parts whose
// merge costs more than the streaming (a one-request round ran in 65 us on
// 1024 waves and 29 us on 64); too few waves leave HBM idle.  Measured on
// MI355X: the separate attention (four-block spans) is best at about one
// wave per 20 blocks; the fused pass at B / (15 + B / 1000) waves (about 15
// blocks per wave at 1k blocks, 30 at 10-20k, 80 at 60k), and with every
// resident wave once that passes 7/8 of them.  Every kernel derives the
// same count from the segments' spans.
constexpr int kMinWaves = 64;
constexpr int kMinCopyWaves = 64;   // surplus waves that take over the fused pass's pool writes

template <int D, int MT>
__device__ inline int64_t segment_blocks(int64_t ta, int64_t tb) {
  return ta * span_blocks(D, MT, false) + tb * span_blocks(D, MT, true);
}

template <int D, int MT, bool FUSE>
__device__ inline int64_t waves_for(int64_t ta, int64_t tb, int64_t W) {
  const int64_t B = segment_blocks<D, MT>(ta, tb);
  int64_t want = FUSE ? B * 1000 / (15000 + B) : (B + 19) / 20;
  if (FUSE && 8 * want > 7 * W) want = W;
  return min(W, max((int64_t)kMinWaves, (want + 3) / 4 * 4));
}

// Work-order position whose spans [hkv*pre[i], hkv*pre[i+1]) contain span s.
__device__ inline int find_position(const uint32_t* pre, int bs, int hkv, int64_t s) {
  int lo = 0, hi = bs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if ((int64_t)hkv * pre[mid] <= s) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Span of `next` requested during the last span of `it`: next's first span,
// or kSpare when the range holds nothing after `it` (next is it).
__device__ inline int first_or_spare(const Item& it, const Item& next) {
  return next.base == it.base ? kSpare : next.j0;
}

// Table entries of the span after span j of `it`: span j+1, or next's first
// span when j is the item's last (when next is it, unused).
template <int NB, bool ARR>
__device__ inline SpanIds<NB> ids_after(const Params& p, const int32_t* __restrict__ block_table,
                                        const int32_t* __restrict__ stage_table, const Item& it,
                                        const Item& next, int j) {
  return j + 1 < it.j1 ? load_ids<NB, ARR>(p, block_table, stage_table, it, j + 1)
                       : load_ids<NB, ARR>(p, block_table, stage_table, next, next.j0);
}

// Spans [j0, j1) of one item.  The loads of the item's first span were issued
// by the caller; during its last span the first span of `next` is requested.
// When the range ends inside `it` (or with it), `next` is `it` and those
// loads are spare (every vector load of the loop is unconditional): they
// read block 0's tile of the item's KV head, which every wave's spare loads
// share, so they come from the L2 rather than HBM.
// Table entries are fetched one step before the step that uses them.
template <int D, int MT, int NB, bool ARR, bool STORE>
__device__ inline void run_item(const Params& p, const int32_t* __restrict__ block_table,
                                const int32_t* __restrict__ stage_table, const Item& it,
                                const Item& next, KOps<D, NB>& kreg, VOps<D, NB>& vreg,
                                SpanRef<NB>& cur, QOps<MT, D>& q, Acc<D, MT>& a, int total_q,
                                int lane) {
  SpanIds<NB> ids = ids_after<NB, ARR>(p, block_table, stage_table, it, next, it.j0);
  for (int j = it.j0; j + 1 < it.j1; ++j) {
    const SpanIds<NB> ids2 = ids_after<NB, ARR>(p, block_table, stage_table, it, next, j + 1);
    span_step<D, MT, NB, ARR, STORE, false>(kreg, vreg, cur, it, j + 1, ids, q, p, a, it.win,
                                            it.L, total_q, lane);
    ids = ids2;
  }
  // the last span also brings in the next item's first K/V, and (reading
  // only) its Q; the writing tile has no registers to spare there (its Q
  // loaded here spilled and cost 4 %), so it loads Q at the switch
  span_step<D, MT, NB, ARR, STORE, !ARR>(kreg, vreg, cur, next, first_or_spare(it, next), ids, q,
                                         p, a, it.win, it.L, total_q, lane);
}

// The record of range rid for the merge: the item it cuts at its end (if that
// item began in the range), or none.
__device__ __attribute__((always_inline)) inline void write_cut_rec(
    const Params& p, int64_t rid, int lane, bool cut, int64_t base, int n, int r, int g, int qo,
    int nq) {
  if (lane != 0) return;
  CutRec* c = p.cut_rec + rid;
  c->base = base;
  c->n = cut ? n : -1;
  c->r = r;
  c->g = g;
  c->qo = qo;
  c->nq = nq;
}

__device__ __attribute__((always_inline)) inline void write_no_cut(const Params& p, int64_t rid,
                                                                    int lane) {
  write_cut_rec(p, rid, lane, false, 0, 0, 0, 0, 0, 0);
}

// One range [s, s1) of global spans, range id rid: online softmax over every
// (request, KV head) item the range touches.  ORD: positions map to requests
// through the fused pass's work order; ARR: the range lies in the arriving
// segment (tiles read from the staging pool and, with `store`, written to the
// worker pool).
template <int D, int MT, int NB, bool ORD, bool ARR>
__device__ void process_range(const Params& p, const int32_t* __restrict__ block_table,
                              const int32_t* __restrict__ stage_table,
                              const int32_t* __restrict__ seq_lens,
                              const int32_t* __restrict__ q_indptr, const uint32_t* pre,
                              const uint16_t* order, int total_q, int64_t rid, int64_t s,
                              int64_t s1, int lane, OutBuf& ob, bool store) {
  const int hkv = p.num_kv_heads;
  const int pos0 = uniform(find_position(pre, p.bs, hkv, s));
  const int r0 = uniform(request_at<ORD>(order, pos0));
  const int64_t pr0 = uniform64(pre[pos0]);
  // the item holding span position s
  const int n0 = spans_of<NB>(clamp_len(p, seq_lens, r0));
  const int g0 = (int)min((int64_t)hkv - 1, (s - (int64_t)hkv * pr0) / n0);
  Item it = make_item<NB, ARR>(p, seq_lens, q_indptr, stage_table, pos0, r0, g0, pr0, s, s1,
                               total_q);
  if (it.j0 >= it.j1) {
    if (it.pos == p.bs - 1 && it.g == hkv - 1) return write_no_cut(p, rid, lane);
    it = next_item<NB, ORD, ARR>(p, seq_lens, q_indptr, stage_table, order, it, s, s1, total_q);
    if (it.j0 >= it.j1) return write_no_cut(p, rid, lane);   // no span lies here
  }
  // next item with a span in the range (or `it` itself when none)
  auto following = [&](const Item& cur) {
    const bool last = cur.pos == p.bs - 1 && cur.g == hkv - 1;
    if (last || cur.base + (int64_t)cur.n >= s1) return cur;
    return next_item<NB, ORD, ARR>(p, seq_lens, q_indptr, stage_table, order, cur, s, s1,
                                   total_q);
  };
  Item next = following(it);
  bool more = next.base != it.base;

  // the first item's Q; reading only, each later item's Q comes with its
  // first K/V loads, during the previous item's last span (one set of Q
  // registers: a second copy for a prefetch one item ahead spilled in the
  // writing tile, and moving it between register files made the wave wait
  // for all its loads at every item switch)
  QOps<MT, D> qc;
  load_q<D, MT>(qc, p, it, total_q, lane);
  SpanRef<NB> cur =
      make_ref<NB, ARR>(p, it, it.j0, load_ids<NB, ARR>(p, block_table, stage_table, it, it.j0));
  KOps<D, NB> kreg;
  VOps<D, NB> vreg;
  load_k<D, NB>(kreg, cur, lane);
  load_v<D, NB>(vreg, cur, lane);
  while (true) {
    Acc<D, MT> a;
    init_acc<D, MT>(a, p, it, lane);
    if (ARR && store)
      run_item<D, MT, NB, ARR, ARR>(p, block_table, stage_table, it, next, kreg, vreg, cur, qc, a,
                                    total_q, lane);
    else
      run_item<D, MT, NB, ARR, false>(p, block_table, stage_table, it, next, kreg, vreg, cur, qc,
                                      a, total_q, lane);
    finish_item<D, MT>(p, a, it, rid, lane, ob);
    if (!more) {
      // the range's last item, if it began here and continues past the range
      const bool cut = it.j0 == 0 && it.j1 < it.n && it.rows > 0;
      write_cut_rec(p, rid, lane, cut, it.base, it.n, it.r, it.g, it.qo, it.nq);
      break;
    }
    // switch to the next item (its first span, and Q when reading only, are
    // already requested)
    if constexpr (ARR) load_q<D, MT>(qc, p, next, total_q, lane);
    it = next;
    next = following(it);
    more = next.base != it.base;
  }
}

// Sum of x over the workgroup's 256 threads, in every thread.
__device__ inline uint32_t block_sum(uint32_t x, uint32_t* s_tmp, int lane, int wave) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  __syncthreads();   // s_tmp may still be read from the previous call
  if (lane == 0) s_tmp[wave] = x;
  __syncthreads();
  return s_tmp[0] + s_tmp[1] + s_tmp[2] + s_tmp[3];
}

// The fused pass's pool writes done by waves of their own: copy wave c of n
// takes arriving spans c, c + n, ... (per request, in work order) and copies
// each of their blocks, all KV heads and both planes, from the staging pool to
// the worker pool.  The blocks written are exactly those the attention waves
// would store: a span's blocks up to the context (at least one), with staging
// and destination ids in range.
template <int D, int NB>
__device__ void copy_staged(const Params& p, const int32_t* __restrict__ block_table,
                            const int32_t* __restrict__ stage_table,
                            const int32_t* __restrict__ seq_lens, const uint32_t* pre,
                            const uint16_t* order, int n_res, int64_t c, int64_t n, int lane) {
  const int64_t s0 = pre[n_res], s_end = pre[p.bs];
  const int64_t words = (int64_t)p.num_kv_heads * kBlock * D * 2 / 16;   // 16-byte words per block
  for (int64_t s = s0 + c; s < s_end; s += n) {
    const int pos = uniform(find_position(pre, p.bs, 1, s));
    const int r = uniform((int)order[pos]);
    const int L = clamp_len(p, seq_lens, r);
    const int j = (int)(s - pre[pos]);
    const int t = j * NB * kBlock;
    const int nb = max(1, min(NB, (L - t + kBlock - 1) / kBlock));
    const int64_t row = (int64_t)r * p.max_blocks_per_seq;
    for (int b = 0; b < nb; ++b) {
      const int e = j * NB + b;
      const int32_t sid = uniform(stage_table[row + e]);
      const int32_t did = uniform(block_table[row + e]);
      if (sid < 0 || sid >= p.stage_blocks || did < 0 || did >= p.num_blocks) continue;
      const u32x4* ks = (const u32x4*)p.k_stage + (int64_t)sid * words;
      const u32x4* vs = (const u32x4*)p.v_stage + (int64_t)sid * words;
      u32x4* kd = (u32x4*)p.k_dst + (int64_t)did * words;
      u32x4* vd = (u32x4*)p.v_dst + (int64_t)did * words;
      for (int64_t w0 = 0; w0 < words; w0 += 4 * 64) {
        u32x4 kv[4], vv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int64_t w = w0 + u * 64 + lane;
          kv[u] = w < words ? __builtin_nontemporal_load(ks + w) : u32x4{0, 0, 0, 0};
          vv[u] = w < words ? __builtin_nontemporal_load(vs + w) : u32x4{0, 0, 0, 0};
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int64_t w = w0 + u * 64 + lane;
          if (w < words) {
            __builtin_nontemporal_store(kv[u], kd + w);
            __builtin_nontemporal_store(vv[u], vd + w);
          }
        }
      }
    }
  }
}

// One dispatch of W waves (W / 4 workgroups of 4 independent waves).
//
// Work order: the fused variant places the batch's resident requests first
// (positions [0, nA)) and its arriving requests after them, each group in
// request order; the spans of the two segments are split separately into W
// ranges each, and wave w takes range w of both segments, one after the
// other.  Every wave therefore does its share of the arriving requests (the
// reads and the write-back of staged tiles) in the same phase of the launch:
// HBM serves reads and writes gathered in time markedly faster than the same
// writes spread through a read stream.  Without fusion there is one segment
// and position i is request i.
template <int D, int MT, bool FUSE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(waves_per_simd(D, MT, FUSE))))
void verify_attention_kernel(Params p, const int32_t* __restrict__ block_table,
                             const int32_t* __restrict__ stage_table,
                             const int32_t* __restrict__ seq_lens,
                             const int32_t* __restrict__ q_indptr) {
  constexpr int NBA = span_blocks(D, MT, false);   // resident (or only) segment
  constexpr int NBB = span_blocks(D, MT, true);    // arriving segment
  extern __shared__ uint32_t s_pre[];   // [bs + 1] span prefix by position, then uint16 order[bs]
  uint16_t* s_order = (uint16_t*)(s_pre + p.bs + 1);
  __shared__ uint32_t s_wsum[3][4];
  __shared__ uint32_t s_red[4];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = uniform(tid >> 6);
  const int total_q = uniform(q_indptr[p.bs]);

  // resident requests and their spans (the first segment)
  uint32_t n_res = p.bs, u_res = 0;
  if constexpr (FUSE) {
    uint32_t c = 0, u = 0;
    for (int r = tid; r < p.bs; r += 256)
      if (!is_arriving(p, stage_table, r)) {
        ++c;
        u += spans_of<NBA>(clamp_len(p, seq_lens, r));
      }
    n_res = block_sum(c, s_red, lane, wave);
    u_res = block_sum(u, s_red, lane, wave);
  }
  // positions and span prefixes; every workgroup keeps its own copy, the
  // first also stores them for the merge kernel
  uint32_t c_arr = 0, c_ua = 0, c_ur = 0;   // before the chunk: arriving requests,
                                            // their spans, resident spans
  for (int base = 0; base < p.bs; base += 256) {
    const int r = base + tid;
    const bool in = r < p.bs;
    const bool arr = in && FUSE && is_arriving(p, stage_table, r);
    const int L = in ? clamp_len(p, seq_lens, r) : 0;
    const uint32_t n = in ? (arr ? spans_of<NBB>(L) : spans_of<NBA>(L)) : 0;
    uint32_t v[3] = {arr ? 1u : 0u, arr ? n : 0u, arr ? 0u : n};
    uint32_t incl[3] = {v[0], v[1], v[2]};
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
#pragma unroll
      for (int k = 0; k < 3; ++k) {
        const uint32_t y = __shfl_up(incl[k], o);
        if (lane >= o) incl[k] += y;
      }
    }
    if (lane == 63) {
#pragma unroll
      for (int k = 0; k < 3; ++k) s_wsum[k][wave] = incl[k];
    }
    __syncthreads();
    uint32_t before[3] = {c_arr, c_ua, c_ur};
#pragma unroll
    for (int k = 0; k < 3; ++k)
      for (int i = 0; i < wave; ++i) before[k] += s_wsum[k][i];
    if (in) {
      const uint32_t a_before = before[0] + incl[0] - v[0];
      const int pos = arr ? (int)(n_res + a_before) : r - (int)a_before;
      const uint32_t pre = arr ? u_res + before[1] + incl[1] - v[1] : before[2] + incl[2] - v[2];
      s_pre[pos] = pre;
      if constexpr (FUSE) s_order[pos] = (uint16_t)r;
      if (blockIdx.x == 0) {
        p.prefix[pos] = pre;
        p.pos_of[r] = pos;
      }
    }
    c_arr += s_wsum[0][0] + s_wsum[0][1] + s_wsum[0][2] + s_wsum[0][3];
    c_ua += s_wsum[1][0] + s_wsum[1][1] + s_wsum[1][2] + s_wsum[1][3];
    c_ur += s_wsum[2][0] + s_wsum[2][1] + s_wsum[2][2] + s_wsum[2][3];
    __syncthreads();
  }
  if (tid == 0) {
    s_pre[p.bs] = c_ua + c_ur;
    if (blockIdx.x == 0) {
      p.prefix[p.bs] = c_ua + c_ur;
      p.pos_of[p.bs] = n_res;
      p.pos_of[p.bs + 1] = c_ur;   // spans of the resident segment, per KV head
      p.pos_of[p.bs + 2] = c_ua;   // of the arriving segment
    }
  }
  __syncthreads();

  const int64_t hkv = p.num_kv_heads;
  const int64_t ta = hkv * s_pre[n_res], tb = hkv * s_pre[p.bs] - ta;
  const int64_t rid = (int64_t)blockIdx.x * 4 + wave;
  if (total_q <= 0) {
    // no query rows: nothing to attend, but the arriving requests' blocks
    // still move to the worker pool (the preparation does not depend on the
    // queries), copied by every wave
    if (FUSE && tb > 0)
      copy_staged<D, NBB>(p, block_table, stage_table, seq_lens, s_pre, s_order, (int)n_res, rid,
                          p.num_waves, lane);
    return;
  }
  const int64_t W = waves_for<D, MT, FUSE>(ta, tb, p.num_waves);
  // a batch too small for every resident wave: the surplus waves write the
  // staged blocks to the worker pool, so the attention waves stream without
  // stores, when there are enough of them and the batch is small enough for
  // the second read of the staged blocks to stay hidden (the copy's bytes per
  // copy wave at most 0.4 of the attention's per wave; measured: 4 requests
  // 6 % faster, 8 requests 3 %, 16 requests 21 % slower without that bound)
  const int64_t ncopy = p.num_waves - W;
  const int64_t tb_blocks = tb * NBB;
  const bool copy_mode = FUSE && tb > 0 && ncopy >= kMinCopyWaves &&
                         5 * tb_blocks * W <= segment_blocks<D, MT>(ta, tb) * ncopy;
  if (rid >= W) {
    if (copy_mode)
      copy_staged<D, NBB>(p, block_table, stage_table, seq_lens, s_pre, s_order, (int)n_res,
                          rid - W, ncopy, lane);
    return;
  }
  const Ranges ra(ta, W, p.w_even, p.w_odd), rb(tb, W, p.w_even, p.w_odd_b);
  // this wave's output buffer follows the span prefix and the work order
  OutBuf ob;
  ob.base = (char*)s_pre + p.out_off + wave * p.out_cap;
  ob.cap = p.out_cap;
  ob.used = 0;
  // resident range first (reading only, the reading tile's spans), then the
  // arriving range (writes last, the writing tile's spans)
  {
    const int64_t b = uniform64(ra.begin(rid)), e = uniform64(ra.end(rid));
    if (b < e)
      process_range<D, MT, NBA, FUSE, false>(p, block_table, stage_table, seq_lens, q_indptr,
                                             s_pre, s_order, total_q, rid, b, e, lane, ob, false);
    else
      write_no_cut(p, rid, lane);
  }
  if constexpr (FUSE) {
    const int64_t b = uniform64(ta + rb.begin(rid)), e = uniform64(ta + rb.end(rid));
    const int64_t rid_b = p.num_waves + rid;
    if (b < e)
      process_range<D, MT, NBB, true, true>(p, block_table, stage_table, seq_lens, q_indptr,
                                            s_pre, s_order, total_q, rid_b, b, e, lane, ob,
                                            !copy_mode);
    else
      write_no_cut(p, rid_b, lane);
  }
  out_flush<D, MT>(p, ob, lane);
}

// Threads per row of the merge kernel's 256: a power of two dividing the
// row's float4 count, with every row of a 16-row-tile item covered.
__host__ __device__ constexpr int merge_threads_per_row(int vec, int rows) {
  int t = 1;
  while (t * 2 <= 256 / rows && t * 2 <= vec) t *= 2;
  return t;
}

// Merge the partials of every item that a range boundary cut, in range order
// (deterministic, no atomics).  One workgroup per range (of each segment):
// it finishes the item the range cuts at its end, if that item began in the
// range, from the range's record; the ranges holding the item's other parts
// and their partial slots are found once per workgroup.
template <int D, int MT, bool FUSE>
__global__ __launch_bounds__(256) void combine_kernel(Params p) {
  __shared__ int64_t s_slot[256];   // partial slots of the item, in range order
  __shared__ int s_nslot;
  const int x = blockIdx.x;
  const int tid = threadIdx.x;
  const bool seg_b = x >= p.num_waves;
  const int64_t q = seg_b ? x - p.num_waves : x;
  const int hkv = p.num_kv_heads;
  // all independent loads: the row count, the batch's spans, the record
  const int total_q = p.q_indptr[p.bs];
  const int64_t ta = (int64_t)hkv * p.pos_of[p.bs + 1];
  const int64_t tb = (int64_t)hkv * p.pos_of[p.bs + 2];
  const CutRec rec = p.cut_rec[x];
  if (total_q <= 0) return;   // the main kernel attended nothing and wrote no record
  const int64_t W = waves_for<D, MT, FUSE>(ta, tb, p.num_waves);
  if (q >= W) return;         // no wave took this range: its record is stale
  if (rec.n < 0 || rec.nq <= 0) return;
  const int64_t off = seg_b ? ta : 0;
  const int64_t qoff = seg_b ? p.num_waves : 0;
  const Ranges R(seg_b ? tb : ta, W, p.w_even, seg_b ? p.w_odd_b : p.w_odd);
  const int n = rec.n, g = rec.g, qo = rec.qo;
  const int nq = min(rec.nq, max(0, total_q - qo));
  const int64_t base = rec.base;
  const int64_t ra = q;                                      // the item began in this range
  const int64_t rb = uniform64(R.of(base - off + n - 1));   // its last span's range
  if (rb <= ra || nq == 0) return;
  const int rows = p.group * nq;
  // thread layout: kTPR threads per row, each holding kPer float4 elements of
  // it (lane-contiguous per element index), so a thread reads one (max, sum)
  // per part; few registers, so every range's workgroup is resident at once
  constexpr int kVec = D / 4;
  constexpr int kTPR = merge_threads_per_row(kVec, MT * 16);
  constexpr int kPer = kVec / kTPR;
  const int m = tid / kTPR;                 // this thread's row (idle when >= rows)
  const int c = tid % kTPR;
  const int mld = min(m, rows - 1);         // loads clamped into the item's rows
  float mrun = -INFINITY, drun = 0.f;
  f32x4 orun[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) orun[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  // running merge over the ranges, 256 at a time (an item rarely spans more
  // than a few)
  for (int64_t q0 = ra; q0 <= rb; q0 += 256) {
    const int64_t q = q0 + tid;
    if (q <= rb) {
      int j0, j1;
      spans_in(base, n, off + R.begin(q), off + R.end(q), j0, j1);
      s_slot[tid] = j0 < j1 ? 2 * (qoff + q) + (j0 > 0 ? 0 : 1) : -1;
    }
    __syncthreads();
    if (tid == 0) {   // keep the ranges holding a part, in order
      const int span = (int)min((int64_t)256, rb - q0 + 1);
      int n = 0;
      for (int k = 0; k < span; ++k)
        if (s_slot[k] >= 0) s_slot[n++] = s_slot[k];
      s_nslot = n;
    }
    __syncthreads();
    const int cnt = s_nslot;
    // two parts at a time (a cut item has two in most cases): every load is
    // issued before the first merge
    for (int k0 = 0; k0 < cnt; k0 += 2) {
      float2 ml[2];
      f32x4 o[2][kPer];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int64_t slot = s_slot[min(k0 + u, cnt - 1)];
        const int64_t row = slot * (MT * 16) + mld;
        ml[u] = p.part_ml[row];
        const u32x2* src = (const u32x2*)(p.part_o + row * D) + c;
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
          // bf16 to fp32 by placing each half in the high bits (exact); the
          // compiler's conversion of bf16 vector elements read the low word
          // for both halves here
          const u32x2 w = src[i * kTPR];
          o[u][i] = f32x4{__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u),
                          __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xffff0000u)};
        }
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        if (k0 + u >= cnt || ml[u].x == -INFINITY) continue;   // no visible token there
        const float mx = fmaxf(mrun, ml[u].x);
        const float a = mrun == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mrun - mx);
        const float b = __builtin_amdgcn_exp2f(ml[u].x - mx);
        const float bl = b * ml[u].y;   // the part's weight: its rows are O / sum
#pragma unroll
        for (int i = 0; i < kPer; ++i) orun[i] = a * orun[i] + bl * o[u][i];
        drun = a * drun + bl;
        mrun = mx;
      }
    }
    __syncthreads();
  }
  if (m >= rows) return;
  const float inv = drun > 0.f ? 1.f / drun : 0.f;
  const int j = m / p.group;
  const int h = g * p.group + m % p.group;
  uint16_t* dst = p.out + ((int64_t)(qo + j) * p.num_q_heads + h) * D;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const bf16x2 lo = {(__bf16)(orun[i][0] * inv), (__bf16)(orun[i][1] * inv)};
    const bf16x2 hi = {(__bf16)(orun[i][2] * inv), (__bf16)(orun[i][3] * inv)};
    *(u32x2*)(dst + (i * kTPR + c) * 4) =
        u32x2{__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
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
  size_t lds_bytes;  // dynamic LDS of the span prefix and work order
  size_t prefix_bytes, part_o_bytes, part_ml_bytes, cut_rec_bytes, ws_bytes;
};

// Launch facts of one kernel instantiation on one device, queried once per
// (device, instantiation) and kept for the process: the waves the device
// keeps resident (CUs x workgroups per CU x 4), the LDS a workgroup may use
// and the kernel's static LDS.
struct KernelInfo {
  int cus;
  int blocks;         // workgroups per CU the registers allow (capped by waves_per_simd)
  int lds_block;      // LDS one workgroup may address
  int lds_cu;         // LDS of one CU
  size_t static_lds;
  bool ok;
};

constexpr int kMaxDevices = 64;
std::mutex g_info_mu;
KernelInfo g_info[kMaxDevices][2][2][4];   // [device][fuse][head_dim 128][mt - 1]
bool g_info_set[kMaxDevices][2][2][4];
// Test and tuning hook (nsd_set_attention_waves): a wave count replacing
// the device's, 0 for the device's own.
std::atomic<int> g_waves_override{0};

KernelInfo kernel_info(int d, int mt, bool fuse) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return KernelInfo{0, 0, 0, 0, 0, false};
  }
  const int f = fuse ? 1 : 0, h = d == 128 ? 1 : 0, m = std::min(std::max(mt, 1), 4) - 1;
  std::lock_guard<std::mutex> lock(g_info_mu);
  if (g_info_set[dev][f][h][m]) return g_info[dev][f][h][m];
  KernelInfo ki{0, 0, 0, 0, 0, false};
  int cus = 0, blocks = 0, lds_block = 0, lds_cu = 0;
  hipFuncAttributes fa;
  const void* k = fuse ? kernel_for<true>(d, mt) : kernel_for<false>(d, mt);
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k, 256, 0) == hipSuccess &&
      hipDeviceGetAttribute(&lds_block, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) ==
          hipSuccess &&
      hipDeviceGetAttribute(&lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) ==
          hipSuccess &&
      hipFuncGetAttributes(&fa, k) == hipSuccess && cus > 0 && blocks > 0 && lds_cu > 0) {
    // as many workgroups per CU as the registers allow, up to the waves per
    // SIMD the kernel is compiled for
    ki.cus = cus;
    ki.blocks = std::min(blocks, waves_per_simd(d, mt, fuse));
    ki.lds_block = lds_block;
    ki.lds_cu = lds_cu;
    ki.static_lds = fa.sharedSizeBytes;
    ki.ok = true;
    g_info[dev][f][h][m] = ki;
    g_info_set[dev][f][h][m] = true;
  } else {
    (void)hipGetLastError();
  }
  return ki;
}

// Workgroups per CU for a launch whose span prefix and work order take
// pre_bytes of LDS: the kernel's register limit, unless that leaves a
// workgroup (with its share of the CU's LDS, so that all of them are resident
// at once, as the static split assumes) too little room for four output
// buffers of one record each; then fewer.
int blocks_for(const KernelInfo& ki, int d, size_t pre_bytes) {
  const size_t min_cap = d == 64 ? out_record_bytes<64>(kOutP, 16) : out_record_bytes<128>(kOutP, 16);
  for (int b = ki.blocks; b > 1; --b)
    if ((size_t)std::min(ki.lds_block, ki.lds_cu / b) >= ki.static_lds + pre_bytes + 4 * min_cap)
      return b;
  return 1;
}

// LDS one workgroup of the launch may use.
int lds_budget(const KernelInfo& ki, int d, size_t pre_bytes) {
  return std::min(ki.lds_block, ki.lds_cu / blocks_for(ki, d, pre_bytes));
}

// Waves a launch uses: the override when set, else the device's resident
// waves for this launch (256 CUs x 2 workgroups when the device cannot be
// queried, which only sizes a workspace query; a launch then fails on the
// LDS query).
int resident_waves(int d, int mt, bool fuse, size_t pre_bytes) {
  const int w = g_waves_override.load(std::memory_order_relaxed);
  if (w > 0) return w;
  const KernelInfo ki = kernel_info(d, mt, fuse);
  return ki.ok ? ki.cus * blocks_for(ki, d, pre_bytes) * 4 : 256 * 2 * 4;
}

bool make_plan(int bs, int hq, int hkv, int d, int max_q, int max_seq_len, bool fuse,
               Plan* pl) {
  if (bs < 0 || bs > kMaxBatch || hq < 1 || hkv < 1 || hq % hkv || (d != 64 && d != 128) ||
      max_q < 1 || max_seq_len < 0)
    return false;
  const int64_t rows = (int64_t)(hq / hkv) * max_q;
  if (rows > kMaxRows) return false;
  pl->mt = (rows + 15) / 16;
  pl->lds_bytes = ((size_t)bs + 1) * sizeof(uint32_t) + ((size_t)bs * sizeof(uint16_t) + 3) / 4 * 4;
  pl->num_waves = resident_waves(d, pl->mt, fuse, (pl->lds_bytes + 15) / 16 * 16);
  // a head and a tail slot per range, W ranges in each of the two segments
  const size_t slots = 4 * (size_t)pl->num_waves * pl->mt * 16;
  pl->prefix_bytes = ((2 * ((size_t)bs + 1) + 2) * sizeof(uint32_t) + 255) / 256 * 256;
  pl->part_o_bytes = slots * d * sizeof(uint16_t);
  pl->part_ml_bytes = slots * sizeof(float2);
  pl->cut_rec_bytes = 2 * (size_t)pl->num_waves * sizeof(CutRec);
  pl->ws_bytes = pl->prefix_bytes + pl->part_o_bytes + pl->part_ml_bytes + pl->cut_rec_bytes;
  return true;
}

template <int D, int MT, bool FUSE>
void launch(const Params& p, int bs, size_t lds_bytes, hipStream_t stream) {
  hipLaunchKernelGGL((verify_attention_kernel<D, MT, FUSE>), dim3(p.num_waves / 4), dim3(256),
                     lds_bytes, stream, p, p.block_table, p.stage_table, p.seq_lens,
                     p.q_indptr);
  hipLaunchKernelGGL((combine_kernel<D, MT, FUSE>), dim3((FUSE ? 2 : 1) * p.num_waves),
                     dim3(256), 0, stream, p);
  (void)bs;
}

template <int D, bool FUSE>
void launch_d(const Params& p, int mt, int bs, size_t lds_bytes, hipStream_t stream) {
  switch (mt) {
    case 1: launch<D, 1, FUSE>(p, bs, lds_bytes, stream); break;
    case 2: launch<D, 2, FUSE>(p, bs, lds_bytes, stream); break;
    case 3: launch<D, 3, FUSE>(p, bs, lds_bytes, stream); break;
    default: launch<D, 4, FUSE>(p, bs, lds_bytes, stream); break;
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
  if ((int64_t)(num_q_heads / num_kv_heads) * max_q_per_seq > kMaxRows)
    return fail(NSD_ERR_UNSUPPORTED, "%s: (Hq/Hkv)*max_q_per_seq = %lld exceeds %d", fn,
                (long long)(num_q_heads / num_kv_heads) * max_q_per_seq, kMaxRows);
  if (max_seq_len < 1 || max_blocks_per_seq < 1 || num_blocks < 1)
    return fail(NSD_ERR_SHAPE, "%s: max_seq_len, max_blocks_per_seq and num_blocks must be "
                ">= 1", fn);
  if (fuse && stage_blocks < 0) return fail(NSD_ERR_SHAPE, "%s: stage_num_blocks < 0", fn);
  // tiles (block, KV head) are indexed with 32-bit integers
  if (num_blocks > INT32_MAX / num_kv_heads || (fuse && stage_blocks > INT32_MAX / num_kv_heads))
    return fail(NSD_ERR_UNSUPPORTED, "%s: more than 2^31-1 (block, KV head) tiles in a pool", fn);
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
  // dynamic LDS: the span prefix and work order, then one output buffer per
  // wave taking the rest of what a workgroup may have (at least one record)
  const KernelInfo ki = kernel_info(head_dim, pl.mt, fuse);
  if (!ki.ok) return fail(NSD_ERR_HIP, "%s: the device's LDS size could not be queried", fn);
  const size_t pre_bytes = (pl.lds_bytes + 15) / 16 * 16;
  const int lds_max = lds_budget(ki, head_dim, pre_bytes);
  const size_t fixed = ki.static_lds + pre_bytes;
  const size_t per_wave = (size_t)lds_max > fixed ? ((size_t)lds_max - fixed) / 4 / 16 * 16 : 0;
  const size_t min_cap = head_dim == 64 ? out_record_bytes<64>(kOutP, 16)
                                        : out_record_bytes<128>(kOutP, 16);
  if (per_wave < min_cap)
    return fail(NSD_ERR_UNSUPPORTED, "%s: bs=%d needs %zu bytes of LDS, %d available", fn, bs,
                fixed + 4 * min_cap, lds_max);

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
  p.prefix = (uint32_t*)ws;
  p.pos_of = p.prefix + bs + 1;
  p.part_o = (uint16_t*)(ws + pl.prefix_bytes);
  p.part_ml = (float2*)(ws + pl.prefix_bytes + pl.part_o_bytes);
  p.cut_rec = (CutRec*)(ws + pl.prefix_bytes + pl.part_o_bytes + pl.part_ml_bytes);
  p.num_blocks = (int32_t)num_blocks;
  p.stage_blocks = fuse ? (int32_t)stage_blocks : 0;
  p.bs = bs;
  p.max_blocks_per_seq = max_blocks_per_seq;
  p.num_q_heads = num_q_heads;
  p.num_kv_heads = num_kv_heads;
  p.group = num_q_heads / num_kv_heads;
  p.max_q = max_q_per_seq;
  p.max_seq_len = max_seq_len;
  p.num_waves = pl.num_waves;
  // measured HBM streaming speed of odd-XCD waves relative to even ones, in
  // the read-only resident segment and in the arriving segment (which also
  // writes, widening the gap)
  p.w_even = 100;
  p.w_odd = 94;
  p.w_odd_b = 91;
  p.scale_log2 = scale * 1.4426950408889634f;
  p.out_off = (int32_t)pre_bytes;
  p.out_cap = (int32_t)per_wave;
  const size_t lds_bytes = pre_bytes + 4 * per_wave;

  clear_stale_error();
  if (fuse) {
    if (head_dim == 64) launch_d<64, true>(p, pl.mt, bs, lds_bytes, (hipStream_t)stream);
    else launch_d<128, true>(p, pl.mt, bs, lds_bytes, (hipStream_t)stream);
  } else {
    if (head_dim == 64) launch_d<64, false>(p, pl.mt, bs, lds_bytes, (hipStream_t)stream);
    else launch_d<128, false>(p, pl.mt, bs, lds_bytes, (hipStream_t)stream);
  }
  return check_launch(fn);
}

}  // namespace

extern "C" nsd_status nsd_set_attention_waves(int32_t waves) {
  if (waves < 0 || waves % 4 || waves > (1 << 20))
    return nsd::fail(NSD_ERR_SHAPE, "set_attention_waves: waves must be 0 or a positive "
                     "multiple of 4 up to 2^20 (got %d)", waves);
  g_waves_override.store(waves, std::memory_order_relaxed);
  return NSD_OK;
}

extern "C" int32_t nsd_attention_waves(void) {
  return g_waves_override.load(std::memory_order_relaxed);
}

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
