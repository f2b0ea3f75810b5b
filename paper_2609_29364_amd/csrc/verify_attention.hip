// Verification attention: every request's anchor + K proposal queries attend,
// causally, to its paged KV cache (Section 1: one target forward verifies all
// proposals; Appendix G.2/H: anchor plus depth-d proposals; Section 3: paged,
// append-dominant cache that already holds the window).
//
// Design (gfx950, wave64, bf16 MFMA 16x16x32):
// * Work item = (request r, KV head g, context split).  One wave owns an item;
//   the (Hq/Hkv) query heads x n_q queries that share KV head g form the M
//   rows of its tile products, so each K/V byte is read from HBM once for the
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
//   lane-local.
// * Two 16-token blocks (a 32-token span) per step; the next span's loads are
//   issued before the current span's math (register double buffering).
// * Long contexts are cut into splits of `split_tokens`; each split writes
//   (O unnormalised, running max, sum) partials and a second kernel merges
//   them in split order (deterministic, no atomics).  A request that fits one
//   split writes its output directly.
// * Masked tokens (past a query's position, past L_r, or in a block whose id
//   is out of range) are removed by selection: scores become -inf and V
//   elements past L_r are zeroed, so NaN-filled unused slots never leak.
#include "nsd_internal.h"

#include <math.h>
#include <stdlib.h>

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

constexpr int kBlock = 16;   // token slots per KV block
constexpr int kSpan = 32;    // tokens per main-loop step
constexpr int kMaxRows = 64; // (Hq/Hkv) * max_q_per_seq limit

struct Params {
  const uint16_t* q;
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  const int32_t* block_table;
  const int32_t* seq_lens;
  const int32_t* q_indptr;
  uint16_t* out;
  float* part_o;     // [bs][Hkv][max_splits][MT*16][D]
  float2* part_ml;   // [bs][Hkv][max_splits][MT*16]: (running max, sum)
  int64_t num_blocks;
  int32_t max_blocks_per_seq;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t group;
  int32_t max_q;
  int32_t max_seq_len;
  int32_t split_tokens;
  int32_t max_splits;
  int32_t waves_per_wg;
  float scale_log2;  // softmax scale * log2(e)
};

template <int D>
struct Span {
  u32x4 k[2][D / 32];   // K operands of the span's two blocks
  u32x2 v[2][D / 16];   // V^T operand halves of the two blocks
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

__device__ inline uint32_t keep_mask(int n_valid_pairs_elems) {
  // mask for one 32-bit word holding two bf16 (element 0 in the low half)
  return n_valid_pairs_elems <= 0 ? 0u : (n_valid_pairs_elems == 1 ? 0x0000ffffu : 0xffffffffu);
}

template <int D>
__device__ inline void issue_span(Span<D>& s, const Params& p, const int32_t* bt, int g,
                                  int t, int L, int lane) {
  const int row = lane & 15, grp = lane >> 4;
  s.t = t;
  const int b0 = t / kBlock;
  int32_t id0 = bt[b0];
  int32_t id1 = (t + kBlock < L) ? bt[b0 + 1] : id0;
  s.bad0 = id0 < 0 || id0 >= p.num_blocks;
  if (s.bad0) id0 = 0;
  s.bad1 = (t + kBlock < L) && (id1 < 0 || id1 >= p.num_blocks);
  if (id1 < 0 || id1 >= p.num_blocks) id1 = id0;
  const int64_t hb0 = ((int64_t)id0 * p.num_kv_heads + g) * (D * kBlock);
  const int64_t hb1 = ((int64_t)id1 * p.num_kv_heads + g) * (D * kBlock);
  const uint16_t* k0 = p.k_cache + hb0;
  const uint16_t* k1 = p.k_cache + hb1;
  const uint16_t* v0 = p.v_cache + hb0;
  const uint16_t* v1 = p.v_cache + hb1;
#pragma unroll
  for (int kk = 0; kk < D / 32; ++kk) {
    const int off = ((kk * 4 + grp) * kBlock + row) * 8;
    s.k[0][kk] = *(const u32x4*)(k0 + off);
    s.k[1][kk] = *(const u32x4*)(k1 + off);
  }
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const int off = (dt * 16 + row) * kBlock + grp * 4;
    s.v[0][dt] = *(const u32x2*)(v0 + off);
    s.v[1][dt] = *(const u32x2*)(v1 + off);
  }
}

template <int D, int MT>
__device__ inline void compute_span(const Span<D>& s, const bf16x8 (&qop)[MT][D / 32],
                                    f32x4 (&acc)[MT][D / 16], float (&m_run)[MT],
                                    float (&l_run)[MT], const int (&pos)[MT], int L,
                                    int win, float scale_log2, int lane) {
  const int grp = lane >> 4;
  // scores S^T[token][row] for both blocks
  f32x4 st[2][MT];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < D / 32; ++kk)
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, s.k[h][kk]),
                                                    qop[mt][kk], c, 0, 0, 0);
      st[h][mt] = c;
    }
  const bool need_mask = (s.t + kSpan > win) || s.bad0 || s.bad1;
  bf16x8 pop[MT];
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
  // V^T operands; elements of tokens >= L (or of bad blocks) are zeroed
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
    const u32x4 w = {s.v[0][dt].x & keep[0], s.v[0][dt].y & keep[1], s.v[1][dt].x & keep[2],
                     s.v[1][dt].y & keep[3]};
    const bf16x8 vop = __builtin_bit_cast(bf16x8, w);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
      acc[mt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pop[mt], acc[mt][dt], 0, 0, 0);
  }
}

template <int D, int MT, bool PREFETCH>
__global__ __launch_bounds__(256) void verify_attention_kernel(Params p) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int grp = lane >> 4;
  const int split = blockIdx.x;
  const int g = blockIdx.y * p.waves_per_wg + wave;
  const int r = blockIdx.z;

  int L = p.seq_lens[r];
  L = max(0, min(L, min(p.max_seq_len, p.max_blocks_per_seq * kBlock)));
  const int qo = p.q_indptr[r];
  const int nq = max(0, min(p.q_indptr[r + 1] - qo, p.max_q));
  if (nq == 0) return;
  const int nsplit = L > 0 ? (L + p.split_tokens - 1) / p.split_tokens : 1;
  if (split >= nsplit) return;
  const int t0 = split * p.split_tokens;
  const int t1 = min(L, t0 + p.split_tokens);
  const int rows = p.group * nq;
  const int win = L - nq;   // position of the anchor query

  bf16x8 qop[MT][D / 32];
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
        qop[mt][kk] = __builtin_bit_cast(bf16x8, *(const u32x4*)(src + kk * 32 + grp * 8));
      pos[mt] = win + j;
    } else {
#pragma unroll
      for (int kk = 0; kk < D / 32; ++kk) qop[mt][kk] = bf16x8{};
      pos[mt] = L - 1;
    }
  }

  f32x4 acc[MT][D / 16];
  float m_run[MT], l_run[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    m_run[mt] = -INFINITY;
    l_run[mt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) acc[mt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  const int32_t* bt = p.block_table + (int64_t)r * p.max_blocks_per_seq;
  const int n_span = (t1 - t0 + kSpan - 1) / kSpan;
  if constexpr (PREFETCH) {
    // register double buffering: the next span's loads fly during this span's math
    Span<D> a, b;
    if (n_span > 0) issue_span<D>(a, p, bt, g, t0, L, lane);
    for (int si = 0; si < n_span; si += 2) {
      if (si + 1 < n_span) issue_span<D>(b, p, bt, g, t0 + (si + 1) * kSpan, L, lane);
      compute_span<D, MT>(a, qop, acc, m_run, l_run, pos, L, win, p.scale_log2, lane);
      if (si + 1 >= n_span) break;
      if (si + 2 < n_span) issue_span<D>(a, p, bt, g, t0 + (si + 2) * kSpan, L, lane);
      compute_span<D, MT>(b, qop, acc, m_run, l_run, pos, L, win, p.scale_log2, lane);
    }
  } else {
    // one span buffer; latency is hidden by the other resident waves
    for (int si = 0; si < n_span; ++si) {
      Span<D> a;
      issue_span<D>(a, p, bt, g, t0 + si * kSpan, L, lane);
      compute_span<D, MT>(a, qop, acc, m_run, l_run, pos, L, win, p.scale_log2, lane);
    }
  }

#pragma unroll
  for (int mt = 0; mt < MT; ++mt) l_run[mt] = wave_sum_groups(l_run[mt]);

  if (nsplit == 1) {
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
    const int64_t item = ((int64_t)r * p.num_kv_heads + g) * p.max_splits + split;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = mt * 16 + (lane & 15);
      if (m >= rows) continue;
      float* dst = p.part_o + (item * (MT * 16) + m) * D + grp * 4;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) *(f32x4*)(dst + dt * 16) = acc[mt][dt];
      if (grp == 0) p.part_ml[item * (MT * 16) + m] = make_float2(m_run[mt], l_run[mt]);
    }
  }
}

// Merge split partials of one (request, KV head) in split order.
template <int D, int MT>
__global__ __launch_bounds__(256) void combine_kernel(Params p) {
  const int g = blockIdx.x;
  const int r = blockIdx.y;
  int L = p.seq_lens[r];
  L = max(0, min(L, min(p.max_seq_len, p.max_blocks_per_seq * kBlock)));
  const int qo = p.q_indptr[r];
  const int nq = max(0, min(p.q_indptr[r + 1] - qo, p.max_q));
  const int nsplit = L > 0 ? (L + p.split_tokens - 1) / p.split_tokens : 1;
  if (nq == 0 || nsplit <= 1) return;
  const int rows = p.group * nq;
  const int64_t item0 = ((int64_t)r * p.num_kv_heads + g) * p.max_splits;
  constexpr int kVec = D / 4;
  for (int idx = threadIdx.x; idx < rows * kVec; idx += blockDim.x) {
    const int m = idx / kVec;
    const int d = (idx % kVec) * 4;
    float mx = -INFINITY;
    for (int s = 0; s < nsplit; ++s) mx = fmaxf(mx, p.part_ml[(item0 + s) * (MT * 16) + m].x);
    f32x4 num = {0.f, 0.f, 0.f, 0.f};
    float den = 0.f;
    for (int s = 0; s < nsplit; ++s) {
      const float2 ml = p.part_ml[(item0 + s) * (MT * 16) + m];
      const float w = (ml.x == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(ml.x - mx);
      const f32x4 o = *(const f32x4*)(p.part_o + ((item0 + s) * (MT * 16) + m) * D + d);
      num += w * o;
      den += w * ml.y;
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

struct Plan {
  int mt;            // 16-row tiles
  int split_tokens;
  int max_splits;
  size_t ws_bytes;
};

// Split length: the longest power-of-two multiple of 32 tokens that still
// gives the launch at least kMinItems (request, KV head, split) items, so the
// 256 CUs stay busy with ragged contexts, while long splits keep the partial
// traffic small.
int choose_split_tokens(int bs, int hkv, int max_seq_len) {
  const char* env = getenv("NSD_SPLIT_TOKENS");
  if (env) {
    const int v = atoi(env);
    if (v >= kSpan && v % kSpan == 0) return v;
  }
  constexpr int64_t kMinItems = 8192;
  int s = kSpan;
  while (s < max_seq_len) {
    const int64_t next = 2 * (int64_t)s;
    const int64_t items = (int64_t)bs * hkv * ((max_seq_len + next - 1) / next);
    if (items < kMinItems) break;
    s = (int)next;
  }
  return s;
}

bool make_plan(int bs, int hq, int hkv, int d, int max_q, int max_seq_len, Plan* pl) {
  if (bs < 0 || hq < 1 || hkv < 1 || hq % hkv || (d != 64 && d != 128) || max_q < 1 ||
      max_seq_len < 0)
    return false;
  const int rows = (hq / hkv) * max_q;
  if (rows > kMaxRows) return false;
  pl->mt = (rows + 15) / 16;
  pl->split_tokens = choose_split_tokens(bs, hkv, max_seq_len);
  pl->max_splits = max(1, (max_seq_len + pl->split_tokens - 1) / pl->split_tokens);
  if (pl->max_splits == 1) {
    pl->ws_bytes = 0;
  } else {
    const size_t items = (size_t)bs * hkv * pl->max_splits * pl->mt * 16;
    pl->ws_bytes = items * (size_t)d * sizeof(float) + items * sizeof(float2);
  }
  return true;
}

bool use_prefetch(int d, int mt) {
  const char* env = getenv("NSD_ATTN_PREFETCH");
  if (env) return atoi(env) != 0;
  return d == 64 ? mt <= 2 : mt <= 1;
}

template <int D, int MT>
void launch(const Params& p, int bs, hipStream_t stream) {
  dim3 grid(p.max_splits, p.num_kv_heads / p.waves_per_wg, bs);
  if (MT <= 2 && use_prefetch(D, MT))
    hipLaunchKernelGGL((verify_attention_kernel<D, MT, MT <= 2>), grid, dim3(64 * p.waves_per_wg),
                       0, stream, p);
  else
    hipLaunchKernelGGL((verify_attention_kernel<D, MT, false>), grid, dim3(64 * p.waves_per_wg),
                       0, stream, p);
  if (p.max_splits > 1)
    hipLaunchKernelGGL((combine_kernel<D, MT>), dim3(p.num_kv_heads, bs), dim3(256), 0, stream,
                       p);
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
  if (bs < 0 || bs > 65535) return fail(NSD_ERR_SHAPE, "verify_attention: bs must be in [0, 65535]");
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
  if (pl.ws_bytes > 0 && (!workspace || workspace_bytes < pl.ws_bytes))
    return fail(NSD_ERR_WORKSPACE, "verify_attention: workspace of %zu bytes needed, %zu given",
                pl.ws_bytes, workspace ? workspace_bytes : (size_t)0);

  Params p;
  p.q = (const uint16_t*)q;
  p.k_cache = (const uint16_t*)k_cache;
  p.v_cache = (const uint16_t*)v_cache;
  p.block_table = block_table;
  p.seq_lens = seq_lens;
  p.q_indptr = q_indptr;
  p.out = (uint16_t*)out;
  const size_t items = (size_t)bs * num_kv_heads * pl.max_splits * pl.mt * 16;
  p.part_o = (float*)workspace;
  p.part_ml = pl.ws_bytes ? (float2*)((char*)workspace + items * head_dim * sizeof(float)) : nullptr;
  p.num_blocks = num_blocks;
  p.max_blocks_per_seq = max_blocks_per_seq;
  p.num_q_heads = num_q_heads;
  p.num_kv_heads = num_kv_heads;
  p.group = num_q_heads / num_kv_heads;
  p.max_q = max_q_per_seq;
  p.max_seq_len = max_seq_len;
  p.split_tokens = pl.split_tokens;
  p.max_splits = pl.max_splits;
  p.waves_per_wg = num_kv_heads % 4 == 0 ? 4 : (num_kv_heads % 2 == 0 ? 2 : 1);
  p.scale_log2 = scale * 1.4426950408889634f;

  clear_stale_error();
  if (head_dim == 64)
    launch_d<64>(p, pl.mt, bs, (hipStream_t)stream);
  else
    launch_d<128>(p, pl.mt, bs, (hipStream_t)stream);
  return check_launch("verify_attention");
}
