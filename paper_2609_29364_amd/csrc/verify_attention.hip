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
  float* part_o;     // [2 * num_waves][MT*16][D]: head/tail partial O per wave
  float2* part_ml;   // [2 * num_waves][MT*16]: (running max, sum)
  int64_t* prefix;   // [bs+1]: exclusive prefix of per-request span counts
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
    s.k[0][kk] = __builtin_nontemporal_load((const u32x4*)(k0 + off));
    s.k[1][kk] = __builtin_nontemporal_load((const u32x4*)(k1 + off));
  }
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const int off = (dt * 16 + row) * kBlock + grp * 4;
    s.v[0][dt] = __builtin_nontemporal_load((const u32x2*)(v0 + off));
    s.v[1][dt] = __builtin_nontemporal_load((const u32x2*)(v1 + off));
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

__device__ inline int clamp_len(const Params& p, int r) {
  const int L = p.seq_lens[r];
  return max(0, min(L, min(p.max_seq_len, p.max_blocks_per_seq * kBlock)));
}

// Spans of one (request, KV head) item; an empty context still owns one span
// so that its rows are written (as zeros).
__device__ inline int spans_of(int L) { return max(1, (L + kSpan - 1) / kSpan); }

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

// First span of wave w's range of the T global spans split over W waves.
__device__ inline int64_t range_start(int64_t w, int64_t total, int64_t waves) {
  return w * total / waves;
}

// The wave whose range holds global span s.
__device__ inline int64_t wave_of(int64_t s, int64_t total, int64_t waves) {
  return ((s + 1) * waves - 1) / total;
}

// Stream-K decomposition: the global sequence of spans, ordered by request,
// then KV head, then position, is cut into W equal contiguous ranges, one per
// resident wave.  A wave runs the online softmax over every (request, KV head)
// item its range touches; an item wholly inside the range is finished and
// written directly, an item cut by a range boundary leaves a partial (running
// max, sum, unnormalised O) in the wave's head slot (item began in an earlier
// range) or tail slot (item continues in a later range) for the merge kernel.
template <int D, int MT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(MT <= 2 ? 2 : 1)))
void verify_attention_kernel(Params p) {
  __shared__ int64_t s_wsum[4];
  __shared__ int s_r0[4];
  __shared__ int64_t s_p0[4];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int grp = lane >> 4;
  const int64_t W = p.num_waves;
  const int hkv = p.num_kv_heads;

  // total spans T
  int64_t local = 0;
  for (int r = tid; r < p.bs; r += 256) local += spans_of(clamp_len(p, r));
  local = wave_sum_i64(local);
  if (lane == 0) s_wsum[wave] = local;
  if (tid < 4) s_r0[tid] = -1;
  __syncthreads();
  const int64_t T = (s_wsum[0] + s_wsum[1] + s_wsum[2] + s_wsum[3]) * hkv;
  int64_t ws0[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t w = (int64_t)blockIdx.x * 4 + i;
    ws0[i] = range_start(w, T, W);
    if (tid == 0 && (w >= W || ws0[i] >= range_start(w + 1, T, W))) s_r0[i] = -2;  // empty
  }
  // exclusive prefix of per-request span counts; locate each wave's first request
  int64_t carry = 0;
  for (int base = 0; base < p.bs; base += 256) {
    const int r = base + tid;
    const int64_t n = r < p.bs ? spans_of(clamp_len(p, r)) : 0;
    const int64_t incl = wave_incl_scan_i64(n, lane);
    __syncthreads();
    if (lane == 63) s_wsum[wave] = incl;
    __syncthreads();
    int64_t before = carry;
    for (int i = 0; i < wave; ++i) before += s_wsum[i];
    const int64_t excl = before + incl - n;
    if (r < p.bs) {
      if (blockIdx.x == 0) p.prefix[r] = excl;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (hkv * excl <= ws0[i] && ws0[i] < hkv * (excl + n)) {
          s_r0[i] = r;
          s_p0[i] = excl;
        }
    }
    carry += s_wsum[0] + s_wsum[1] + s_wsum[2] + s_wsum[3];
    __syncthreads();
    const bool found = s_r0[0] != -1 && s_r0[1] != -1 && s_r0[2] != -1 && s_r0[3] != -1;
    if (blockIdx.x != 0 && found) break;
  }
  if (blockIdx.x == 0 && tid == 0) p.prefix[p.bs] = carry;
  __syncthreads();

  const int64_t w = (int64_t)blockIdx.x * 4 + wave;
  int r = s_r0[wave];
  if (r < 0) return;
  int64_t pr = s_p0[wave];
  int64_t s = ws0[wave];
  const int64_t s1 = range_start(w + 1, T, W);

  while (s < s1) {
    const int L = clamp_len(p, r);
    const int n = spans_of(L);
    const int qo = p.q_indptr[r];
    const int nq = max(0, min(p.q_indptr[r + 1] - qo, p.max_q));
    const int64_t off = s - hkv * pr;
    const int g = (int)(off / n);
    const int j0 = (int)(off - (int64_t)g * n);
    const int j1 = (int)min((int64_t)n, j0 + (s1 - s));
    const int rows = p.group * nq;
    const int win = L - nq;

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
    for (int j = j0; j < j1; ++j) {
      Span<D> sp;
      issue_span<D>(sp, p, bt, g, j * kSpan, L, lane);
      compute_span<D, MT>(sp, qop, acc, m_run, l_run, pos, L, win, p.scale_log2, lane);
    }
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
      const int64_t slot = 2 * w + (j0 > 0 ? 0 : 1);
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

// Merge the partials of every item that a range boundary cut, in wave order
// (deterministic, no atomics).
template <int D, int MT>
__global__ __launch_bounds__(256) void combine_kernel(Params p) {
  const int g = blockIdx.x;
  const int r = blockIdx.y;
  const int hkv = p.num_kv_heads;
  const int64_t W = p.num_waves;
  const int64_t T = p.prefix[p.bs] * hkv;
  const int L = clamp_len(p, r);
  const int n = spans_of(L);
  const int qo = p.q_indptr[r];
  const int nq = max(0, min(p.q_indptr[r + 1] - qo, p.max_q));
  const int64_t a = p.prefix[r] * hkv + (int64_t)g * n;
  const int64_t wa = wave_of(a, T, W);
  const int64_t wb = wave_of(a + n - 1, T, W);
  if (wa == wb || nq == 0) return;
  const int rows = p.group * nq;
  constexpr int kVec = D / 4;
  for (int idx = threadIdx.x; idx < rows * kVec; idx += blockDim.x) {
    const int m = idx / kVec;
    const int d = (idx % kVec) * 4;
    float mx = -INFINITY;
    for (int64_t w = wa; w <= wb; ++w) {
      if (w > wa && range_start(w, T, W) == range_start(w + 1, T, W)) continue;
      const int64_t slot = 2 * w + (w == wa ? 1 : 0);
      mx = fmaxf(mx, p.part_ml[slot * (MT * 16) + m].x);
    }
    f32x4 num = {0.f, 0.f, 0.f, 0.f};
    float den = 0.f;
    for (int64_t w = wa; w <= wb; ++w) {
      if (w > wa && range_start(w, T, W) == range_start(w + 1, T, W)) continue;
      const int64_t slot = 2 * w + (w == wa ? 1 : 0);
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
  size_t prefix_bytes, part_o_bytes, part_ml_bytes, ws_bytes;
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
  if (bs < 0 || hq < 1 || hkv < 1 || hq % hkv || (d != 64 && d != 128) || max_q < 1 ||
      max_seq_len < 0)
    return false;
  const int rows = (hq / hkv) * max_q;
  if (rows > kMaxRows) return false;
  pl->mt = (rows + 15) / 16;
  pl->num_waves = resident_waves(d, pl->mt);
  const size_t slots = 2 * (size_t)pl->num_waves * pl->mt * 16;
  pl->prefix_bytes = (((size_t)bs + 1) * sizeof(int64_t) + 255) / 256 * 256;
  pl->part_o_bytes = slots * d * sizeof(float);
  pl->part_ml_bytes = slots * sizeof(float2);
  pl->ws_bytes = pl->prefix_bytes + pl->part_o_bytes + pl->part_ml_bytes;
  return true;
}

template <int D, int MT>
void launch(const Params& p, int bs, hipStream_t stream) {
  hipLaunchKernelGGL((verify_attention_kernel<D, MT>), dim3(p.num_waves / 4), dim3(256), 0,
                     stream, p);
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
  if (!workspace || workspace_bytes < pl.ws_bytes)
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
  p.prefix = (int64_t*)workspace;
  p.part_o = (float*)((char*)workspace + pl.prefix_bytes);
  p.part_ml = (float2*)((char*)workspace + pl.prefix_bytes + pl.part_o_bytes);
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
