// Speculative acceptance with residual resampling, the verification rule of
// the speculative-decoding works the paper builds on (Leviathan et al. 2023;
// Chen et al. 2023; cited in Sections 1 and 2).
//
// One 1024-thread workgroup per request:
// 1. Wave 0 evaluates the K_r acceptance tests u_i * q_i(x_i) <= p_i(x_i)
//    exactly in fp64, one proposal per lane; a ballot gives the first
//    rejection n.
// 2. All 16 waves stream the weight row (max(0, p_n - q_n), or p_K) once in
//    256-element chunks (one float4 per lane), reducing each chunk's fp64 sum
//    with wave shuffles into LDS.  Loads for four chunks are issued before
//    their arithmetic.
// 3. Wave 0 scans the chunk sums (fp64 wave prefix scans with a carry) and
//    finds, by ballot, the first chunk whose inclusive prefix exceeds
//    tau = u_K * S.
// 4. Wave 0 re-reads that one chunk, scans it across lanes and picks the
//    first token t with w(t) > 0 whose running prefix exceeds tau.
// Total traffic: each needed row once plus one 1 KiB chunk.
//
// The same kernel, instantiated with SAMPLE, draws x ~ w from one row per
// workgroup (the draft step's sampling x_i ~ q_i): steps 2-4 with w the row.
#include "nsd_internal.h"

namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kChunk = 256;       // weights per chunk: 64 lanes x float4
constexpr int kUnroll = 4;
constexpr int kMaxVocab = 1 << 19;
constexpr int kMaxK = 63;

__device__ inline double wave_sum(double x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

// Inclusive prefix sum across the wave (Hillis-Steele).
__device__ inline double wave_incl_scan(double x, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  return x;
}

__device__ inline void weights4(const float4& pv, const float4& qv, bool resid, double w[4]) {
  if (resid) {
    w[0] = fmax(0.0, (double)pv.x - (double)qv.x);
    w[1] = fmax(0.0, (double)pv.y - (double)qv.y);
    w[2] = fmax(0.0, (double)pv.z - (double)qv.z);
    w[3] = fmax(0.0, (double)pv.w - (double)qv.w);
  } else {
    w[0] = pv.x;
    w[1] = pv.y;
    w[2] = pv.z;
    w[3] = pv.w;
  }
}

// SAMPLE: plain draw x ~ w from row r (w = the row itself, steps 2-4 only):
// row r at p_target + r * row_stride, uniform uniforms[r], token written to
// out_tokens[r * out_stride]; q_indptr, q_draft, draft_tokens and
// accepted_len are not used.
template <bool SAMPLE>
__global__ __launch_bounds__(kThreads) void spec_accept_kernel(
    const float* __restrict__ p_target, const float* __restrict__ q_draft,
    const int32_t* __restrict__ draft_tokens, const float* __restrict__ uniforms,
    const int32_t* __restrict__ q_indptr, int32_t vocab, int32_t max_k,
    int32_t* __restrict__ accepted_len, int32_t* __restrict__ out_tokens, int64_t row_stride,
    int32_t out_stride) {
  extern __shared__ double lds[];   // [nchunk] chunk sums, then [nchunk] exclusive prefixes
  __shared__ int s_n;
  __shared__ double s_total;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r = blockIdx.x;
  const int a = SAMPLE ? r : q_indptr[r];
  const int k = SAMPLE ? 0 : max(0, min(q_indptr[r + 1] - a - 1, max_k));
  const int nchunk = (vocab + kChunk - 1) / kChunk;
  double* csum = lds;
  double* cpre = lds + nchunk;

  if (SAMPLE) {
    if (threadIdx.x == 0) s_n = 0;
  } else if (wave == 0) {
    bool ok = true;
    if (lane < k) {
      const int x = draft_tokens[a - r + lane];
      if (x < 0 || x >= vocab) {
        ok = false;
      } else {
        const double uq = (double)uniforms[a + lane] *
                          (double)q_draft[(int64_t)(a - r + lane) * vocab + x];
        ok = uq <= (double)p_target[(int64_t)(a + lane) * vocab + x];
      }
    }
    const uint64_t rejected = __ballot(!ok);
    if (lane == 0) s_n = rejected ? (__ffsll((unsigned long long)rejected) - 1) : k;
  }
  __syncthreads();
  const int n = s_n;
  bool resid = n < k;
  const float* prow = SAMPLE ? p_target + (int64_t)r * row_stride
                            : p_target + (int64_t)(a + n) * vocab;
  const float* qrow = resid ? q_draft + (int64_t)(a - r + n) * vocab : prow;

  for (int attempt = 0; attempt < 2; ++attempt) {
    // 2. chunk sums
    for (int c0 = wave; c0 < nchunk; c0 += kWaves * kUnroll) {
      float4 pv[kUnroll], qv[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int c = c0 + u * kWaves;
        const int idx = c * kChunk + lane * 4;
        pv[u] = make_float4(0.f, 0.f, 0.f, 0.f);
        qv[u] = pv[u];
        if (c < nchunk && idx < vocab) {
          pv[u] = *(const float4*)(prow + idx);
          if (resid) qv[u] = *(const float4*)(qrow + idx);
        }
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int c = c0 + u * kWaves;
        double w[4];
        weights4(pv[u], qv[u], resid, w);
        const double s = wave_sum(((w[0] + w[1]) + w[2]) + w[3]);
        if (lane == 0 && c < nchunk) csum[c] = s;
      }
    }
    __syncthreads();
    // 3a. exclusive prefix of the chunk sums
    if (wave == 0) {
      double carry = 0.0;
      for (int base = 0; base < nchunk; base += 64) {
        const int c = base + lane;
        const double v = c < nchunk ? csum[c] : 0.0;
        const double incl = wave_incl_scan(v, lane);
        double excl = __shfl_up(incl, 1);
        if (lane == 0) excl = 0.0;
        if (c < nchunk) cpre[c] = carry + excl;
        carry += __shfl(incl, 63);
      }
      if (lane == 0) s_total = cpre[nchunk - 1] + csum[nchunk - 1];
    }
    __syncthreads();
    if (s_total > 0.0 || !resid) break;
    resid = false;   // residual without mass: draw from p_n itself
    qrow = prow;
    __syncthreads();
  }

  if (wave != 0) return;
  const double total = s_total;
  const double tau = (double)uniforms[a + k] * total;
  int y = -1;
  if (total > 0.0) {
    // 3b. first chunk whose inclusive prefix exceeds tau
    int cstar = -1;
    for (int base = 0; base < nchunk && cstar < 0; base += 64) {
      const int c = base + lane;
      const bool hit = c < nchunk && cpre[c] + csum[c] > tau;
      const uint64_t m = __ballot(hit);
      if (m) cstar = base + __ffsll((unsigned long long)m) - 1;
    }
    if (cstar < 0) {   // rounding: take the last chunk with mass
      for (int base = ((nchunk - 1) / 64) * 64; base >= 0 && cstar < 0; base -= 64) {
        const int c = base + lane;
        const uint64_t m = __ballot(c < nchunk && csum[c] > 0.0);
        if (m) cstar = base + 63 - __clzll((long long)m);
      }
    }
    // 4. scan inside the chosen chunk
    if (cstar < 0) cstar = 0;   // unreachable when total > 0; keeps addresses in range
    const int idx = cstar * kChunk + lane * 4;
    float4 pv = make_float4(0.f, 0.f, 0.f, 0.f), qv = pv;
    if (idx < vocab) {
      pv = *(const float4*)(prow + idx);
      if (resid) qv = *(const float4*)(qrow + idx);
    }
    double w[4];
    weights4(pv, qv, resid, w);
    const double ls = ((w[0] + w[1]) + w[2]) + w[3];
    const double incl = wave_incl_scan(ls, lane);
    double run = __shfl_up(incl, 1);
    if (lane == 0) run = 0.0;
    run += cpre[cstar];
    int found = -1, last_pos = -1;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      run += w[e];
      if (w[e] > 0.0) {
        last_pos = e;
        if (found < 0 && run > tau) found = e;
      }
    }
    const uint64_t fm = __ballot(found >= 0);
    if (fm) {
      const int fl = __ffsll((unsigned long long)fm) - 1;
      y = cstar * kChunk + fl * 4 + __shfl(found, fl);
    } else {
      const uint64_t pm = __ballot(last_pos >= 0);
      if (pm) {
        const int pl = 63 - __clzll((long long)pm);
        y = cstar * kChunk + pl * 4 + __shfl(last_pos, pl);
      }
    }
  }
  if (SAMPLE) {
    if (lane == 0) out_tokens[(int64_t)r * out_stride] = y;
    return;
  }
  if (lane <= k) {
    int tok = -1;
    if (lane < n) tok = draft_tokens[a - r + lane];
    else if (lane == n) tok = y;
    out_tokens[a + lane] = tok;
  }
  if (lane == 0) accepted_len[r] = n;
}

}  // namespace

extern "C" nsd_status nsd_spec_accept(const float* p_target, const float* q_draft,
                                      const int32_t* draft_tokens, const float* uniforms,
                                      const int32_t* q_indptr, int32_t bs, int32_t vocab,
                                      int32_t max_k, int32_t* accepted_len,
                                      int32_t* out_tokens, void* stream) {
  using namespace nsd;
  if (bs < 0) return fail(NSD_ERR_SHAPE, "spec_accept: bs < 0");
  if (vocab < 4 || vocab > kMaxVocab || vocab % 4)
    return fail(NSD_ERR_UNSUPPORTED, "spec_accept: vocab must be a multiple of 4 in [4, %d] "
                "(got %d)", kMaxVocab, vocab);
  if (max_k < 0 || max_k > kMaxK)
    return fail(NSD_ERR_UNSUPPORTED, "spec_accept: max_k must be in [0, %d] (got %d)", kMaxK, max_k);
  if (bs == 0) return NSD_OK;
  if (!p_target || !uniforms || !q_indptr || !accepted_len || !out_tokens ||
      (max_k > 0 && (!q_draft || !draft_tokens)))
    return fail(NSD_ERR_NULL, "spec_accept: NULL pointer argument");
  if (((uintptr_t)p_target | (uintptr_t)(max_k > 0 ? q_draft : p_target)) & 15)
    return fail(NSD_ERR_SHAPE, "spec_accept: probability rows must be 16-byte aligned");
  const int nchunk = (vocab + kChunk - 1) / kChunk;
  const size_t lds = 2 * (size_t)nchunk * sizeof(double);
  clear_stale_error();
  hipLaunchKernelGGL(spec_accept_kernel<false>, dim3(bs), dim3(kThreads), lds,
                     (hipStream_t)stream, p_target, q_draft, draft_tokens, uniforms, q_indptr,
                     vocab, max_k, accepted_len, out_tokens, (int64_t)vocab, 1);
  return check_launch("spec_accept");
}

extern "C" nsd_status nsd_sample(const float* probs, int64_t row_stride, const float* uniforms,
                                 int32_t n_rows, int32_t vocab, int32_t* out_tokens,
                                 int32_t out_stride, void* stream) {
  using namespace nsd;
  if (n_rows < 0) return fail(NSD_ERR_SHAPE, "sample: n_rows < 0");
  if (vocab < 4 || vocab > kMaxVocab || vocab % 4)
    return fail(NSD_ERR_UNSUPPORTED, "sample: vocab must be a multiple of 4 in [4, %d] (got %d)",
                kMaxVocab, vocab);
  if (row_stride < vocab || row_stride % 4)
    return fail(NSD_ERR_SHAPE, "sample: row_stride must be a multiple of 4 and >= vocab "
                "(got %lld)", (long long)row_stride);
  if (out_stride < 1) return fail(NSD_ERR_SHAPE, "sample: out_stride < 1");
  if (n_rows == 0) return NSD_OK;
  if (!probs || !uniforms || !out_tokens) return fail(NSD_ERR_NULL, "sample: NULL pointer argument");
  if ((uintptr_t)probs & 15) return fail(NSD_ERR_SHAPE, "sample: probs must be 16-byte aligned");
  const int nchunk = (vocab + kChunk - 1) / kChunk;
  const size_t lds = 2 * (size_t)nchunk * sizeof(double);
  clear_stale_error();
  hipLaunchKernelGGL(spec_accept_kernel<true>, dim3(n_rows), dim3(kThreads), lds,
                     (hipStream_t)stream, probs, nullptr, nullptr, uniforms, nullptr, vocab, 0,
                     nullptr, out_tokens, row_stride, out_stride);
  return check_launch("sample");
}
