// Speculative acceptance with residual resampling, the verification rule of
// the speculative-decoding works the paper builds on (Leviathan et al. 2023;
// Chen et al. 2023; cited in Sections 1 and 2); and plain inverse-CDF
// sampling of one row (the draft step's x_i ~ q_i).
//
// A request's weight row (max(0, p_n - q_n) after a rejection at n, or the
// bonus row p_K) is 151936 floats in the workloads: streaming it is the whole
// cost.  A batch with a row for every CU (exactly one, or at least 1.375)
// runs accept_row_kernel: one 256-thread workgroup per row takes the
// acceptance tests, streams the row into chunk sums held in LDS, and draws
// with one wave, in one launch.  Other batches spread each row over several
// workgroups, in two kernels:
//
// 1. row_sums_kernel, one 256-thread workgroup per (row, segment of 32
//    chunks).  Every workgroup first evaluates the request's K acceptance
//    tests u_i * q_i(x_i) <= p_i(x_i) exactly in fp64 (one proposal per lane;
//    a ballot gives the first rejection n; redundant across a request's
//    segments, a few scattered loads), then streams its segment of the
//    weight row in 256-element chunks (one 16-byte load per lane, four chunks
//    of loads in flight per wave, reduced together in one butterfly) and
//    writes each chunk's fp64 sum to the workspace.  The row is spread over
//    the whole chip instead of one workgroup per request.
// 2. pick_kernel, one 256-thread workgroup per row: loads the row's chunk
//    sums into LDS; one wave scans them (a lane owns consecutive chunks; a
//    wave scan of the lane totals), finds the first chunk whose inclusive
//    prefix exceeds tau = u_K * S, re-reads that one chunk and picks the
//    first token t with w(t) > 0 whose running prefix exceeds tau.  A
//    residual without mass (only possible through fp32 rounding) falls back
//    to p_n, streamed here.
// Traffic: each needed row once, plus the chunk sums (8 bytes per 1 KiB) and
// one 1 KiB chunk per row.
#include "nsd_internal.h"

#include <atomic>
#include <mutex>

namespace {

typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kChunk = 256;       // weights per chunk: 64 lanes x 4
constexpr int kUnroll = 4;
constexpr int kRowThreads = 256;   // accept_row_kernel: 4 waves per row
constexpr int kSegChunks = kWaves * kUnroll * 2;   // chunks per row_sums workgroup
constexpr int kOnePassChunks = 64;   // rows this short always take one workgroup each
constexpr int kMaxVocab = 1 << 19;
constexpr int kMaxChunks = kMaxVocab / kChunk;
constexpr int kMaxK = 63;
constexpr int kMaxSegs = kMaxChunks / kSegChunks;
constexpr int kMaxRows = 0x7fffffff / kMaxSegs;   // row_sums_kernel grid: segments x rows

struct Args {
  const float* p;              // target rows, or the rows to sample (SAMPLE)
  const float* q;              // draft rows
  const int32_t* x;            // proposal tokens
  const float* u;              // uniforms
  const int32_t* q_indptr;     // [rows + 1] (not SAMPLE)
  int32_t rows;                // requests (not SAMPLE) or sample rows
  int32_t vocab, max_k, nchunk;
  int64_t row_stride;          // SAMPLE: elements between rows
  int32_t out_stride;          // SAMPLE: entries between output tokens
  double* ws_sum;              // [rows][nchunk]
  int32_t* ws_n;               // [rows]
  int32_t* accepted_len;
  int32_t* out_tokens;
};

// Lane l's view of x in lane src(l) under a DPP control (row_mask and
// bank_mask select the lanes that take it; the others, and lanes whose source
// is outside the row or wave, get 0).  fp64 moves as two 32-bit DPP moves.
template <int CTRL, int ROW_MASK, int BANK_MASK>
__device__ __attribute__((always_inline)) inline double dpp_f64(double x) {
  const uint64_t b = (uint64_t)__double_as_longlong(x);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, CTRL, ROW_MASK, BANK_MASK, true);
  const int hi =
      __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), CTRL, ROW_MASK, BANK_MASK, true);
  return __longlong_as_double((long long)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
}

// Inclusive prefix sum across the wave with DPP lane moves: within each row
// of 16 lanes the sums of 4 (shifts by 1, 2 and 3), then 8 and 16 (shifts by
// 4 and 8 into the upper banks), then the row totals carried across rows
// (broadcasts of lanes 15 and 31).
__device__ __attribute__((always_inline)) inline double wave_incl_scan(double v) {
  double s = v + dpp_f64<0x111, 0xf, 0xf>(v);   // row_shr:1
  s += dpp_f64<0x112, 0xf, 0xf>(v);             // row_shr:2
  s += dpp_f64<0x113, 0xf, 0xf>(v);             // row_shr:3
  s += dpp_f64<0x114, 0xf, 0xe>(s);             // row_shr:4, banks 1-3
  s += dpp_f64<0x118, 0xf, 0xc>(s);             // row_shr:8, banks 2-3
  s += dpp_f64<0x142, 0xa, 0xf>(s);             // row_bcast:15, rows 1 and 3
  s += dpp_f64<0x143, 0xc, 0xf>(s);             // row_bcast:31, rows 2 and 3
  return s;
}

// Lane l's value in every lane; l must be the same in all lanes.
__device__ __attribute__((always_inline)) inline int lane_value(int v, int l) {
  return __builtin_amdgcn_readlane(v, l);
}
__device__ __attribute__((always_inline)) inline double lane_value(double v, int l) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)b, l);
  const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), l);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// The previous lane's value (0 in lane 0): DPP wave_shr:1.
__device__ __attribute__((always_inline)) inline double wave_prev(double v) {
  return dpp_f64<0x138, 0xf, 0xf>(v);
}

__device__ inline void weights4(const f32x4& pv, const f32x4& qv, bool resid, double w[4]) {
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

// Request r's first target row a and proposal count k, read from q_indptr
// and clamped so that every row the request touches lies in the buffers the
// row count total_q = q_indptr[rows] describes: target rows a .. a + k <
// total_q, draft rows a - r .. a - r + k - 1 inside [0, total_q - rows).  For
// a well-formed q_indptr (non-decreasing, every request at least one row)
// nothing changes.  Returns false when the request has no target row (its
// start clamps to total_q); it then draws nothing and writes no token.
__device__ inline bool request_rows(const Args& A, int r, int& a, int& k) {
  const int total = max(0, A.q_indptr[A.rows]);
  a = min(max(A.q_indptr[r], 0), total);
  k = max(0, min(min(A.q_indptr[r + 1] - a - 1, A.max_k), total - a - 1));
  const int db = a - r;   // first draft row
  if (db < 0) k = 0;
  k = min(k, max(0, total - A.rows - db));
  return a < total;
}

// Request r's first row a and clamped proposal count k; wave 0 evaluates the
// acceptance tests and leaves the first rejection n in *s_n.  Returns false
// when the request has no row (nothing to test or draw).
template <bool SAMPLE>
__device__ inline bool acceptance(const Args& A, int r, int lane, int wave, int& a, int& k,
                                  int* s_n, int& x_lane) {
  x_lane = -1;
  if (SAMPLE) {
    a = r;
    k = 0;
    return true;
  }
  if (!request_rows(A, r, a, k)) return false;
  if (wave == 0) {
    bool ok = true;
    if (lane < k) {
      const int x = A.x[a - r + lane];
      x_lane = x;
      if (x < 0 || x >= A.vocab) {
        ok = false;
      } else {
        const double uq =
            (double)A.u[a + lane] * (double)A.q[(int64_t)(a - r + lane) * A.vocab + x];
        ok = uq <= (double)A.p[(int64_t)(a + lane) * A.vocab + x];
      }
    }
    const uint64_t rejected = __ballot(!ok);
    if (lane == 0) *s_n = rejected ? (__ffsll((unsigned long long)rejected) - 1) : k;
  }
  return true;
}

template <bool SAMPLE>
__device__ inline const float* row_p(const Args& A, int r, int a, int n) {
  return SAMPLE ? A.p + (int64_t)r * A.row_stride : A.p + (int64_t)(a + n) * A.vocab;
}

// One iteration's loads: chunks c0 + u * NW (u < kUnroll) of the weight
// row, one 16-byte load per lane and chunk (and the draft row's with RESID).
// Without CHECK every chunk must be whole and inside [., c_end); with it,
// chunks past c_end load chunk c_end - 1 again and lanes past the vocabulary
// its last four weights, so every load is unconditional and in bounds (the
// reduction drops both).
template <bool RESID, bool CHECK, int NW>
__device__ __attribute__((always_inline)) inline void load_chunks(const float* prow, const float* qrow, int vocab, int c0,
                                   int c_end, int lane, f32x4 (&pv)[kUnroll],
                                   f32x4 (&qv)[kUnroll]) {
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int c = CHECK ? min(c0 + u * NW, c_end - 1) : c0 + u * NW;
    const int idx = CHECK ? min(c * kChunk + lane * 4, vocab - 4) : c * kChunk + lane * 4;
    pv[u] = __builtin_nontemporal_load((const f32x4*)(prow + idx));
    qv[u] = RESID ? __builtin_nontemporal_load((const f32x4*)(qrow + idx)) : pv[u];
  }
  // keep the reduction of the previous iteration after these loads: they go
  // out first, so the wave always has an iteration's loads in flight
  __builtin_amdgcn_sched_barrier(0);
}

// The four chunk sums of one iteration in one butterfly, into dst: halves of
// the lanes swap two chunks' values (xor 32), then one (xor 16), then 16-lane
// sums; lanes 0, 16, 32, 48 end with chunks 0, 1, 2, 3.  Chunks past c_end
// are not stored; with CHECK, lanes past the vocabulary count zero.
template <bool RESID, bool CHECK, int NW>
__device__ __attribute__((always_inline)) inline void reduce_chunks(const f32x4 (&pv)[kUnroll], const f32x4 (&qv)[kUnroll],
                                     int c0, int c_end, int vocab, int lane, double* dst) {
  double v[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    double w[4];
    weights4(pv[u], qv[u], RESID, w);
    v[u] = ((w[0] + w[1]) + w[2]) + w[3];
    if (CHECK && (c0 + u * NW) * kChunk + lane * 4 >= vocab) v[u] = 0.0;
  }
  const bool h5 = lane & 32, h4 = lane & 16;
  const double r0 = (h5 ? v[2] : v[0]) + __shfl_xor(h5 ? v[0] : v[2], 32);
  const double r1 = (h5 ? v[3] : v[1]) + __shfl_xor(h5 ? v[1] : v[3], 32);
  double s = (h4 ? r1 : r0) + __shfl_xor(h4 ? r0 : r1, 16);
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) s += __shfl_xor(s, o);
  if ((lane & 15) == 0) {
    const int c = c0 + ((h5 ? 2 : 0) + (h4 ? 1 : 0)) * NW;
    if (c < c_end) dst[c] = s;
  }
}
static_assert(kUnroll == 4, "the butterfly in reduce_chunks reduces four chunks");

// Sums of chunks [c_beg, c_end) of the weight row into dst[c], by the NW
// waves of a workgroup: wave w takes iterations of kUnroll chunks w, w + NW,
// ...  The loads are double-buffered, so a wave always has the next
// iteration's loads in flight while it reduces the current one.  Every
// iteration but a wave's last covers whole chunks inside the range (only the
// range's last chunk can be partial, and it falls in the last iteration of
// the wave holding it), so the loop's loads need no checks; the last
// iteration's addresses are clamped into the range.
template <int NW, bool RESID>
__device__ __attribute__((always_inline)) inline void chunk_sums_t(const float* prow, const float* qrow, int vocab, int c_beg,
                                    int c_end, int lane, int wave, double* dst) {
  constexpr int kStep = NW * kUnroll;
  const int first = c_beg + wave;
  if (first >= c_end) return;
  const int n_iter = (c_end - first + kStep - 1) / kStep;
  f32x4 pa[kUnroll], qa[kUnroll], pb[kUnroll], qb[kUnroll];
  if (n_iter == 1) {
    load_chunks<RESID, true, NW>(prow, qrow, vocab, first, c_end, lane, pa, qa);
    reduce_chunks<RESID, true, NW>(pa, qa, first, c_end, vocab, lane, dst);
    return;
  }
  // two register sets used in turn (unrolled by two, so no set is copied: a
  // copy would wait for the loads still landing in it)
  load_chunks<RESID, false, NW>(prow, qrow, vocab, first, c_end, lane, pa, qa);
  int c0 = first, it = 0;
  for (; it + 3 < n_iter; it += 2, c0 += 2 * kStep) {
    load_chunks<RESID, false, NW>(prow, qrow, vocab, c0 + kStep, c_end, lane, pb, qb);
    reduce_chunks<RESID, false, NW>(pa, qa, c0, c_end, vocab, lane, dst);
    load_chunks<RESID, false, NW>(prow, qrow, vocab, c0 + 2 * kStep, c_end, lane, pa, qa);
    reduce_chunks<RESID, false, NW>(pb, qb, c0 + kStep, c_end, vocab, lane, dst);
  }
  // two or three iterations left, the first of them loaded
  if (n_iter - it == 3) {
    load_chunks<RESID, false, NW>(prow, qrow, vocab, c0 + kStep, c_end, lane, pb, qb);
    reduce_chunks<RESID, false, NW>(pa, qa, c0, c_end, vocab, lane, dst);
    load_chunks<RESID, true, NW>(prow, qrow, vocab, c0 + 2 * kStep, c_end, lane, pa, qa);
    reduce_chunks<RESID, false, NW>(pb, qb, c0 + kStep, c_end, vocab, lane, dst);
    reduce_chunks<RESID, true, NW>(pa, qa, c0 + 2 * kStep, c_end, vocab, lane, dst);
  } else {
    load_chunks<RESID, true, NW>(prow, qrow, vocab, c0 + kStep, c_end, lane, pb, qb);
    reduce_chunks<RESID, false, NW>(pa, qa, c0, c_end, vocab, lane, dst);
    reduce_chunks<RESID, true, NW>(pb, qb, c0 + kStep, c_end, vocab, lane, dst);
  }
}

template <int NW>
__device__ __attribute__((always_inline)) inline void chunk_sums(const float* prow, const float* qrow, bool resid, int vocab,
                                  int c_beg, int c_end, int lane, int wave, double* dst) {
  if (resid)
    chunk_sums_t<NW, true>(prow, qrow, vocab, c_beg, c_end, lane, wave, dst);
  else
    chunk_sums_t<NW, false>(prow, qrow, vocab, c_beg, c_end, lane, wave, dst);
}

template <bool SAMPLE>
__global__ __launch_bounds__(kThreads) void row_sums_kernel(Args A) {
  __shared__ int s_n;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nseg = (A.nchunk + kSegChunks - 1) / kSegChunks;
  const int r = blockIdx.x / nseg;
  const int seg = blockIdx.x - r * nseg;
  int a, k, x_lane;
  if (!acceptance<SAMPLE>(A, r, lane, wave, a, k, &s_n, x_lane)) {
    if (seg == 0 && threadIdx.x == 0) A.ws_n[r] = 0;
    return;   // uniform over the workgroup: no row to stream
  }
  int n = 0;
  if (!SAMPLE) {
    __syncthreads();
    n = s_n;
  }
  const bool resid = n < k;
  const float* prow = row_p<SAMPLE>(A, r, a, n);
  const float* qrow = resid ? A.q + (int64_t)(a - r + n) * A.vocab : prow;
  const int c_beg = seg * kSegChunks;
  const int c_end = min(A.nchunk, c_beg + kSegChunks);
  chunk_sums<kWaves>(prow, qrow, resid, A.vocab, c_beg, c_end, lane, wave,
                     A.ws_sum + (int64_t)r * A.nchunk);
  if (!SAMPLE && seg == 0 && threadIdx.x == 0) A.ws_n[r] = n;
}

// The draw of request r (or sample row r) from its chunk sums s_sum[0,
// nchunk), by one wave with no workgroup barrier: lane l owns consecutive
// chunks and sums them, a wave scan gives every lane its prefix, the first
// lane whose inclusive prefix exceeds tau = u_K * S finds its first chunk
// whose inclusive prefix does (else the last chunk with mass is taken), and
// the wave scans inside that chunk.  u_draw is u_K and x_lane this lane's
// proposal token (lanes < K), both loaded early so their latency is hidden.
// Writes the request's tokens and accepted length.
template <bool SAMPLE>
__device__ inline void draw_wave(const Args& A, int r, int a, int k, int n, double* s_sum,
                                 float u_draw, int x_lane, int lane) {
  const int nchunk = A.nchunk;
  bool resid = n < k;
  const float* prow = row_p<SAMPLE>(A, r, a, n);
  const float* qrow = resid ? A.q + (int64_t)(a - r + n) * A.vocab : prow;
  const int per = (nchunk + 63) / 64;
  const int c0 = min(nchunk, lane * per), c1 = min(nchunk, c0 + per);
  double local = 0.0, incl = 0.0, total = 0.0;
  for (int attempt = 0; attempt < 2; ++attempt) {
    local = 0.0;
    for (int c = c0; c < c1; ++c) local += s_sum[c];
    incl = wave_incl_scan(local);
    total = lane_value(incl, 63);
    if (total > 0.0 || !resid) break;
    // residual without mass: draw from p_n itself (its sums, by this wave)
    resid = false;
    qrow = prow;
    chunk_sums<1>(prow, qrow, false, A.vocab, 0, nchunk, lane, 0, s_sum);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the wave's sums are in LDS
  }
  const double excl = wave_prev(incl);
  const double tau = (double)u_draw * total;
  int cstar = -1;
  double cpre = 0.0;
  if (total > 0.0) {
    // each lane's first chunk whose inclusive prefix exceeds tau, and its last
    // chunk with mass; the first lane with such a chunk gives it, else
    // (rounding left tau at or past the total) the last lane with mass does
    int found = -1, last = -1;
    double fpre = 0.0, lpre = 0.0, run = excl;
    for (int c = c0; c < c1; ++c) {
      const double v = s_sum[c];
      if (found < 0 && run + v > tau) {
        found = c;
        fpre = run;
      }
      if (v > 0.0) {
        last = c;
        lpre = run;
      }
      run += v;
    }
    const uint64_t over = __ballot(found >= 0);
    if (over) {
      const int owner = __ffsll((unsigned long long)over) - 1;
      cstar = lane_value(found, owner);
      cpre = lane_value(fpre, owner);
    } else {
      const uint64_t has = __ballot(last >= 0);
      if (has) {
        const int owner = 63 - __clzll((long long)has);
        cstar = lane_value(last, owner);
        cpre = lane_value(lpre, owner);
      }
    }
  }
  int y = -1;
  if (cstar >= 0) {
    // scan inside the chosen chunk
    const int idx = cstar * kChunk + lane * 4;
    f32x4 pv = (f32x4){0.f, 0.f, 0.f, 0.f}, qv = pv;
    if (idx < A.vocab) {
      pv = *(const f32x4*)(prow + idx);
      if (resid) qv = *(const f32x4*)(qrow + idx);
    }
    double w[4];
    weights4(pv, qv, resid, w);
    const double ls = ((w[0] + w[1]) + w[2]) + w[3];
    double rr = wave_prev(wave_incl_scan(ls)) + cpre;
    int f = -1, last_pos = -1;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      rr += w[e];
      if (w[e] > 0.0) {
        last_pos = e;
        if (f < 0 && rr > tau) f = e;
      }
    }
    const uint64_t fm = __ballot(f >= 0);
    if (fm) {
      const int fl = __ffsll((unsigned long long)fm) - 1;
      y = cstar * kChunk + fl * 4 + lane_value(f, fl);
    } else {
      const uint64_t pm = __ballot(last_pos >= 0);
      if (pm) {
        const int pl = 63 - __clzll((long long)pm);
        y = cstar * kChunk + pl * 4 + lane_value(last_pos, pl);
      }
    }
  }
  if (SAMPLE) {
    if (lane == 0) A.out_tokens[(int64_t)r * A.out_stride] = y;
    return;
  }
  if (lane <= k) {
    int tok = -1;
    if (lane < n) tok = x_lane;
    else if (lane == n) tok = y;
    A.out_tokens[a + lane] = tok;
  }
  if (lane == 0) A.accepted_len[r] = n;
}

template <bool SAMPLE>
__global__ __launch_bounds__(kThreads) void pick_kernel(Args A) {
  __shared__ double s_sum[kMaxChunks];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int r = blockIdx.x;
  int a = r, k = 0, n = 0, x_lane = -1;
  if (!SAMPLE) {
    if (!request_rows(A, r, a, k)) {
      if (tid == 0) A.accepted_len[r] = 0;
      return;
    }
    n = min(max(A.ws_n[r], 0), k);
    if (tid < k) x_lane = A.x[a - r + tid];
  }
  const float u_draw = A.u[a + k];
  const double* sums = A.ws_sum + (int64_t)r * A.nchunk;
  for (int c = tid; c < A.nchunk; c += kThreads) s_sum[c] = sums[c];
  __syncthreads();
  if (tid >= 64) return;
  draw_wave<SAMPLE>(A, r, a, k, n, s_sum, u_draw, x_lane, lane);
}

// Both steps for one row per workgroup of kRowThreads threads (used when the
// batch has at least a row per CU): the acceptance tests, the row's chunk
// sums into LDS, then the draw, with no second launch and no round trip of
// the sums through memory.
template <bool SAMPLE>
__global__ __launch_bounds__(kRowThreads) void accept_row_kernel(Args A) {
  __shared__ double s_sum[kMaxChunks];
  __shared__ int s_n;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r = blockIdx.x;
  int a, k, x_lane;
  if (!acceptance<SAMPLE>(A, r, lane, wave, a, k, &s_n, x_lane)) {
    if (threadIdx.x == 0) A.accepted_len[r] = 0;
    return;
  }
  int n = 0;
  if (!SAMPLE) {
    __syncthreads();
    n = s_n;
  }
  const bool resid = n < k;
  const float* prow = row_p<SAMPLE>(A, r, a, n);
  const float* qrow = resid ? A.q + (int64_t)(a - r + n) * A.vocab : prow;
  const float u_draw = wave == 0 ? A.u[a + k] : 0.f;   // in flight while the row streams
  chunk_sums<kRowThreads / 64>(prow, qrow, resid, A.vocab, 0, A.nchunk, lane, wave, s_sum);
  __syncthreads();
  if (wave != 0) return;
  draw_wave<SAMPLE>(A, r, a, k, n, s_sum, u_draw, x_lane, lane);
}

// CUs of the current device, queried once per device and kept (256 when the
// device cannot be queried, which only picks the kernel layout).
int device_cus() {
  constexpr int kMaxDev = 64;
  static std::atomic<int> cached[kMaxDev];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDev) {
    (void)hipGetLastError();
    return 256;
  }
  int cus = cached[dev].load(std::memory_order_relaxed);
  if (cus > 0) return cus;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0) {
    (void)hipGetLastError();
    return 256;
  }
  cached[dev].store(cus, std::memory_order_relaxed);
  return cus;
}

int64_t sums_bytes(int64_t rows, int32_t vocab) {
  const int64_t nchunk = (vocab + kChunk - 1) / kChunk;
  return (rows * nchunk * 8 + 255) / 256 * 256;
}

nsd_status launch(bool sample, Args A, int32_t rows, void* workspace, size_t workspace_bytes,
                  void* stream, const char* fn) {
  using namespace nsd;
  const size_t need = (size_t)(sums_bytes(rows, A.vocab) + (int64_t)rows * 4);
  if (!workspace || workspace_bytes < need)
    return fail(NSD_ERR_WORKSPACE, "%s: a workspace of %zu bytes is needed (got %zu)", fn, need,
                workspace ? workspace_bytes : (size_t)0);
  if ((uintptr_t)workspace & 7)
    return fail(NSD_ERR_SHAPE, "%s: the workspace must be 8-byte aligned", fn);
  A.nchunk = (A.vocab + kChunk - 1) / kChunk;
  A.ws_sum = (double*)workspace;
  A.ws_n = (int32_t*)((char*)workspace + sums_bytes(rows, A.vocab));
  const dim3 g1((uint32_t)((A.nchunk + kSegChunks - 1) / kSegChunks) * (uint32_t)rows);
  // one workgroup per row does both steps (a second launch would add
  // nothing) for rows of at most 64 chunks, or when the batch has a row for
  // every CU: exactly one, or at least 1.375 (just over one, the few CUs
  // holding a second row would set the end; below 1.375 rows per CU the
  // rows spread over all CUs measured faster); otherwise every row is spread
  // over several workgroups
  const int cus = device_cus();
  const bool one_pass =
      A.nchunk <= kOnePassChunks || rows == cus || (int64_t)rows * 8 >= (int64_t)cus * 11;
  clear_stale_error();
  if (one_pass) {
    if (sample)
      hipLaunchKernelGGL(accept_row_kernel<true>, dim3(rows), dim3(kRowThreads), 0,
                         (hipStream_t)stream, A);
    else
      hipLaunchKernelGGL(accept_row_kernel<false>, dim3(rows), dim3(kRowThreads), 0,
                         (hipStream_t)stream, A);
  } else if (sample) {
    hipLaunchKernelGGL(row_sums_kernel<true>, g1, dim3(kThreads), 0, (hipStream_t)stream, A);
    hipLaunchKernelGGL(pick_kernel<true>, dim3(rows), dim3(kThreads), 0, (hipStream_t)stream, A);
  } else {
    hipLaunchKernelGGL(row_sums_kernel<false>, g1, dim3(kThreads), 0, (hipStream_t)stream, A);
    hipLaunchKernelGGL(pick_kernel<false>, dim3(rows), dim3(kThreads), 0, (hipStream_t)stream, A);
  }
  return check_launch(fn);
}

}  // namespace

extern "C" size_t nsd_spec_accept_workspace_size(int32_t rows, int32_t vocab) {
  if (rows < 0 || vocab < 1 || vocab > kMaxVocab) return 0;
  return (size_t)(sums_bytes(rows, vocab) + (int64_t)rows * 4);
}

// Validation and launch shared by nsd_spec_accept and nsd_spec_accept_static.
static nsd_status spec_accept_impl(const char* fn, const float* p_target, const float* q_draft,
                            const int32_t* draft_tokens, const float* uniforms,
                            const int32_t* q_indptr, int32_t bs, int32_t vocab, int32_t max_k,
                            int32_t* accepted_len, int32_t* out_tokens, void* workspace,
                            size_t workspace_bytes, void* stream) {
  using namespace nsd;
  if (bs < 0 || bs > kMaxRows)
    return fail(NSD_ERR_SHAPE, "%s: bs must be in [0, %d]", fn, kMaxRows);
  if (vocab < 4 || vocab > kMaxVocab || vocab % 4)
    return fail(NSD_ERR_UNSUPPORTED, "%s: vocab must be a multiple of 4 in [4, %d] "
                "(got %d)", fn, kMaxVocab, vocab);
  if (max_k < 0 || max_k > kMaxK)
    return fail(NSD_ERR_UNSUPPORTED, "%s: max_k must be in [0, %d] (got %d)", fn, kMaxK, max_k);
  if (bs == 0) return NSD_OK;
  if (!p_target || !uniforms || !q_indptr || !accepted_len || !out_tokens ||
      (max_k > 0 && (!q_draft || !draft_tokens)))
    return fail(NSD_ERR_NULL, "%s: NULL pointer argument", fn);
  if (((uintptr_t)p_target | (uintptr_t)(max_k > 0 ? q_draft : p_target)) & 15)
    return fail(NSD_ERR_SHAPE, "%s: probability rows must be 16-byte aligned", fn);
  Args A{p_target, q_draft, draft_tokens, uniforms, q_indptr, bs, vocab, max_k, 0,
         (int64_t)vocab, 1, nullptr, nullptr, accepted_len, out_tokens};
  return launch(false, A, bs, workspace, workspace_bytes, stream, fn);
}

// The workspace of nsd_spec_accept_static: a static device array, one copy
// per GPU the library runs on, held until the process ends.  Its host-side
// name is not a device address; kernels get the address hipGetSymbolAddress
// returns for the current device, looked up once per device and kept.
static constexpr size_t kScratchBytes = (size_t)8 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

static constexpr int kMaxScratchDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxScratchDevices];

static nsd_status scratch_address(void** out) {
  using namespace nsd;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return fail(NSD_ERR_HIP, "spec_accept_static: no current HIP device");
  }
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(NSD_ERR_UNSUPPORTED, "spec_accept_static: device %d beyond %d", dev,
                kMaxScratchDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      return fail(NSD_ERR_HIP, "spec_accept_static: the scratch array's address: %s",
                  hipGetErrorString(e));
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return NSD_OK;
}

extern "C" nsd_status nsd_spec_accept(const float* p_target, const float* q_draft,
                                      const int32_t* draft_tokens, const float* uniforms,
                                      const int32_t* q_indptr, int32_t bs, int32_t vocab,
                                      int32_t max_k, int32_t* accepted_len,
                                      int32_t* out_tokens, void* workspace,
                                      size_t workspace_bytes, void* stream) {
  return spec_accept_impl("spec_accept", p_target, q_draft, draft_tokens, uniforms, q_indptr, bs,
                          vocab, max_k, accepted_len, out_tokens, workspace, workspace_bytes,
                          stream);
}

extern "C" size_t nsd_spec_accept_static_max_bytes(void) { return kScratchBytes; }

extern "C" nsd_status nsd_spec_accept_static(const float* p_target, const float* q_draft,
                                             const int32_t* draft_tokens, const float* uniforms,
                                             const int32_t* q_indptr, int32_t bs, int32_t vocab,
                                             int32_t max_k, int32_t* accepted_len,
                                             int32_t* out_tokens, void* stream) {
  using namespace nsd;
  const char* fn = "spec_accept_static";
  if (bs > 0 && vocab >= 4 && vocab <= kMaxVocab &&
      nsd_spec_accept_workspace_size(bs, vocab) > kScratchBytes)
    return fail(NSD_ERR_WORKSPACE, "%s: bs %d at vocab %d needs %zu bytes of scratch, more "
                "than its %zu", fn, bs, vocab, nsd_spec_accept_workspace_size(bs, vocab),
                kScratchBytes);
  void* ws = nullptr;
  if (bs > 0) {
    const nsd_status st = scratch_address(&ws);
    if (st != NSD_OK) return st;
  }
  return spec_accept_impl(fn, p_target, q_draft, draft_tokens, uniforms, q_indptr, bs, vocab,
                          max_k, accepted_len, out_tokens, ws, kScratchBytes, stream);
}

extern "C" nsd_status nsd_sample(const float* probs, int64_t row_stride, const float* uniforms,
                                 int32_t n_rows, int32_t vocab, int32_t* out_tokens,
                                 int32_t out_stride, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  using namespace nsd;
  if (n_rows < 0 || n_rows > kMaxRows)
    return fail(NSD_ERR_SHAPE, "sample: n_rows must be in [0, %d]", kMaxRows);
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
  Args A{probs, nullptr, nullptr, uniforms, nullptr, n_rows, vocab, 0, 0, row_stride,
         out_stride, nullptr, nullptr, nullptr, out_tokens};
  return launch(true, A, n_rows, workspace, workspace_bytes, stream, "sample");
}
