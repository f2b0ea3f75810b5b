// Closing a verification round: the window's new K/V rows are appended to the
// paged cache, and each request's accepted length is committed.
//
// The cache is append-dominant: an iteration only adds the K/V of the tokens
// it processed (Section 3).  Request r's window (anchor + K_r proposals) sits
// at positions L_r - n_q .. L_r - 1; token t lives in slot t % 16 of block
// block_table[r][t / 16].  After acceptance the request keeps its anchor and
// its n_r accepted proposals: L'_r = L_r - K_r + n_r (the resampled or bonus
// token is the next round's anchor).
//
// kv_append: one workgroup per (KV head, request).  Memory writes whole
// 32-byte sectors cheaply and partial ones with a read-modify-write in the
// memory system, which also delays the kernels that follow (a decode
// attention launched right after an append made of 2-byte element stores
// ran 6 % slower).  So the kernel writes whole sectors only: for every block
// the window touches, thread d rewrites dimension d's 16-slot V row (32
// bytes) and thread (run c, slot pair) the two 16-byte K runs of a slot
// pair, taking the window's slots from the new rows and every other slot
// from the sector's current contents.  Only this workgroup writes the
// (block, KV head) tile, so the merge needs no ordering.  Volume: the
// sectors the window touches, read and written (about 4.5 KiB each way per
// (request, KV head) for a one-token window at head_dim 128, 13 MB each way
// for a verify_8b layer's five-token windows).
#include "nsd_internal.h"

namespace {

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

// 32 bytes as 16 bf16 (two 16-byte accesses)
struct Sector {
  uint16_t e[16];
};

__device__ inline Sector load_sector(const uint16_t* p) {
  Sector s;
  const u32x4 a = ((const u32x4*)p)[0], b = ((const u32x4*)p)[1];
  __builtin_memcpy(&s.e[0], &a, 16);
  __builtin_memcpy(&s.e[8], &b, 16);
  return s;
}

__device__ inline void store_sector(uint16_t* p, const Sector& s) {
  u32x4 a, b;
  __builtin_memcpy(&a, &s.e[0], 16);
  __builtin_memcpy(&b, &s.e[8], 16);
  ((u32x4*)p)[0] = a;
  ((u32x4*)p)[1] = b;
}

__global__ __launch_bounds__(128) void kv_append_kernel(
    uint16_t* __restrict__ k_pool, uint16_t* __restrict__ v_pool,
    const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new,
    const int32_t* __restrict__ block_table, const int32_t* __restrict__ seq_lens,
    const int32_t* __restrict__ q_indptr, int64_t num_blocks, int32_t max_blocks_per_seq,
    int32_t num_kv_heads, int32_t head_dim, int32_t total_q) {
  const int g = blockIdx.x;
  const int r = blockIdx.y;
  const int tid = threadIdx.x;
  const int a = q_indptr[r];
  const int nq = q_indptr[r + 1] - a;
  const int L = seq_lens[r];
  if (nq <= 0) return;
  // window positions inside [0, 16 * max_blocks_per_seq)
  const int64_t t0 = max((int64_t)L - nq, (int64_t)0);
  const int64_t t1 = min((int64_t)L - 1, (int64_t)max_blocks_per_seq * 16 - 1);
  const int runs = head_dim / 8;
  for (int64_t blk = t0 / 16; blk <= t1 / 16 && t0 <= t1; ++blk) {
    const int32_t id = block_table[(int64_t)r * max_blocks_per_seq + blk];
    if (id < 0 || id >= num_blocks) continue;   // an invalid id is not written
    const int s_lo = (int)(max(t0, blk * 16) - blk * 16);
    const int s_hi = (int)(min(t1, blk * 16 + 15) - blk * 16);
    const int64_t tile = ((int64_t)id * num_kv_heads + g) * head_dim * 16;
    // the window row of slot s (a row outside [0, total_q) leaves the slot)
    auto row_of = [&](int s) -> int64_t {
      const int64_t row = (int64_t)a + (blk * 16 + s) - ((int64_t)L - nq);
      return row >= 0 && row < total_q ? row : -1;
    };
    if (tid < head_dim) {
      uint16_t* vp = v_pool + tile + (int64_t)tid * 16;
      Sector row = load_sector(vp);
#pragma unroll
      for (int s = 0; s < 16; ++s) {   // fixed indices keep the sector in registers
        const int64_t q = s >= s_lo && s <= s_hi ? row_of(s) : -1;
        if (q >= 0) row.e[s] = v_new[(q * num_kv_heads + g) * head_dim + tid];
      }
      store_sector(vp, row);
    }
    const int p_lo = s_lo / 2, np = s_hi / 2 - p_lo + 1;
    if (tid < runs * np) {
      const int c = tid % runs, pr = p_lo + tid / runs;
      uint16_t* kp = k_pool + tile + (int64_t)(c * 16 + 2 * pr) * 8;
      Sector run2 = load_sector(kp);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int s = 2 * pr + u;
        const int64_t q = s >= s_lo && s <= s_hi ? row_of(s) : -1;
        if (q < 0) continue;
        const uint16_t* src = k_new + (q * num_kv_heads + g) * head_dim + c * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) run2.e[u * 8 + e] = src[e];
      }
      store_sector(kp, run2);
    }
  }
}

__global__ __launch_bounds__(256) void commit_kernel(const int32_t* __restrict__ seq_lens,
                                                     const int32_t* __restrict__ q_indptr,
                                                     const int32_t* __restrict__ accepted_len,
                                                     int32_t* __restrict__ new_lens, int32_t bs) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= bs) return;
  const int k = max(0, q_indptr[r + 1] - q_indptr[r] - 1);
  const int n = min(max(accepted_len[r], 0), k);
  new_lens[r] = seq_lens[r] - k + n;
}

}  // namespace

extern "C" nsd_status nsd_kv_append(void* k_pool, void* v_pool, int64_t num_blocks,
                                    const void* k_new, const void* v_new,
                                    const int32_t* block_table, int32_t max_blocks_per_seq,
                                    const int32_t* seq_lens, const int32_t* q_indptr,
                                    int32_t bs, int32_t total_q, int32_t num_kv_heads,
                                    int32_t block_size, int32_t head_dim, void* stream) {
  using namespace nsd;
  const char* fn = "kv_append";
  if (block_size != NSD_BLOCK_SIZE)
    return fail(NSD_ERR_UNSUPPORTED, "%s: block_size must be 16 (got %d)", fn, block_size);
  if (head_dim != 64 && head_dim != 128)
    return fail(NSD_ERR_UNSUPPORTED, "%s: head_dim must be 64 or 128 (got %d)", fn, head_dim);
  if (bs < 0 || total_q < 0 || num_kv_heads < 1 || num_kv_heads > 65535 || bs > 65535 ||
      max_blocks_per_seq < 1 || num_blocks < 0)
    return fail(NSD_ERR_SHAPE, "%s: bad sizes", fn);
  if (bs == 0 || total_q == 0) return NSD_OK;
  if (!k_pool || !v_pool || !k_new || !v_new || !block_table || !seq_lens || !q_indptr)
    return fail(NSD_ERR_NULL, "%s: NULL pointer argument", fn);
  if (((uintptr_t)k_pool | (uintptr_t)v_pool) % 16)
    return fail(NSD_ERR_SHAPE, "%s: k_pool and v_pool must be 16-byte aligned", fn);
  clear_stale_error();
  hipLaunchKernelGGL(kv_append_kernel, dim3(num_kv_heads, bs), dim3(128), 0, (hipStream_t)stream,
                     (uint16_t*)k_pool, (uint16_t*)v_pool, (const uint16_t*)k_new,
                     (const uint16_t*)v_new, block_table, seq_lens, q_indptr, num_blocks,
                     max_blocks_per_seq, num_kv_heads, head_dim, total_q);
  return check_launch(fn);
}

extern "C" nsd_status nsd_commit_lengths(const int32_t* seq_lens, const int32_t* q_indptr,
                                         const int32_t* accepted_len, int32_t* new_lens,
                                         int32_t bs, void* stream) {
  using namespace nsd;
  const char* fn = "commit_lengths";
  if (bs < 0) return fail(NSD_ERR_SHAPE, "%s: bs < 0", fn);
  if (bs == 0) return NSD_OK;
  if (!seq_lens || !q_indptr || !accepted_len || !new_lens)
    return fail(NSD_ERR_NULL, "%s: NULL pointer argument", fn);
  clear_stale_error();
  hipLaunchKernelGGL(commit_kernel, dim3((uint32_t)(((int64_t)bs + 255) / 256)), dim3(256), 0,
                     (hipStream_t)stream,
                     seq_lens, q_indptr, accepted_len, new_lens, bs);
  return check_launch(fn);
}

extern "C" nsd_status nsd_host_alias(const void* host, void** device_alias) {
  using namespace nsd;
  if (!host || !device_alias) return fail(NSD_ERR_NULL, "host_alias: NULL pointer argument");
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, host) != hipSuccess || a.type != hipMemoryTypeHost ||
      !a.devicePointer) {
    (void)hipGetLastError();
    return fail(NSD_ERR_UNSUPPORTED, "host_alias: not pinned host memory mapped for the device");
  }
  // the alias of the allocation base, shifted to this pointer
  *device_alias = (char*)a.devicePointer + ((const char*)host - (const char*)a.hostPointer);
  return NSD_OK;
}
