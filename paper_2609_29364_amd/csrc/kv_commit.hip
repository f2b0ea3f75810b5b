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
// kv_append: one workgroup per (KV head, request), one lane per dimension;
// the lanes of a 16-byte K run write one contiguous run, V elements land at
// their slot of each dimension's 16-slot row.  The volume is the window only
// (verify_8b: 1280 rows x 8 heads x 128 dims x 2 planes x 2 bytes = 5 MB).
#include "nsd_internal.h"

namespace {

__global__ __launch_bounds__(128) void kv_append_kernel(
    uint16_t* __restrict__ k_pool, uint16_t* __restrict__ v_pool,
    const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new,
    const int32_t* __restrict__ block_table, const int32_t* __restrict__ seq_lens,
    const int32_t* __restrict__ q_indptr, int64_t num_blocks, int32_t max_blocks_per_seq,
    int32_t num_kv_heads, int32_t head_dim, int32_t total_q) {
  const int g = blockIdx.x;
  const int r = blockIdx.y;
  const int d = threadIdx.x;
  if (d >= head_dim) return;
  const int a = q_indptr[r];
  const int nq = q_indptr[r + 1] - a;
  const int L = seq_lens[r];
  for (int j = 0; j < nq; ++j) {
    const int t = L - nq + j;
    const int row = a + j;
    if (t < 0 || t >= max_blocks_per_seq * 16 || row < 0 || row >= total_q) continue;
    const int32_t id = block_table[(int64_t)r * max_blocks_per_seq + t / 16];
    if (id < 0 || id >= num_blocks) continue;   // an invalid id is not written
    const int s = t % 16;
    const int64_t tile = ((int64_t)id * num_kv_heads + g) * head_dim * 16;
    const int64_t src = ((int64_t)row * num_kv_heads + g) * head_dim + d;
    k_pool[tile + ((d / 8) * 16 + s) * 8 + d % 8] = k_new[src];
    v_pool[tile + (int64_t)d * 16 + s] = v_new[src];
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
  hipLaunchKernelGGL(commit_kernel, dim3((bs + 255) / 256), dim3(256), 0, (hipStream_t)stream,
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
