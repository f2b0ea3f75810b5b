// KV-state preparation: copy arriving requests' KV blocks from the staging
// pool into the worker's paged pool (Prepare(B, w), Algorithm 1; extents of
// Appendix E.1; descriptor-driven copy plans of Appendix E.4).
//
// A pure HBM copy: every byte is read once and written once.  One workgroup
// moves one (pair, layer, plane) block with 16-byte vector loads; each thread
// issues all its loads before its stores so a workgroup keeps a whole block
// (4-32 KiB) in flight.
#include "nsd_internal.h"

namespace {

constexpr int kThreads = 256;
constexpr int kMaxVecPerThread = 8;   // 256 threads x 8 x 16 B = 32 KiB per pass

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

__global__ __launch_bounds__(kThreads)
void kv_gather_kernel(const u32x4* __restrict__ src_k, const u32x4* __restrict__ src_v,
                      int64_t src_num_blocks,
                      u32x4* __restrict__ dst_k, u32x4* __restrict__ dst_v,
                      int64_t dst_num_blocks,
                      const int32_t* __restrict__ src_ids, const int32_t* __restrict__ dst_ids,
                      int64_t n_pairs, int32_t layer0, int32_t n_layers,
                      int32_t vec_per_block) {
  // grid.x: pair, grid.y: layer offset * 2 + plane
  const int64_t pair = blockIdx.x;
  const int32_t layer = layer0 + (int32_t)(blockIdx.y >> 1);
  const bool is_v = blockIdx.y & 1;
  const int32_t s = src_ids[pair];
  const int32_t d = dst_ids[pair];
  if (s < 0 || s >= src_num_blocks || d < 0 || d >= dst_num_blocks) return;
  const u32x4* src = (is_v ? src_v : src_k) + ((int64_t)layer * src_num_blocks + s) * vec_per_block;
  u32x4* dst = (is_v ? dst_v : dst_k) + ((int64_t)layer * dst_num_blocks + d) * vec_per_block;
  for (int base = 0; base < vec_per_block; base += kThreads * kMaxVecPerThread) {
    u32x4 buf[kMaxVecPerThread];
#pragma unroll
    for (int i = 0; i < kMaxVecPerThread; ++i) {
      const int idx = base + i * kThreads + threadIdx.x;
      if (idx < vec_per_block) buf[i] = __builtin_nontemporal_load(src + idx);
    }
#pragma unroll
    for (int i = 0; i < kMaxVecPerThread; ++i) {
      const int idx = base + i * kThreads + threadIdx.x;
      if (idx < vec_per_block) __builtin_nontemporal_store(buf[i], dst + idx);
    }
  }
}

}  // namespace

extern "C" nsd_status nsd_kv_gather(const void* src_k, const void* src_v, int64_t src_num_blocks,
                                    void* dst_k, void* dst_v, int64_t dst_num_blocks,
                                    const int32_t* src_ids, const int32_t* dst_ids,
                                    int64_t n_pairs, int32_t num_layers, int32_t layer0,
                                    int32_t n_layers, int32_t num_kv_heads, int32_t block_size,
                                    int32_t head_dim, void* stream) {
  using namespace nsd;
  if (n_pairs < 0) return fail(NSD_ERR_SHAPE, "kv_gather: n_pairs < 0");
  if (num_layers < 1 || layer0 < 0 || n_layers < 0 || (int64_t)layer0 + n_layers > num_layers)
    return fail(NSD_ERR_SHAPE, "kv_gather: layer range [%d, %lld) outside [0, %d)", layer0,
                (long long)layer0 + n_layers, num_layers);
  if (block_size != NSD_BLOCK_SIZE)
    return fail(NSD_ERR_UNSUPPORTED, "kv_gather: block_size must be 16 (got %d)", block_size);
  if (head_dim != 64 && head_dim != 128)
    return fail(NSD_ERR_UNSUPPORTED, "kv_gather: head_dim must be 64 or 128 (got %d)", head_dim);
  if (num_kv_heads < 1 || num_kv_heads > 16)
    return fail(NSD_ERR_UNSUPPORTED, "kv_gather: num_kv_heads must be in [1, 16] (got %d)",
                num_kv_heads);
  if (src_num_blocks < 0 || dst_num_blocks < 0)
    return fail(NSD_ERR_SHAPE, "kv_gather: negative pool size");
  if (n_pairs == 0 || n_layers == 0) return NSD_OK;
  if (!src_k || !src_v || !dst_k || !dst_v || !src_ids || !dst_ids)
    return fail(NSD_ERR_NULL, "kv_gather: NULL pointer argument");
  if (n_pairs > 0x7fffffffLL) return fail(NSD_ERR_SHAPE, "kv_gather: n_pairs too large");
  const int64_t block_bytes = (int64_t)num_kv_heads * block_size * head_dim * 2;
  const int32_t vec = (int32_t)(block_bytes / 16);
  clear_stale_error();
  dim3 grid((uint32_t)n_pairs, (uint32_t)(2 * n_layers));
  hipLaunchKernelGGL(kv_gather_kernel, grid, dim3(kThreads), 0, (hipStream_t)stream,
                     (const u32x4*)src_k, (const u32x4*)src_v, src_num_blocks,
                     (u32x4*)dst_k, (u32x4*)dst_v, dst_num_blocks, src_ids, dst_ids, n_pairs,
                     layer0, n_layers, vec);
  return check_launch("kv_gather");
}
