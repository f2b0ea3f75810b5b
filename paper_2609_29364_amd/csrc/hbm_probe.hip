// HBM probes: the practical bandwidth ceiling of the access patterns the round's
// kernels make, measured with kernels that do nothing but move those bytes.
//
// The verification-attention pass streams 4 KiB (block, KV head) tiles of K
// and V from random pool positions (a shuffled paged cache), one resident
// wave per SIMD, with up to 32 KiB of tiles in flight per wave; the fused
// preparation pass also writes the tiles of arriving requests back to other
// random positions.  nsd_probe_tiles reproduces exactly that traffic without
// any arithmetic, so its rate is what the memory system gives this pattern,
// the rate the real kernels are measured against (beside the 8 TB/s peak).
//
// Separate library (libnsd_probe.so): measurement only, not part of the round.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "nsd_probe.h"

namespace {

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

constexpr int kTileVec = 4096 / (64 * 16);   // 16-byte loads per lane per 4 KiB tile
constexpr int kGroup = 4;                     // tiles per group; two groups in flight

// One wave streams `steps` groups of G tiles, ids wid[0 .. steps*G), the next
// group requested before the current one is consumed.  With STORE, a tile
// whose wdst entry is in [0, dst_tiles) is stored to that destination tile
// right after it is used.
template <bool STORE>
__device__ inline void stream_tiles(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                    int64_t src_tiles, int64_t dst_tiles,
                                    const int32_t* __restrict__ wid,
                                    const int32_t* __restrict__ wdst, int32_t steps, int lane,
                                    u32x4* __restrict__ sink) {
  u32x4 a[kGroup][kTileVec], b[kGroup][kTileVec];
  u32x4 acc = {0, 0, 0, 0};
  auto load = [&](u32x4(&r)[kGroup][kTileVec], int s) {
#pragma unroll
    for (int g = 0; g < kGroup; ++g) {
      int64_t t = __builtin_amdgcn_readfirstlane(wid[s * kGroup + g]);
      t = t < 0 ? 0 : (t >= src_tiles ? src_tiles - 1 : t);   // ids are clamped into the buffer
      const u32x4* p = src + t * (64 * kTileVec) + lane;
#pragma unroll
      for (int i = 0; i < kTileVec; ++i) r[g][i] = __builtin_nontemporal_load(p + i * 64);
    }
  };
  auto use = [&](u32x4(&r)[kGroup][kTileVec], int s) {
#pragma unroll
    for (int g = 0; g < kGroup; ++g)
#pragma unroll
      for (int i = 0; i < kTileVec; ++i) acc ^= r[g][i];
    if constexpr (STORE) {
#pragma unroll
      for (int g = 0; g < kGroup; ++g) {
        const int64_t d = __builtin_amdgcn_readfirstlane(wdst[s * kGroup + g]);
        if (d < 0 || d >= dst_tiles) continue;
        u32x4* q = dst + d * (64 * kTileVec) + lane;
#pragma unroll
        for (int i = 0; i < kTileVec; ++i) __builtin_nontemporal_store(r[g][i], q + i * 64);
      }
    }
  };
  if (steps <= 0) return;
  load(a, 0);
  for (int s = 0; s + 1 < steps; s += 2) {
    load(b, s + 1);
    use(a, s);
    if (s + 2 < steps) load(a, s + 2);
    use(b, s + 1);
  }
  if (steps & 1) use(a, steps - 1);
  // keeps the loads alive; the data are never all-ones words in practice
  if ((acc.x & acc.y & acc.z & acc.w) == 0xffffffffu) *sink = acc;
}

// Wave w streams tiles ids[w*steps*G .. (w+1)*steps*G).
template <bool STORE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1)))
void tiles_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                  int64_t src_tiles, int64_t dst_tiles, const int32_t* __restrict__ ids,
                  const int32_t* __restrict__ dst_ids, int32_t steps,
                  u32x4* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  stream_tiles<STORE>(src, dst, src_tiles, dst_tiles, ids + wave * steps * kGroup,
                      STORE ? dst_ids + wave * steps * kGroup : nullptr, steps, lane,
                      sink + wave * 64 + lane);
}

// Workgroups of five waves: waves 0-3 only read (reader wave 4k+i of the
// launch streams tiles ids[(4k+i)*steps*G ...]), wave 4 of workgroup k only
// writes: the tiles write_ids[k*write_per .. (k+1)*write_per) of dst, from
// registers (entries outside [0, dst_tiles) are skipped).
__global__ __launch_bounds__(320) __attribute__((amdgpu_waves_per_eu(2)))
void writer_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst, int64_t src_tiles,
                   int64_t dst_tiles, const int32_t* __restrict__ ids,
                   const int32_t* __restrict__ write_ids, int32_t write_per, int32_t steps,
                   u32x4* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  if (w == 4) {
    const int32_t* my = write_ids + (int64_t)blockIdx.x * write_per;
    const u32x4 v = {(uint32_t)lane, (uint32_t)blockIdx.x, 0u, 0u};
    for (int i = 0; i < write_per; ++i) {
      const int64_t d = __builtin_amdgcn_readfirstlane(my[i]);
      if (d < 0 || d >= dst_tiles) continue;
      u32x4* q = dst + d * (64 * kTileVec) + lane;
#pragma unroll
      for (int k = 0; k < kTileVec; ++k) __builtin_nontemporal_store(v, q + k * 64);
    }
    return;
  }
  const int64_t wave = (int64_t)blockIdx.x * 4 + w;
  stream_tiles<false>(src, nullptr, src_tiles, 0, ids + wave * steps * kGroup, nullptr, steps,
                      lane, sink + wave * 64 + lane);
}

}  // namespace

extern "C" int32_t nsd_probe_tiles(const void* src, int64_t src_tiles, void* dst,
                                   int64_t dst_tiles, const int32_t* ids,
                                   const int32_t* dst_ids, int32_t waves, int32_t steps,
                                   void* sink, void* stream) {
  if (!src || !ids || !sink || (dst_ids && !dst)) return 1;
  if (waves <= 0 || waves % 4 != 0 || steps < 0 || src_tiles <= 0 || (dst_ids && dst_tiles <= 0))
    return 2;
  hipStream_t s = (hipStream_t)stream;
  const dim3 grid(waves / 4), block(256);
  if (dst_ids)
    hipLaunchKernelGGL(tiles_kernel<true>, grid, block, 0, s, (const u32x4*)src, (u32x4*)dst,
                       src_tiles, dst_tiles, ids, dst_ids, steps, (u32x4*)sink);
  else
    hipLaunchKernelGGL(tiles_kernel<false>, grid, block, 0, s, (const u32x4*)src, nullptr,
                       src_tiles, (int64_t)0, ids, nullptr, steps, (u32x4*)sink);
  return hipGetLastError() == hipSuccess ? 0 : 5;
}

extern "C" int32_t nsd_probe_tiles_writer(const void* src, int64_t src_tiles, void* dst,
                                          int64_t dst_tiles, const int32_t* ids,
                                          const int32_t* write_ids, int32_t write_per,
                                          int32_t waves, int32_t steps, void* sink,
                                          void* stream) {
  if (!dst || !write_ids || !sink || (steps > 0 && (!src || !ids))) return 1;
  if (waves <= 0 || waves % 4 != 0 || steps < 0 || write_per < 0 || dst_tiles <= 0 ||
      (steps > 0 && src_tiles <= 0))
    return 2;
  // more than half the LDS a workgroup may use, so that one workgroup runs per
  // CU, as in the attention pass
  int dev = 0, lds_max = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) !=
          hipSuccess)
    return 5;
  const size_t lds = lds_max > 65536 ? (size_t)lds_max / 2 + 4096 : 0;
  hipLaunchKernelGGL(writer_kernel, dim3(waves / 4), dim3(320), lds, (hipStream_t)stream,
                     (const u32x4*)src, (u32x4*)dst, src_tiles, dst_tiles, ids, write_ids,
                     write_per, steps, (u32x4*)sink);
  return hipGetLastError() == hipSuccess ? 0 : 5;
}
