// Execution of a KV copy plan between pinned host memory (the HostKV arena)
// and device memory (a KV bank), on the DMA engines.
//
// Passage: Appendix E.1 (long-lived host KV arenas addressed by numeric
// offsets; stable per-request extents, Eq. E.1), Appendix E.4 (copy plans
// travel as compact descriptors), Appendix E.5 (large H2D plans are split
// into bounded chunks, 32 MiB by default, so that one bank's restore cannot
// queue far ahead of the other bank's writeback on the shared copy path).
//
// A plan is a list of (source offset, destination offset, bytes) triples.
// Triples that continue each other in both buffers are merged, then every
// run is issued as asynchronous copies of at most chunk_bytes on the caller's
// stream (the caller uses a stream of its own for background preparation).
// No kernel runs: the copies use the SDMA engines, not the compute units.
#include "nsd_internal.h"

namespace {

bool pinned_host(const void* p) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return a.type == hipMemoryTypeHost;
}

bool device_mem(const void* p) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return a.type == hipMemoryTypeDevice;
}

}  // namespace

extern "C" nsd_status nsd_copy_plan(const void* src, int64_t src_bytes, void* dst,
                                    int64_t dst_bytes, const int64_t* copies, int64_t n_copies,
                                    int64_t chunk_bytes, int32_t direction, void* stream) {
  using namespace nsd;
  const char* fn = "copy_plan";
  if (n_copies < 0) return fail(NSD_ERR_SHAPE, "%s: n_copies < 0", fn);
  if (direction != NSD_COPY_H2D && direction != NSD_COPY_D2H)
    return fail(NSD_ERR_SHAPE, "%s: direction must be NSD_COPY_H2D or NSD_COPY_D2H", fn);
  if (chunk_bytes < 1) return fail(NSD_ERR_SHAPE, "%s: chunk_bytes < 1", fn);
  if (n_copies == 0) return NSD_OK;
  if (!src || !dst || !copies) return fail(NSD_ERR_NULL, "%s: NULL pointer argument", fn);
  if (src_bytes < 0 || dst_bytes < 0) return fail(NSD_ERR_SHAPE, "%s: negative buffer size", fn);
  for (int64_t i = 0; i < n_copies; ++i) {
    const int64_t s = copies[3 * i], d = copies[3 * i + 1], b = copies[3 * i + 2];
    if (s < 0 || d < 0 || b < 0 || s > src_bytes - b || d > dst_bytes - b)
      return fail(NSD_ERR_SHAPE,
                  "%s: copy %lld (src %lld, dst %lld, %lld bytes) leaves its buffers", fn,
                  (long long)i, (long long)s, (long long)d, (long long)b);
  }
  const void* host = direction == NSD_COPY_H2D ? src : (const void*)dst;
  const void* dev = direction == NSD_COPY_H2D ? (const void*)dst : src;
  if (!pinned_host(host))
    return fail(NSD_ERR_UNSUPPORTED, "%s: the host buffer is not pinned (allocate it with "
                "hipHostMalloc)", fn);
  if (!device_mem(dev)) return fail(NSD_ERR_UNSUPPORTED, "%s: the device buffer is not "
                                    "device memory", fn);
  const hipMemcpyKind kind =
      direction == NSD_COPY_H2D ? hipMemcpyHostToDevice : hipMemcpyDeviceToHost;
  const char* s8 = (const char*)src;
  char* d8 = (char*)dst;
  clear_stale_error();
  int64_t i = 0;
  while (i < n_copies) {
    // merge the triples that continue this run in both buffers
    int64_t s = copies[3 * i], d = copies[3 * i + 1], b = copies[3 * i + 2];
    ++i;
    while (i < n_copies && copies[3 * i] == s + b && copies[3 * i + 1] == d + b) {
      b += copies[3 * i + 2];
      ++i;
    }
    for (int64_t o = 0; o < b; o += chunk_bytes) {
      const int64_t len = b - o < chunk_bytes ? b - o : chunk_bytes;
      const hipError_t e = hipMemcpyAsync(d8 + d + o, s8 + s + o, (size_t)len, kind,
                                          (hipStream_t)stream);
      if (e != hipSuccess)
        return fail(NSD_ERR_HIP, "%s: hipMemcpyAsync: %s", fn, hipGetErrorString(e));
    }
  }
  return NSD_OK;
}
