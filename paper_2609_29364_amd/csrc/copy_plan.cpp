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
// The windowed variant is the bounded submission of Appendix E.5: only a
// group of chunks up to window_bytes is queued at a time, and the calling
// (DMA) thread waits for each group to complete before it submits the next,
// so a large restore cannot queue far ahead of the other bank's writeback.
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

// Validation and submission shared by both entry points.  window_bytes > 0
// bounds the bytes submitted ahead of completion: before a chunk that would
// take the bytes in flight past the window is submitted, the calling thread
// waits until the oldest chunks in flight have completed (an event recorded
// after each chunk, kept in a ring), so the copy path holds at most a window
// of this plan at any time while the next chunk is already queued behind the
// one running.
nsd_status submit_plan(const char* fn, const void* src, int64_t src_bytes, void* dst,
                       int64_t dst_bytes, const int64_t* copies, int64_t n_copies,
                       int64_t chunk_bytes, int64_t window_bytes, int32_t direction,
                       void* stream) {
  using namespace nsd;
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
  // ring of the chunks in flight: completion event and bytes, oldest first
  constexpr int kRing = 64;
  hipEvent_t ring[kRing] = {};
  int64_t ring_bytes[kRing] = {};
  int head = 0, count = 0;
  int64_t in_flight = 0;
  auto finish = [&](nsd_status st) {
    for (int k = 0; k < kRing; ++k)
      if (ring[k]) (void)hipEventDestroy(ring[k]);
    return st;
  };
  if (window_bytes > 0) {
    for (int k = 0; k < kRing; ++k) {
      const hipError_t e = hipEventCreateWithFlags(&ring[k], hipEventDisableTiming);
      if (e != hipSuccess)
        return finish(fail(NSD_ERR_HIP, "%s: hipEventCreateWithFlags: %s", fn,
                           hipGetErrorString(e)));
    }
  }
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
      // wait for the oldest chunks until this one fits in the window (and
      // the ring has a free entry)
      while (window_bytes > 0 && count > 0 &&
             (in_flight + len > window_bytes || count == kRing)) {
        const hipError_t e = hipEventSynchronize(ring[head]);
        if (e != hipSuccess)
          return finish(fail(NSD_ERR_HIP, "%s: waiting for a chunk: %s", fn,
                             hipGetErrorString(e)));
        in_flight -= ring_bytes[head];
        head = (head + 1) % kRing;
        --count;
      }
      hipError_t e = hipMemcpyAsync(d8 + d + o, s8 + s + o, (size_t)len, kind,
                                    (hipStream_t)stream);
      if (e != hipSuccess)
        return finish(fail(NSD_ERR_HIP, "%s: hipMemcpyAsync: %s", fn, hipGetErrorString(e)));
      if (window_bytes > 0) {
        const int k = (head + count) % kRing;
        e = hipEventRecord(ring[k], (hipStream_t)stream);
        if (e != hipSuccess)
          return finish(fail(NSD_ERR_HIP, "%s: hipEventRecord: %s", fn, hipGetErrorString(e)));
        ring_bytes[k] = len;
        in_flight += len;
        ++count;
      }
    }
  }
  return finish(NSD_OK);
}

}  // namespace

extern "C" nsd_status nsd_copy_plan(const void* src, int64_t src_bytes, void* dst,
                                    int64_t dst_bytes, const int64_t* copies, int64_t n_copies,
                                    int64_t chunk_bytes, int32_t direction, void* stream) {
  return submit_plan("copy_plan", src, src_bytes, dst, dst_bytes, copies, n_copies, chunk_bytes,
                     0, direction, stream);
}

extern "C" nsd_status nsd_copy_plan_windowed(const void* src, int64_t src_bytes, void* dst,
                                             int64_t dst_bytes, const int64_t* copies,
                                             int64_t n_copies, int64_t chunk_bytes,
                                             int64_t window_bytes, int32_t direction,
                                             void* stream) {
  if (window_bytes < 1)
    return nsd::fail(NSD_ERR_SHAPE, "copy_plan_windowed: window_bytes < 1");
  return submit_plan("copy_plan_windowed", src, src_bytes, dst, dst_bytes, copies, n_copies,
                     chunk_bytes, window_bytes, direction, stream);
}

// Plan arithmetic of the preparation and the writeback (host code).
//
// H2D plan (Algorithm 1, Prepare; Appendix E.1, Eq. E.1): block j of
// arriving request r goes from arena block extent[r] + j to bank block
// stage_table[r][j], for j < ceil(seq_lens[r] / 16), request by request (a
// request whose staging ids are consecutive becomes one run once merged).
extern "C" nsd_status nsd_h2d_plan(const int64_t* extent, const int32_t* stage_table,
                                   int32_t max_blocks_per_seq, const uint8_t* arriving,
                                   const int32_t* seq_lens, int32_t bs, int64_t block_bytes,
                                   int64_t* copies, int64_t capacity, int64_t* n_copies) {
  using namespace nsd;
  const char* fn = "h2d_plan";
  if (bs < 0 || max_blocks_per_seq < 1 || block_bytes < 1 || capacity < 0)
    return fail(NSD_ERR_SHAPE, "%s: bad sizes", fn);
  if (!n_copies) return fail(NSD_ERR_NULL, "%s: NULL pointer argument", fn);
  if (bs > 0 && (!extent || !stage_table || !arriving || !seq_lens))
    return fail(NSD_ERR_NULL, "%s: NULL pointer argument", fn);
  int64_t n = 0;
  for (int32_t r = 0; r < bs; ++r) {
    if (!arriving[r]) continue;
    const int64_t nb = seq_lens[r] > 0 ? ((int64_t)seq_lens[r] + NSD_BLOCK_SIZE - 1) / NSD_BLOCK_SIZE
                                       : 0;
    if (nb > max_blocks_per_seq)
      return fail(NSD_ERR_SHAPE, "%s: request %d has %lld blocks, more than the table's %d", fn,
                  r, (long long)nb, max_blocks_per_seq);
    // every byte offset of the request must be a non-negative int64
    const int64_t max_block = INT64_MAX / block_bytes - 1;
    if (nb > 0 && (extent[r] < 0 || extent[r] > max_block - nb + 1))
      return fail(NSD_ERR_SHAPE, "%s: request %d: arena extent %lld outside [0, %lld]", fn, r,
                  (long long)extent[r], (long long)(max_block - nb + 1));
    for (int64_t j = 0; j < nb; ++j, ++n) {
      const int32_t sid = stage_table[(int64_t)r * max_blocks_per_seq + j];
      if (sid < 0 || sid > max_block)
        return fail(NSD_ERR_SHAPE, "%s: request %d block %lld: staging id %d outside [0, %lld]",
                    fn, r, (long long)j, sid, (long long)max_block);
      if (n >= capacity || !copies) continue;   // counted, not written
      copies[3 * n] = (extent[r] + j) * block_bytes;
      copies[3 * n + 1] = (int64_t)sid * block_bytes;
      copies[3 * n + 2] = block_bytes;
    }
  }
  *n_copies = n;
  if (n > capacity) return fail(NSD_ERR_WORKSPACE, "%s: %lld copies, room for %lld", fn,
                                (long long)n, (long long)capacity);
  return NSD_OK;
}

// Writeback pairs (Section 5: incremental writeback of the valid suffix;
// Appendix E.1 extents): with host_len[r] tokens already in the arena and
// new_len[r] committed, the blocks holding tokens host_len .. new_len - 1 go
// from pool block block_table[r][j] to arena block extent[r] + j, request by
// request.
extern "C" nsd_status nsd_writeback_pairs(const int32_t* block_table, int32_t max_blocks_per_seq,
                                          const int64_t* extent, const int32_t* host_len,
                                          const int32_t* new_len, int32_t bs, int32_t* src_ids,
                                          int32_t* dst_ids, int64_t capacity, int64_t* n_pairs) {
  using namespace nsd;
  const char* fn = "writeback_pairs";
  if (bs < 0 || max_blocks_per_seq < 1 || capacity < 0)
    return fail(NSD_ERR_SHAPE, "%s: bad sizes", fn);
  if (!n_pairs) return fail(NSD_ERR_NULL, "%s: NULL pointer argument", fn);
  if (bs > 0 && (!block_table || !extent || !host_len || !new_len))
    return fail(NSD_ERR_NULL, "%s: NULL pointer argument", fn);
  int64_t n = 0;
  for (int32_t r = 0; r < bs; ++r) {
    const int64_t h = host_len[r], l = new_len[r];
    if (l <= h) continue;
    if (h < 0 || (l - 1) / NSD_BLOCK_SIZE >= max_blocks_per_seq)
      return fail(NSD_ERR_SHAPE, "%s: request %d: tokens [%lld, %lld) outside its block table", fn,
                  r, (long long)h, (long long)l);
    if (extent[r] < 0)
      return fail(NSD_ERR_SHAPE, "%s: request %d: negative arena extent %lld", fn, r,
                  (long long)extent[r]);
    if (extent[r] > INT32_MAX)
      return fail(NSD_ERR_UNSUPPORTED, "%s: arena block %lld beyond 2^31 - 1", fn,
                  (long long)extent[r]);
    for (int64_t j = h / NSD_BLOCK_SIZE; j <= (l - 1) / NSD_BLOCK_SIZE; ++j, ++n) {
      if (n >= capacity || !src_ids || !dst_ids) continue;
      const int64_t a = extent[r] + j;   // both below 2^31: no overflow
      if (a > INT32_MAX)
        return fail(NSD_ERR_UNSUPPORTED, "%s: arena block %lld beyond 2^31 - 1", fn, (long long)a);
      src_ids[n] = block_table[(int64_t)r * max_blocks_per_seq + j];
      dst_ids[n] = (int32_t)a;
    }
  }
  *n_pairs = n;
  if (n > capacity) return fail(NSD_ERR_WORKSPACE, "%s: %lld pairs, room for %lld", fn,
                                (long long)n, (long long)capacity);
  return NSD_OK;
}
