/*
 * nsd_probe.h -- HBM probes (libnsd_probe.so): the practical bandwidth
 * ceiling of the access pattern of the round's attention and fused
 * preparation passes, measured by a kernel that only moves the same bytes.
 * Measurement only; not part of the verification round.
 *
 * Conventions as in nebulasd.h: device pointers, work enqueued on `stream`
 * (a hipStream_t), nothing allocated, nothing waited for; 0 = OK,
 * 1 = a required pointer is NULL, 2 = a size out of range, 5 = launch error.
 */
#ifndef NSD_PROBE_H
#define NSD_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Stream 4 KiB tiles the way verification attention streams its paged K/V
 * (Section 3: paged blocks at arbitrary positions): `waves` persistent waves
 * (one per SIMD; a multiple of 4), wave w reading the `steps` * 4 tiles
 * ids[w*steps*4 ...] of `src` in groups of four with the next group in
 * flight (up to 32 KiB per wave).  With dst_ids non-NULL, a tile whose
 * dst_ids entry is in [0, dst_tiles) is also written to that tile of `dst`
 * right after it is read (the fused preparation's write-back of arriving
 * tiles, Algorithm 1 Prepare).
 *
 * src: src_tiles * 4096 bytes; dst: dst_tiles * 4096 bytes (may be NULL with
 * dst_ids NULL); ids, dst_ids: int32 [waves * steps * 4], ids clamped into
 * [0, src_tiles); sink: at least waves * 1024 bytes of device memory (written
 * only in a case that does not occur for real data, so the loads stay live).
 */
int32_t nsd_probe_tiles(const void* src, int64_t src_tiles, void* dst, int64_t dst_tiles,
                        const int32_t* ids, const int32_t* dst_ids, int32_t waves,
                        int32_t steps, void* sink, void* stream);

/*
 * The same reads with the write-back moved to waves that do not read:
 * waves / 4 workgroups of five waves (one workgroup per CU), waves 0-3 of
 * workgroup k reading as nsd_probe_tiles' waves 4k..4k+3 do (dst_ids NULL),
 * and wave 4 storing, from registers, the tiles write_ids[k * write_per ..
 * (k + 1) * write_per) of `dst` (entries outside [0, dst_tiles) skipped).
 * Separates the cost of mixing reads and writes in the memory system from
 * the cost of stores issued among a wave's loads.  steps = 0 gives the
 * writes alone (src and ids may then be NULL).
 *
 * write_ids: int32 [waves / 4 * write_per]; other arguments as above.
 */
int32_t nsd_probe_tiles_writer(const void* src, int64_t src_tiles, void* dst, int64_t dst_tiles,
                               const int32_t* ids, const int32_t* write_ids, int32_t write_per,
                               int32_t waves, int32_t steps, void* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif
