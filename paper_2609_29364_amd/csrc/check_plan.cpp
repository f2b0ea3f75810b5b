// Host-side validation of a round's metadata (host copies of the arrays the
// kernels read from device memory).  The kernels clamp device-resident
// contents so that they never address memory outside their buffers, but
// contents outside the documented ranges give unspecified results; these
// checks say, before a round runs, whether a plan is inside those ranges.
//
// What a plan must satisfy follows the statement of the round: every request
// of the batch has a valid length and a block map (Section 3, paged KV blocks;
// Section 5, valid-length metadata), its query window is the anchor plus its
// proposals (Appendix G.2/H), and the capacity checks of batch admission
// (Appendix F.2: block ids inside the bank, lengths inside the token limit,
// requests on blocks of their own where a call writes them).
#include <vector>

#include "nsd_internal.h"

namespace {

constexpr int kBlock = NSD_BLOCK_SIZE;

}  // namespace

extern "C" nsd_status nsd_check_plan(const int32_t* block_table, const int32_t* stage_table,
                                     int32_t max_blocks_per_seq, const int32_t* seq_lens,
                                     const int32_t* q_indptr, int32_t bs, int64_t num_blocks,
                                     int64_t stage_num_blocks, int32_t max_q_per_seq,
                                     int32_t max_seq_len, int64_t total_q) {
  using namespace nsd;
  const char* fn = "check_plan";
  if (bs < 0 || max_blocks_per_seq < 1 || num_blocks < 0 || stage_num_blocks < 0 ||
      max_q_per_seq < 1 || max_seq_len < 1)
    return fail(NSD_ERR_SHAPE, "%s: bad sizes", fn);
  if (bs == 0) {
    if (total_q > 0) return fail(NSD_ERR_SHAPE, "%s: total_q %lld for an empty batch", fn,
                                 (long long)total_q);
    return NSD_OK;
  }
  if (!block_table || !seq_lens || !q_indptr) return fail(NSD_ERR_NULL, "%s: NULL pointer", fn);
  if (q_indptr[0] != 0) return fail(NSD_ERR_SHAPE, "%s: q_indptr[0] = %d, not 0", fn, q_indptr[0]);
  if (total_q >= 0 && q_indptr[bs] != total_q)
    return fail(NSD_ERR_SHAPE, "%s: q_indptr[bs] = %d, but q has %lld rows", fn, q_indptr[bs],
                (long long)total_q);
  std::vector<unsigned char> used_pool(stage_table ? (size_t)num_blocks : 0, 0);
  std::vector<unsigned char> used_stage((size_t)stage_num_blocks, 0);
  for (int32_t r = 0; r < bs; ++r) {
    const int64_t L = seq_lens[r];
    const int64_t nq = (int64_t)q_indptr[r + 1] - q_indptr[r];
    if (L < 1 || L > max_seq_len || L > (int64_t)kBlock * max_blocks_per_seq)
      return fail(NSD_ERR_SHAPE, "%s: request %d: seq_len %lld outside [1, min(max_seq_len %d, "
                  "16 * max_blocks_per_seq %d)]", fn, r, (long long)L, max_seq_len,
                  kBlock * max_blocks_per_seq);
    if (nq < 1 || nq > max_q_per_seq || nq > L)
      return fail(NSD_ERR_SHAPE, "%s: request %d: %lld query rows outside [1, min(max_q_per_seq "
                  "%d, seq_len %lld)] (q_indptr must increase)", fn, r, (long long)nq,
                  max_q_per_seq, (long long)L);
    const int64_t nblk = (L + kBlock - 1) / kBlock;
    const int32_t* row = block_table + (int64_t)r * max_blocks_per_seq;
    for (int64_t b = 0; b < nblk; ++b) {
      const int32_t id = row[b];
      if (id < 0 || id >= num_blocks)
        return fail(NSD_ERR_SHAPE, "%s: request %d block %lld: pool id %d outside [0, %lld)", fn,
                    r, (long long)b, id, (long long)num_blocks);
      // the fused pass writes arriving blocks into the pool: blocks must then
      // be distinct (plain attention only reads, so it may share them)
      if (stage_table && used_pool[id]++)
        return fail(NSD_ERR_SHAPE, "%s: pool block %d is used twice", fn, id);
    }
    if (!stage_table) continue;
    const int32_t* srow = stage_table + (int64_t)r * max_blocks_per_seq;
    if (srow[0] < 0) continue;   // resident request
    for (int64_t b = 0; b < nblk; ++b) {
      const int32_t id = srow[b];
      if (id < 0 || id >= stage_num_blocks)
        return fail(NSD_ERR_SHAPE, "%s: request %d block %lld: staging id %d outside [0, %lld)",
                    fn, r, (long long)b, id, (long long)stage_num_blocks);
      if (used_stage[id]++)
        return fail(NSD_ERR_SHAPE, "%s: staging block %d is used twice", fn, id);
    }
  }
  return NSD_OK;
}

extern "C" nsd_status nsd_check_pairs(const int32_t* src_ids, const int32_t* dst_ids,
                                      int64_t n_pairs, int64_t src_num_blocks,
                                      int64_t dst_num_blocks) {
  using namespace nsd;
  const char* fn = "check_pairs";
  if (n_pairs < 0 || src_num_blocks < 0 || dst_num_blocks < 0)
    return fail(NSD_ERR_SHAPE, "%s: bad sizes", fn);
  if (n_pairs == 0) return NSD_OK;
  if (!src_ids || !dst_ids) return fail(NSD_ERR_NULL, "%s: NULL pointer", fn);
  std::vector<unsigned char> used((size_t)dst_num_blocks, 0);
  for (int64_t i = 0; i < n_pairs; ++i) {
    if (src_ids[i] < 0 || src_ids[i] >= src_num_blocks)
      return fail(NSD_ERR_SHAPE, "%s: pair %lld: source id %d outside [0, %lld)", fn,
                  (long long)i, src_ids[i], (long long)src_num_blocks);
    if (dst_ids[i] < 0 || dst_ids[i] >= dst_num_blocks)
      return fail(NSD_ERR_SHAPE, "%s: pair %lld: destination id %d outside [0, %lld)", fn,
                  (long long)i, dst_ids[i], (long long)dst_num_blocks);
    if (used[dst_ids[i]]++)
      return fail(NSD_ERR_SHAPE, "%s: destination block %d is named twice", fn, dst_ids[i]);
  }
  return NSD_OK;
}
