/*
 * nebulasd.h -- C ABI of the verification-round library (libnebulasd.so).
 *
 * One speculative verification round on a reconstructed batch (NebulaSD,
 * Algorithm 1: Prepare then Run) is three calls on one HIP stream:
 *
 *   nsd_kv_gather         KV-state preparation of arriving requests
 *   nsd_verify_attention  grouped-query attention of the anchor + K proposal
 *                         queries of every request over the paged KV cache
 *   nsd_spec_accept       acceptance of proposals and residual resampling
 *
 * The draft stage before it (Eq. 1) is single-query nsd_verify_attention
 * steps, each after nsd_kv_append of the processed token, and nsd_sample.
 *
 * nsd_gather_verify_attention does the first two in one pass (each staged
 * byte read once); nsd_copy_plan moves KV between a pinned host arena and a
 * device bank (the host-side source of the preparation).
 *
 * Conventions shared by every call
 * --------------------------------
 * - Pointers named as device pointers must address memory the GPU of
 *   `stream` can read/write; all work is enqueued on `stream` (a hipStream_t,
 *   NULL = the null stream) and the call returns without waiting.  The caller
 *   owns every buffer, including workspaces, and keeps it alive until the
 *   stream has passed the call.  The library allocates nothing.  Its state
 *   is a thread-local error message, launch facts it queries once per device
 *   (CU count, occupancy, LDS size) and the wave count of
 *   nsd_set_attention_waves.
 * - Arguments are validated on the host before anything is enqueued; a bad
 *   scalar or NULL pointer returns an error status and enqueues nothing.
 *   Device-resident contents (block ids, lengths, offsets, tokens) are not
 *   visible to the host: contents outside the documented ranges give
 *   unspecified results, but every kernel clamps them so that it never reads
 *   or writes outside the buffers whose sizes the scalars describe.  The one
 *   device-resident size is the row count total_q = q_indptr[bs] of the
 *   query-row buffers (q, out, target rows, uniforms, window rows), which
 *   must equal their rows; every other q_indptr entry is clamped into
 *   [0, total_q].  nsd_check_plan / nsd_check_pairs validate host copies of
 *   the metadata against the documented ranges before a round runs.
 * - Calls never abort and never print.  Calls on different streams with
 *   disjoint outputs may run concurrently.
 * - bf16 is bfloat16 (1 sign, 8 exponent, 7 mantissa bits) stored in 2 bytes.
 *
 * Paged KV layout (Section 3: paged KV blocks; Appendix E.1: separate K and V
 * planes).  A block holds BLOCK_SIZE = 16 consecutive token slots of one
 * request for every KV head.  Per layer:
 *   K plane: bf16 [num_blocks][num_kv_heads][head_dim/8][16][8]
 *            (16-byte runs of 8 dimensions; the 16 slots of one run index are
 *            adjacent)
 *   V plane: bf16 [num_blocks][num_kv_heads][head_dim][16]
 *            (the 16 slots of one dimension are adjacent)
 * A multi-layer pool stacks layers outermost: [num_layers][num_blocks][...].
 * Token t of a request lives in slot t % 16 of block block_table[r][t / 16].
 */
#ifndef NEBULASD_H
#define NEBULASD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t nsd_status;

#define NSD_OK              0
#define NSD_ERR_NULL        1  /* a required pointer is NULL */
#define NSD_ERR_SHAPE       2  /* a size/count argument is out of range */
#define NSD_ERR_UNSUPPORTED 3  /* valid in principle, not implemented (e.g. head_dim) */
#define NSD_ERR_WORKSPACE   4  /* workspace pointer NULL or smaller than required */
#define NSD_ERR_HIP         5  /* the HIP runtime reported an error; see nsd_last_error */

#define NSD_BLOCK_SIZE 16

/* Library version, (major << 16) | minor. */
int32_t nsd_version(void);

/* Message describing the last non-OK status returned on the calling thread.
   Valid until the next library call on that thread.  Never NULL. */
const char* nsd_last_error(void);

/*
 * KV-state preparation: copy whole KV blocks of arriving requests from a
 * staging pool into the worker's paged pool.
 *
 * Passage: Algorithm 1 (Prepare(B, w) makes the batch's KV state resident on
 * worker w before Run); Appendix E.1 (each request's state sits in a stable
 * extent of blocks, Eq. E.1, addressed by numeric offsets); Appendix E.4
 * (copy plans travel as compact descriptors).
 *
 * For every pair i in [0, n_pairs) and every layer l in [layer0, layer0+n_layers):
 *     dst_k[l][dst_ids[i]] <- src_k[l][src_ids[i]]
 *     dst_v[l][dst_ids[i]] <- src_v[l][src_ids[i]]
 * copying the whole block (all KV heads, all 16 slots).  Blocks not named by
 * dst_ids are not written.
 *
 * src_k, src_v : device, bf16 [num_layers][src_num_blocks][block], layout above.
 * dst_k, dst_v : device, bf16 [num_layers][dst_num_blocks][block].
 * src_ids, dst_ids : device, int32 [n_pairs].  Ids must lie in [0, src_num_blocks)
 *                / [0, dst_num_blocks) and dst_ids must be distinct; a pair with
 *                an id out of range is skipped.
 * num_layers : layers in both pools; 0 <= layer0, layer0 + n_layers <= num_layers.
 * num_kv_heads >= 1, block_size == 16, head_dim in {64, 128}.
 * n_pairs == 0 or n_layers == 0 is a no-op returning NSD_OK.
 * Source and destination must not overlap.
 */
nsd_status nsd_kv_gather(const void* src_k, const void* src_v, int64_t src_num_blocks,
                         void* dst_k, void* dst_v, int64_t dst_num_blocks,
                         const int32_t* src_ids, const int32_t* dst_ids, int64_t n_pairs,
                         int32_t num_layers, int32_t layer0, int32_t n_layers,
                         int32_t num_kv_heads, int32_t block_size, int32_t head_dim,
                         void* stream);

/*
 * Bytes of workspace nsd_verify_attention and nsd_gather_verify_attention
 * need for these sizes on the current HIP device (0 if the sizes are
 * invalid).  The size depends on the arguments and on how many waves the
 * device keeps resident (its CU count), or on the count set with
 * nsd_set_attention_waves.
 */
size_t nsd_verify_attention_workspace_size(int32_t bs, int32_t num_q_heads,
                                           int32_t num_kv_heads, int32_t head_dim,
                                           int32_t max_q_per_seq, int32_t max_seq_len);

/*
 * Test and tuning hook: the attention entry points and the workspace query
 * split their work over `waves` resident waves (a positive multiple of 4, at
 * most 2^20) instead of the device's own count; 0 restores the device's
 * count.  Process-wide: set it only while no other thread queries workspace
 * sizes or launches attention.  Any other value returns NSD_ERR_SHAPE.
 * nsd_attention_waves returns the current setting (0: the device's count).
 * Results do not depend on the wave count beyond floating-point summation
 * order; the tests use it to force items cut into partials or whole.
 */
nsd_status nsd_set_attention_waves(int32_t waves);
int32_t    nsd_attention_waves(void);

/*
 * Verification attention for one layer.
 *
 * Passage: Section 1 (the target model verifies the draft's proposals in one
 * forward pass); Appendix G.2 and H (a round scores the anchor token plus d
 * proposal tokens per request); Section 3 (the KV cache is paged and
 * append-dominant: it already holds the window's states).
 *
 * Request r has n_q = q_indptr[r+1] - q_indptr[r] query tokens (anchor plus
 * K_r proposals) and L_r = seq_lens[r] cached tokens including those n_q.
 * Query j sits at position L_r - n_q + j and attends to tokens 0 .. L_r-n_q+j
 * of its request.  Query head h reads KV head h / (num_q_heads/num_kv_heads).
 *     out[q_indptr[r]+j][h] = softmax_t(scale * <q, k_t>) . v_t
 * computed from bf16 inputs with fp32 accumulation (the softmax weights enter
 * the second product as bf16; a row split over several waves is merged from
 * per-part rows stored normalised in bf16 with fp32 max and sum); out is
 * rounded to bf16.
 * A query row with no visible token (only if n_q > L_r) is written as 0.
 *
 * q        : device, bf16 [total_q][num_q_heads][head_dim], total_q = q_indptr[bs].
 * k_cache, v_cache : device, this layer's planes, [num_blocks][...] (layout above).
 * block_table : device, int32 [bs][max_blocks_per_seq]; entries past
 *               ceil(L_r/16) do not affect the result.  Ids outside
 *               [0, num_blocks) make their block's tokens invisible.
 *               num_blocks * num_kv_heads must not exceed 2^31 - 1.
 * seq_lens : device, int32 [bs], 1 <= L_r <= max_seq_len, L_r <= 16*max_blocks_per_seq.
 * q_indptr : device, int32 [bs+1], non-decreasing, q_indptr[0] = 0,
 *            1 <= n_q <= min(max_q_per_seq, L_r); q_indptr[bs] = total_q must
 *            be the row count of q and out (other entries are clamped into
 *            [0, total_q], n_q to max_q_per_seq).
 * num_q_heads % num_kv_heads == 0; (num_q_heads/num_kv_heads) * max_q_per_seq <= 64.
 * head_dim in {64, 128}; block_size == 16.
 * scale : the softmax scale (usually 1/sqrt(head_dim)), finite.
 * out : device, bf16 [total_q][num_q_heads][head_dim]; may not alias q or the caches.
 * workspace : device, at least nsd_verify_attention_workspace_size(...) bytes,
 *             any contents (each call writes what it reads).  Calls sharing a
 *             workspace must be ordered on one stream.
 * 1 <= bs <= 8192 (bs == 0 is a no-op returning NSD_OK).
 */
nsd_status nsd_verify_attention(const void* q, const void* k_cache, const void* v_cache,
                                int64_t num_blocks, const int32_t* block_table,
                                int32_t max_blocks_per_seq, const int32_t* seq_lens,
                                const int32_t* q_indptr, int32_t bs, int32_t num_q_heads,
                                int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                                int32_t max_q_per_seq, int32_t max_seq_len, float scale,
                                void* out, void* workspace, size_t workspace_bytes,
                                void* stream);

/*
 * KV-state preparation fused with verification attention, for one layer.
 *
 * Passage: Algorithm 1 (Prepare makes an arriving request's KV state resident
 * on the worker, then Run verifies); Appendix E.1 (the state comes from a
 * stable per-request extent of blocks).  Same computation and arguments as
 * nsd_verify_attention, plus:
 *   k_stage, v_stage : device, staging planes of this layer, bf16
 *                      [stage_num_blocks][...] (layout above);
 *   stage_table      : device, int32 [bs][max_blocks_per_seq]; row r holds the
 *                      staging block of each of request r's blocks if r is
 *                      arriving (entry 0 >= 0), or -1 in entry 0 if r is
 *                      resident in the worker pool.
 * For an arriving request, block b (b < ceil(L_r/16)) is read from
 * k/v_stage[stage_table[r][b]] instead of the worker pool, and the whole block
 * (all KV heads, all 16 slots) is written to k/v_cache[block_table[r][b]], as
 * nsd_kv_gather with the pairs (stage_table[r][b], block_table[r][b]) would:
 * each staged byte is read from HBM once.  The caches are therefore read and
 * written (non-const); the blocks of different requests must be distinct.
 * stage_num_blocks == 0 treats every request as resident.  A staging id
 * outside [0, stage_num_blocks) makes its block's tokens invisible and the
 * block is not written (as nsd_kv_gather skips such a pair); destination ids
 * outside [0, num_blocks) are not written.  num_blocks * num_kv_heads and
 * stage_num_blocks * num_kv_heads must not exceed 2^31 - 1.
 */
nsd_status nsd_gather_verify_attention(const void* q, void* k_cache, void* v_cache,
                                       int64_t num_blocks, const void* k_stage,
                                       const void* v_stage, int64_t stage_num_blocks,
                                       const int32_t* block_table, const int32_t* stage_table,
                                       int32_t max_blocks_per_seq, const int32_t* seq_lens,
                                       const int32_t* q_indptr, int32_t bs, int32_t num_q_heads,
                                       int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                                       int32_t max_q_per_seq, int32_t max_seq_len, float scale,
                                       void* out, void* workspace, size_t workspace_bytes,
                                       void* stream);

#define NSD_COPY_H2D 1  /* pinned host -> device */
#define NSD_COPY_D2H 2  /* device -> pinned host */

/*
 * Execute a KV copy plan between a pinned host arena (HostKV) and device
 * memory (a KV bank) on the DMA engines, asynchronously on `stream`.
 *
 * Passage: Appendix E.1 (persistent host KV arenas addressed by numeric
 * offsets; each request owns a stable extent of blocks, Eq. E.1), Appendix
 * E.4 (copy plans as compact descriptors), Appendix E.5 (H2D plans are
 * split into bounded chunks, 32 MiB by default).
 *
 * copies : host, int64 [n_copies][3] = (source byte offset, destination byte
 *          offset, bytes).  Each triple must lie inside [0, src_bytes) and
 *          [0, dst_bytes).  Triples that continue the previous one in both
 *          buffers are merged; every run is issued as copies of at most
 *          chunk_bytes (>= 1) bytes, in plan order.
 * direction : NSD_COPY_H2D (src pinned host, dst device) or NSD_COPY_D2H
 *          (src device, dst pinned host).  The host side must be pinned
 *          memory (hipHostMalloc; registering existing pages is not used),
 *          else NSD_ERR_UNSUPPORTED.
 * Overlapping destination ranges give unspecified bytes.  n_copies == 0 is
 * a no-op.  The plan array is read before the call returns; the buffers must
 * stay alive until the stream has passed the copies.
 */
nsd_status nsd_copy_plan(const void* src, int64_t src_bytes, void* dst, int64_t dst_bytes,
                         const int64_t* copies, int64_t n_copies, int64_t chunk_bytes,
                         int32_t direction, void* stream);

/*
 * nsd_copy_plan with bounded submission (Appendix E.5: only a bounded group
 * of chunks of a large H2D plan is submitted before the DMA process waits for
 * its completion and submits the next group, so one bank's restore cannot
 * queue far ahead of the other bank's writeback on the shared copy path).
 * Chunks of at most chunk_bytes are submitted so that at most window_bytes
 * (>= 1; a chunk larger than the window goes alone) and at most 64 chunks of
 * this plan are in flight: before submitting a chunk that would exceed that,
 * the call waits, on the calling host thread, until the oldest chunks in
 * flight have completed.  It returns once the last chunk is submitted (its
 * copies still run); callers run it on a DMA thread of their own.  Other
 * arguments, checks and errors as nsd_copy_plan.
 */
nsd_status nsd_copy_plan_windowed(const void* src, int64_t src_bytes, void* dst,
                                  int64_t dst_bytes, const int64_t* copies, int64_t n_copies,
                                  int64_t chunk_bytes, int64_t window_bytes, int32_t direction,
                                  void* stream);

/*
 * The preparation's copy plan (host code): block j < ceil(seq_lens[r] / 16)
 * of every arriving request r (arriving[r] != 0) goes from arena block
 * extent[r] + j to bank block stage_table[r][j], as the triple
 * (arena byte offset, bank byte offset, block_bytes), request by request.
 *
 * Passage: Algorithm 1 (Prepare restores the batch's state on the worker);
 * Appendix E.1 (stable per-request extents in the host arena, Eq. E.1);
 * Appendix E.4 (copy plans as compact descriptors).
 * extent: int64 [bs]; stage_table: int32 [bs][max_blocks_per_seq];
 * arriving: uint8 [bs]; seq_lens: int32 [bs]; copies: int64 [capacity][3].
 * *n_copies gets the plan's length; if it exceeds capacity only the first
 * capacity triples are written and NSD_ERR_WORKSPACE is returned.  A request
 * with more blocks than the table holds, a negative extent or staging id of an
 * arriving request, or a byte offset beyond 2^63 - 1 returns NSD_ERR_SHAPE.
 * Host memory.
 */
nsd_status nsd_h2d_plan(const int64_t* extent, const int32_t* stage_table,
                        int32_t max_blocks_per_seq, const uint8_t* arriving,
                        const int32_t* seq_lens, int32_t bs, int64_t block_bytes,
                        int64_t* copies, int64_t capacity, int64_t* n_copies);

/*
 * The writeback's block pairs (host code): with host_len[r] tokens already in
 * the arena and new_len[r] committed, the blocks holding tokens host_len[r] ..
 * new_len[r] - 1 go from pool block block_table[r][j] to arena block
 * extent[r] + j, request by request (nsd_kv_gather's (src, dst) pairs, e.g.
 * through nsd_host_alias).
 *
 * Passage: Section 5 (incremental writeback of only the valid suffix not yet
 * persistent); Appendix E.1 (stable extents); Appendix E.2 (a bank exports its
 * updated suffix before it is released).
 * block_table: int32 [bs][max_blocks_per_seq]; extent: int64 [bs]; host_len,
 * new_len: int32 [bs]; src_ids, dst_ids: int32 [capacity].  *n_pairs and
 * NSD_ERR_WORKSPACE as nsd_h2d_plan; tokens outside the table or a negative
 * extent of a request with a suffix return NSD_ERR_SHAPE, an arena block
 * beyond 2^31 - 1 NSD_ERR_UNSUPPORTED.  Host memory.
 */
nsd_status nsd_writeback_pairs(const int32_t* block_table, int32_t max_blocks_per_seq,
                               const int64_t* extent, const int32_t* host_len,
                               const int32_t* new_len, int32_t bs, int32_t* src_ids,
                               int32_t* dst_ids, int64_t capacity, int64_t* n_pairs);

/*
 * Append the window's new K/V rows to the paged cache, for one layer.
 *
 * Passage: Section 3 (the cache is paged and append-dominant: an iteration
 * only adds the K/V of the tokens it processed).
 *
 * Row q_indptr[r] + j of k_new / v_new (bf16 [total_q][num_kv_heads][head_dim])
 * is window token j of request r, at position t = seq_lens[r] - n_q + j; it is
 * written to slot t % 16 of block block_table[r][t / 16] of k_pool / v_pool
 * (this layer's planes, layout above), every KV head.  No other slot
 * changes: the kernel writes whole 32-byte sectors (a V row's 16 slots, a K
 * run pair), so the other slots of a sector the window touches are written
 * back with their own contents, and no other operation may write those
 * blocks while the call runs.  Positions outside [0, 16 * max_blocks_per_seq)
 * and block ids outside [0, num_blocks) are skipped; two requests naming one
 * block give unspecified contents in it.  k_pool and v_pool are 16-byte
 * aligned (NSD_ERR_SHAPE otherwise).  block_size == 16, head_dim in
 * {64, 128}.  bs == 0 or total_q == 0 is a no-op.
 */
nsd_status nsd_kv_append(void* k_pool, void* v_pool, int64_t num_blocks, const void* k_new,
                         const void* v_new, const int32_t* block_table,
                         int32_t max_blocks_per_seq, const int32_t* seq_lens,
                         const int32_t* q_indptr, int32_t bs, int32_t total_q,
                         int32_t num_kv_heads, int32_t block_size, int32_t head_dim,
                         void* stream);

/*
 * Commit accepted lengths: new_lens[r] = seq_lens[r] - K_r + n_r, with
 * K_r = q_indptr[r+1] - q_indptr[r] - 1 and n_r = accepted_len[r] clamped to
 * [0, K_r].  The request keeps its anchor and its accepted proposals; the
 * resampled or bonus token is the next round's anchor.
 *
 * Passage: Sections 1 and 3 (verified tokens are committed; the cache only
 * grows by what an iteration adds); Section 5 (HostKV records each
 * request's valid sequence length).
 * All pointers device, int32 [bs] (q_indptr [bs+1]); new_lens may alias
 * seq_lens.  bs == 0 is a no-op.
 */
nsd_status nsd_commit_lengths(const int32_t* seq_lens, const int32_t* q_indptr,
                              const int32_t* accepted_len, int32_t* new_lens, int32_t bs,
                              void* stream);

/*
 * Device address of pinned host memory (hipHostMalloc), so that kernels, such
 * as nsd_kv_gather writing a request's KV suffix back into its HostKV extent,
 * can read or write it directly.
 *
 * Passage: Section 5 and Appendix E.1 (incremental writeback of the valid
 * suffix into the persistent pinned host arena).
 * Returns NSD_ERR_UNSUPPORTED if `host` is not pinned memory mapped for the
 * current device.
 */
nsd_status nsd_host_alias(const void* host, void** device_alias);

/*
 * Speculative acceptance with residual resampling.
 *
 * Passage: Sections 1 and 2 (speculative decoding as in Leviathan et al. 2023
 * and Chen et al. 2023, which the paper cites for the verification rule).
 *
 * Request r has K_r = q_indptr[r+1] - q_indptr[r] - 1 proposals.  Its target
 * rows are p_target[q_indptr[r] + i] (i = 0..K_r), its draft rows and
 * proposal tokens q_draft[q_indptr[r] - r + i] and draft_tokens[q_indptr[r] - r + i]
 * (i = 0..K_r-1), its uniforms uniforms[q_indptr[r] + i] (i = 0..K_r: K_r
 * acceptance uniforms then one sampling uniform).
 *   1. Proposal i is accepted iff u_i * q_i(x_i) <= p_i(x_i), evaluated exactly
 *      (fp64 product of fp32 values); n = first rejected i, or K_r.  A proposal
 *      token outside [0, vocab) is rejected.
 *   2. Weights w = max(0, p_n - q_n) if n < K_r (p_n if that has no mass),
 *      else w = p_{K_r} (the bonus row); accumulated in fp64.
 *   3. y = min{t : C(t) > u_{K_r} * C(vocab-1)}, C the inclusive prefix sum of
 *      w in token order (last token of positive weight if rounding leaves none);
 *      a token of zero weight is never emitted.
 * Outputs: accepted_len[r] = n; out_tokens[q_indptr[r] + i] = x_i for i < n,
 * y at i = n, -1 for n < i <= K_r.
 *
 * p_target : device, fp32 [total_q][vocab];  q_draft : device, fp32 [total_q-bs][vocab]
 * draft_tokens : device, int32 [total_q-bs];  uniforms : device, fp32 [total_q], in [0,1)
 * q_indptr : device, int32 [bs+1], q_indptr[0] = 0, 0 <= K_r <= max_k;
 *            q_indptr[bs] = total_q must be the row count of p_target and
 *            uniforms.  Other entries are clamped so that a request's target
 *            rows stay below total_q and its draft rows inside [0, total_q-bs);
 *            a request whose first row clamps to total_q gets accepted_len 0
 *            and no token.
 * vocab : 4 <= vocab <= 2^19, vocab % 4 == 0; 0 <= max_k <= 63.
 * accepted_len : device, int32 [bs];  out_tokens : device, int32 [total_q].
 * Row bases must be 16-byte aligned (true for hipMalloc'd/torch tensors).
 * q_draft and draft_tokens may be NULL when max_k == 0.  bs <= 2^31 / 32;
 * bs == 0 is a no-op.
 * workspace : device, 8-byte aligned, at least
 * nsd_spec_accept_workspace_size(bs, vocab) bytes, any contents (per-chunk
 * sums of each request's weight row; the call writes all it reads); calls
 * that overlap in time need separate workspaces.  Too small a workspace
 * returns NSD_ERR_WORKSPACE.
 */
size_t     nsd_spec_accept_workspace_size(int32_t rows, int32_t vocab);
nsd_status nsd_spec_accept(const float* p_target, const float* q_draft,
                           const int32_t* draft_tokens, const float* uniforms,
                           const int32_t* q_indptr, int32_t bs, int32_t vocab, int32_t max_k,
                           int32_t* accepted_len, int32_t* out_tokens, void* workspace,
                           size_t workspace_bytes, void* stream);

/*
 * nsd_spec_accept without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments, semantics and results
 * as nsd_spec_accept; its per-chunk sums live in a static device array of
 * nsd_spec_accept_static_max_bytes() bytes (8 MiB) that each GPU the library
 * runs on holds until the process ends.  A batch whose
 * nsd_spec_accept_workspace_size(bs, vocab) exceeds that returns
 * NSD_ERR_WORKSPACE (e.g. more than 1700 requests at vocab 151936).  The call
 * allocates nothing.  Every call on one GPU shares that GPU's array: calls
 * that overlap in time on one GPU race, so order them on one stream.  The
 * array needs no clearing (each call writes what it reads).
 */
size_t     nsd_spec_accept_static_max_bytes(void);
nsd_status nsd_spec_accept_static(const float* p_target, const float* q_draft,
                                  const int32_t* draft_tokens, const float* uniforms,
                                  const int32_t* q_indptr, int32_t bs, int32_t vocab,
                                  int32_t max_k, int32_t* accepted_len, int32_t* out_tokens,
                                  void* stream);

/*
 * Draw one token per row by inverse CDF: the sampling of a draft step,
 * x_i ~ q_i (the draft stage precedes verification, Eq. 1; speculative
 * decoding as in the works cited in Sections 1 and 2).
 *
 * Row r is w = probs[r * row_stride .. r * row_stride + vocab) (nonnegative
 * weights, any total), its uniform uniforms[r] in [0,1).  The token is step 3
 * of nsd_spec_accept on that row: y = min{t : C(t) > u_r * C(vocab-1)} over
 * fp64 prefix sums in token order (the last token of positive weight if
 * rounding leaves none; -1 if the row has no mass); it is written to
 * out_tokens[r * out_stride].  With probs and out_tokens offset by step i and
 * strides K * vocab and K, step i of a K-step chain reads the draft rows and
 * writes the proposal tokens in the request-major layout nsd_spec_accept
 * takes (q_draft row and draft_tokens entry r * K + i).
 *
 * probs : device fp32, 16-byte aligned; row_stride (elements) >= vocab and a
 * multiple of 4.  uniforms : device fp32 [n_rows].  out_tokens : device int32,
 * n_rows entries at stride out_stride >= 1.  vocab as in nsd_spec_accept;
 * n_rows <= 2^31 / 32.  workspace as in nsd_spec_accept, of
 * nsd_spec_accept_workspace_size(n_rows, vocab) bytes.  n_rows == 0 is a
 * no-op.
 */
nsd_status nsd_sample(const float* probs, int64_t row_stride, const float* uniforms,
                      int32_t n_rows, int32_t vocab, int32_t* out_tokens, int32_t out_stride,
                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * Host validation of a round's metadata: host copies of the arrays the
 * attention, fused and append calls read from device memory, checked against
 * the ranges those calls document (host code; no GPU involved).
 *
 * Passage: Section 3 (paged blocks and a block map per request), Section 5
 * (each request's valid length), Appendix G.2/H (anchor plus proposals per
 * request), Appendix F.2 (capacity checks before a batch runs: block ids
 * inside the bank, lengths inside its token limit).
 *
 * Checks: q_indptr[0] = 0 and, if total_q >= 0, q_indptr[bs] = total_q;
 * every request has 1 <= L_r <= min(max_seq_len, 16 * max_blocks_per_seq)
 * and 1 <= n_q <= min(max_q_per_seq, L_r) (so q_indptr increases); its
 * block ids b < ceil(L_r / 16) lie in [0, num_blocks).  With a stage_table
 * (the fused call), pool blocks are distinct over the batch, and every
 * arriving request (entry 0 >= 0) has staging ids in [0, stage_num_blocks),
 * distinct over the batch.  Returns NSD_OK, or NSD_ERR_SHAPE with
 * nsd_last_error naming the first violation (NSD_ERR_NULL for a missing
 * array).  All pointers are host memory; stage_table may be NULL.
 */
nsd_status nsd_check_plan(const int32_t* block_table, const int32_t* stage_table,
                          int32_t max_blocks_per_seq, const int32_t* seq_lens,
                          const int32_t* q_indptr, int32_t bs, int64_t num_blocks,
                          int64_t stage_num_blocks, int32_t max_q_per_seq, int32_t max_seq_len,
                          int64_t total_q);

/*
 * Host validation of a gather plan (nsd_kv_gather's pairs): every source id
 * in [0, src_num_blocks), every destination id in [0, dst_num_blocks) and
 * destination ids distinct.  Passage: Appendix E.4 (copy plans as numeric
 * descriptors), Appendix F.2 (block capacity).  Host pointers; returns as
 * nsd_check_plan.
 */
nsd_status nsd_check_pairs(const int32_t* src_ids, const int32_t* dst_ids, int64_t n_pairs,
                           int64_t src_num_blocks, int64_t dst_num_blocks);

/*
 * Worker-triggered batch reconstruction: one scheduling opportunity (host
 * code; no GPU involved).
 *
 * Passage: Section 4, Algorithm 1 and Eqs. 4-8 (predicted predecessor
 * completion, batch KV-ready and start times, service-admission bound,
 * admissibility); Appendix F.2 (capacity fit, each request individually).
 *
 * Candidate i is request ids[i] with available predecessor completion time
 * e_tilde[i] and KV-ready time k_hat[i] on the worker, which is available at
 * a_hat.  S({r}) = max(a_hat, e~_r, k^_r); d^_r = max(e~_r + g, S({r})) + delta.
 * Candidates with blocks[i] > block_cap or tokens[i] > token_cap are dropped;
 * the rest are ranked by (d^_r, S({r}), id) ascending (earliest admission
 * bound first: a longer wait gives an earlier bound), the first b_max of them
 * are scanned once in that order and r joins if the batch stays admissible:
 * its blocks and tokens within the capacities and
 * max(a_hat, max e~, max k^) <= min d^ over the batch.
 * blocks / tokens may be NULL (all zero).  ids must be distinct; times may be
 * +/-infinity but not NaN; g, delta >= 0 (delta may be +infinity).
 * Out: batch[0 .. *batch_len) in admission order (batch holds b_max entries),
 * *batch_start = S(B) (NaN when the batch is empty).  n == 0 gives an empty
 * batch.  All pointers host memory.
 */
nsd_status nsd_reconstruct(const int32_t* ids, const double* e_tilde, const double* k_hat,
                           const int64_t* blocks, const int64_t* tokens, int32_t n, double a_hat,
                           int64_t block_cap, int64_t token_cap, int32_t b_max, double g,
                           double delta, int32_t* batch, int32_t* batch_len,
                           double* batch_start);

/*
 * Profiling-driven discrete-event simulation of the two worker pools with
 * ideal migration (host code; no GPU involved).
 *
 * Passage: Appendix H (simulation methodology: virtual clock, all transitions
 * at one time applied before scheduling, compute and Prepare opportunities per
 * worker, zero migration latency; all requests start after prefill at t = 0
 * and run a fixed number of rounds; Eqs. H.1 and H.2 and the request-round
 * rate over a window); Eq. 1 (draft before target in every round); Appendix F
 * (standby-bank planning, early planning with predicted predecessor ends,
 * Prepare then Run on InputReady, KVReady and WorkerReady).
 *
 * Workers 0 .. n_draft-1 serve the draft stage, the next n_target the target
 * stage.  Stage s takes phi_s(b) for a batch of b requests, with SM activity
 * sm_s(b), both interpolated linearly over the table's batch sizes (constant
 * beyond its ends).  At every virtual time: completions; then, until nothing
 * changes, each worker without a prepared batch (index order) reconstructs
 * one (nsd_reconstruct with a_hat = the end of its running batch or now,
 * k^ = now, no capacity limit, stage s's b_max, g, delta) over the requests
 * whose next stage is s and whose latest other-stage instance is running
 * (e~ = its predicted end) or done, and each idle worker whose prepared batch
 * has every predecessor output published starts it.
 *
 * phi_d / phi_t : host double [3][n] = batch sizes (ascending), stage times
 *                 (> 0), SM activity, for the draft and target stages.
 * metrics : U = sum_j tau_j sm_j / ((n_draft + n_target) (w1 - w0)),
 *           S = sum_j tau_j b_j / (n_requests (w1 - w0)), round_rate =
 *           request-level target rounds ending in (w0, w1] / (w1 - w0),
 *           finished requests, batches started; tau_j = overlap of batch j
 *           with [w0, w1].
 * trace / members (optional, NULL with capacity 0): batch j's record and its
 *           request ids at members[first .. first + size), in start order.
 *           If either buffer is too small the simulation still completes,
 *           metrics are valid, *n_trace / *n_members give the sizes needed
 *           and NSD_ERR_WORKSPACE is returned.
 * The run stops when no batch is running, or once virtual time passes t_stop
 * (INFINITY: run to completion).
 */
typedef struct {
  int32_t n_draft, n_target;  /* workers per pool, >= 1 each */
  int32_t n_requests, rounds; /* requests, speculative rounds per request */
  int32_t b_max[2];           /* [draft, target] maximum batch sizes */
  double g[2];                /* target service intervals g_s, >= 0 */
  double delta[2];            /* slacks Delta_s, >= 0 */
  double window[2];           /* measurement window [w0, w1], w0 < w1 */
  double t_stop;
} nsd_sim_config;

typedef struct {
  double U, S, round_rate;
  int64_t finished, batches;
} nsd_sim_metrics;

typedef struct {
  int32_t stage;   /* 0 draft, 1 target */
  int32_t worker;  /* index within its pool */
  int32_t size;
  int64_t first;   /* offset of its members */
  double start, end;
} nsd_sim_batch;

nsd_status nsd_simulate(const nsd_sim_config* cfg, const double* phi_d, int32_t n_phi_d,
                        const double* phi_t, int32_t n_phi_t, nsd_sim_metrics* metrics,
                        nsd_sim_batch* trace, int64_t trace_cap, int32_t* members,
                        int64_t members_cap, int64_t* n_trace, int64_t* n_members);

#ifdef __cplusplus
}
#endif

#endif /* NEBULASD_H */
