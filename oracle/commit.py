"""Oracle for the steps that close a verification round: appending the window's
new K/V to the paged cache, committing the accepted length, and the suffix to
write back to the host arena.

* The cache is append-dominant: each iteration only adds the K/V of the tokens
  it processed (Section 3); the window of request r is its anchor and its K_r
  proposals, at positions L_r - n_q .. L_r - 1 (n_q = K_r + 1), and token t
  lives in slot t % 16 of block block_table[r][t // 16] (Section 3, paged
  cache; the block layout of the boundary).
* After acceptance a request keeps its anchor and the n_r accepted proposals:
  its committed length is L_r - K_r + n_r (the resampled or bonus token has no
  K/V yet; it is the next round's anchor).
* Writeback moves only the suffix that is not yet in the host arena (Section 5,
  incremental KV writeback; Appendix E.1): with H_r tokens already valid there,
  the blocks covering tokens [H_r, L'_r) are copied whole, block j of the
  request to block extent[r] + j of the arena.
"""
import numpy as np

BLOCK = 16


def kv_append(k_pool, v_pool, k_new, v_new, block_table, seq_lens, q_indptr):
    """Return the pool planes after writing the window rows.

    k_pool: [blocks][Hkv][D/8][16][8], v_pool: [blocks][Hkv][D][16] (any dtype,
    values copied).  k_new, v_new: [total_q][Hkv][D], row q_indptr[r] + j is
    window token j of request r.  Pools are left untouched (copies returned)."""
    out_k = np.array(k_pool, copy=True)
    out_v = np.array(v_pool, copy=True)
    bs = len(seq_lens)
    for r in range(bs):
        a, b = int(q_indptr[r]), int(q_indptr[r + 1])
        nq = b - a
        L = int(seq_lens[r])
        for j in range(nq):
            t = L - nq + j
            blk = int(block_table[r, t // BLOCK])
            s = t % BLOCK
            for g in range(k_new.shape[1]):
                for d in range(k_new.shape[2]):
                    out_k[blk, g, d // 8, s, d % 8] = k_new[a + j, g, d]
                    out_v[blk, g, d, s] = v_new[a + j, g, d]
    return out_k, out_v


def commit_lengths(seq_lens, q_indptr, accepted_len):
    """Committed lengths L_r - K_r + n_r."""
    L = np.asarray(seq_lens, dtype=np.int64)
    k = np.diff(np.asarray(q_indptr, dtype=np.int64)) - 1
    return L - k + np.asarray(accepted_len, dtype=np.int64)


def writeback_pairs(block_table, extent, host_len, new_len):
    """(pool block id, arena block id) pairs of the suffix each request writes back:
    the blocks holding its tokens host_len .. new_len - 1, request by request."""
    src, dst = [], []
    for r in range(len(new_len)):
        h, n = int(host_len[r]), int(new_len[r])
        if n <= h:
            continue
        for j in range(h // BLOCK, (n - 1) // BLOCK + 1):
            src.append(int(block_table[r, j]))
            dst.append(int(extent[r]) + j)
    return np.array(src, dtype=np.int64), np.array(dst, dtype=np.int64)
