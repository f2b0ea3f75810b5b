"""Byte layout of the paged KV pools (the format the C-ABI documents).

The KV cache is paged in fixed blocks of 16 token slots (Section 3, KV cache
organization), with K and V held in separate planes (Appendix E.1).  Within a
block, for each KV head:

* K is stored as [head_dim/8][16 slots][8]: each 16-byte run holds 8
  consecutive dimensions of one slot, and the 16 slots of a run index follow
  one another.
* V is stored as [head_dim][16 slots]: the 16 slots of one dimension are
  contiguous.

A pool plane is therefore  K: [layers][blocks][kv_heads][head_dim/8][16][8]
and V: [layers][blocks][kv_heads][head_dim][16], bf16.
"""
import torch

BLOCK_SIZE = 16
K_VEC = 8          # bf16 elements per 16-byte run in the K plane


def k_block_shape(num_kv_heads: int, head_dim: int):
    return (num_kv_heads, head_dim // K_VEC, BLOCK_SIZE, K_VEC)


def v_block_shape(num_kv_heads: int, head_dim: int):
    return (num_kv_heads, head_dim, BLOCK_SIZE)


def logical_kv_from_blocks(k_blocks: torch.Tensor, v_blocks: torch.Tensor, length: int):
    """Logical per-token K/V [length][kv_heads][head_dim] of one request.

    k_blocks: [nb][Hkv][D/8][16][8] and v_blocks: [nb][Hkv][D][16], the request's
    blocks in logical order (block j holds tokens 16j .. 16j+15).
    """
    nb, hkv, dv, bsz, vec = k_blocks.shape
    d = dv * vec
    k = k_blocks.permute(0, 3, 1, 2, 4).reshape(nb * bsz, hkv, d)
    v = v_blocks.permute(0, 3, 1, 2).reshape(nb * bsz, hkv, d)
    return k[:length], v[:length]


def poison_slots(k_block: torch.Tensor, v_block: torch.Tensor, first_slot: int):
    """Fill token slots >= first_slot of one block (both planes) with NaN."""
    if first_slot < BLOCK_SIZE:
        k_block[:, :, first_slot:, :] = float("nan")
        v_block[:, :, first_slot:] = float("nan")
