"""Seeded synthetic verification-round workloads.

This package only draws inputs: context lengths, draft lengths, the arriving
set, physical block permutations, bf16 query/key/value tensors, fp32 target
and draft probability rows, draft tokens and uniforms (and the per-step
inputs of a draft stage), and lays the key/value
tensors out in the paged-pool byte format (and, for the host-side
preparation, in a pinned host arena).  It performs none of the round's own
arithmetic (no gather, attention or acceptance) and is the only code that both
the GPU path's tests and the CPU oracle consume.
"""
from .configs import CONFIGS, RoundConfig, custom_config
from .layout import (k_block_shape, v_block_shape, logical_kv_from_blocks,
                     BLOCK_SIZE, K_VEC)
from .synth import (RoundMeta, LayerData, AcceptData, HostKV, DraftData, make_meta, make_layer,
                    make_accept, make_hostkv, make_draft)

__all__ = ["CONFIGS", "RoundConfig", "custom_config", "k_block_shape", "v_block_shape",
           "logical_kv_from_blocks", "BLOCK_SIZE", "K_VEC", "RoundMeta", "LayerData",
           "AcceptData", "HostKV", "DraftData", "make_meta", "make_layer", "make_accept",
           "make_hostkv", "make_draft"]
