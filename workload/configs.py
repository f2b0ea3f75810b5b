"""Named synthetic verification-round workloads.

Each workload is one target-worker verification round on a reconstructed batch
(Algorithm 1, Section 4): a batch of requests, some of which arrive from
another worker and must have their KV state prepared first (Prepare in
Algorithm 1; HostKV extents, Appendix E.1), then verification of an anchor
token plus K proposal tokens per request (Section 6 setup; Appendix G.2 counts
the target workload as anchor-plus-proposal tokens; Appendix H: post-prefill
requests with an initial anchor token, depth d).  Head geometry follows the
target model family the paper evaluates (Qwen3-8B: 32 query heads, 8 KV heads,
head dimension 128, 36 layers, vocabulary 151936; Qwen3-0.6B: 16/8 heads).
"""
from dataclasses import dataclass, replace
from typing import Optional


@dataclass(frozen=True)
class RoundConfig:
    name: str
    seed: int
    bs: int                 # requests in the reconstructed batch
    num_layers: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    ctx_lo: int             # context length L_r ~ integer-uniform [ctx_lo, ctx_hi]
    ctx_hi: int
    k_lo: int               # proposal depth K_r ~ integer-uniform [k_lo, k_hi]
    k_hi: int
    n_arriving: int         # requests whose KV must be gathered from the staging pool
    vocab: int              # 0: no acceptance step in this round
    pool_blocks: Optional[int] = None   # None: pool sized to exactly hold the batch
    staging_order: str = "extent"       # "extent" (per-request contiguous) or "shuffled"
    block_size: int = 16

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads


CONFIGS = {
    # 4 requests, 1 layer, 4q/2kv heads, D=64, L in [64,256], 64-block pool,
    # K=4, vocab 1000, 2 arriving requests.
    "tiny": RoundConfig("tiny", 0, 4, 1, 4, 2, 64, 64, 256, 4, 4, 2, 1000, pool_blocks=64),
    # draft-side decode shape: bs=512, 16q/8kv, D=128, L in [512,2048], K=0,
    # no acceptance, 25% arriving.
    "draft_decode": RoundConfig("draft_decode", 1, 512, 1, 16, 8, 128, 512, 2048, 0, 0, 128, 0),
    # 8B-shaped verify round: bs=256, 32q/8kv, D=128, L in [1024,4096], K=4,
    # 30% arriving, vocab 151936.
    "verify_8b": RoundConfig("verify_8b", 2, 256, 1, 32, 8, 128, 1024, 4096, 4, 4, 77, 151936),
    # large batch at the latency knee: bs=512, L in [2048,8192], K=6, 50% arriving.
    "knee": RoundConfig("knee", 3, 512, 1, 32, 8, 128, 2048, 8192, 6, 6, 256, 151936),
    # full-depth ragged round: 36 layers, bs=128, L in [16384,32768],
    # K in [1,8] per request, 40% arriving (all 36 layers gathered).
    "full_depth": RoundConfig("full_depth", 4, 128, 36, 32, 8, 128, 16384, 32768, 1, 8, 51,
                              151936),
}


def custom_config(**kw) -> RoundConfig:
    """A small ad-hoc workload for property tests (defaults: the tiny round)."""
    base = CONFIGS["tiny"]
    kw.setdefault("name", "custom")
    return replace(base, **kw)
