"""Drafter shapes and workload descriptions.

Plain data only: no arithmetic of the drafter lives here.  The five named
workloads follow the paper's target families (Vicuna-13B, LLaMA-3.x 8B and
70B; experimental setup of Section 3) at the drafter sizes a FastEagle
cascade for those targets has: hidden width, head layout and MLP width of
the target, N cascade layers (Section 2.1, Eq. 1-2), a draft vocabulary and
a top-k per level for the Backbone Expansion tree (Section 2.2).
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple


@dataclasses.dataclass(frozen=True)
class DrafterConfig:
    name: str
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    intermediate: int
    n_layers: int              # N, cascade depth
    draft_vocab: int           # V
    target_vocab: int          # V_t (embedding table rows, id space of d2t)
    rope_theta: float
    dtype: str                 # "f32" or "bf16": storage of weights, features, KV
    batch: int
    prefix: object             # int (every sequence) or (lo, hi) inclusive range
    topk: int
    rms_eps: float = 1e-5
    cascade_ctx: str = "cascade"   # "cascade", "self" or "parallel" (parallel heads)
    n_feat_levels: int = 3

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def tree_nodes(self) -> int:
        return 1 + self.n_layers * self.topk

    @property
    def n_leaves(self) -> int:
        return self.n_layers * (self.topk - 1) + 1

    def with_(self, **kw) -> "DrafterConfig":
        return dataclasses.replace(self, **kw)

    def weight_bytes(self) -> int:
        """Bytes of every weight matrix the pass reads once (embedding: one row per sequence)."""
        es = 2 if self.dtype == "bf16" else 4
        d, I = self.hidden, self.intermediate
        qd, kvd = self.n_q_heads * self.head_dim, self.n_kv_heads * self.head_dim
        per_layer = (qd * d + 2 * kvd * d + d * qd + 3 * I * d + 2 * d) * es
        return ((3 * d * d + 2 * d * d) * es + self.n_layers * per_layer
                + (self.draft_vocab * d + d) * es)


TINY_F32_B1 = DrafterConfig(
    name="tiny_fp32_b1", hidden=256, n_q_heads=4, n_kv_heads=4, head_dim=64,
    intermediate=704, n_layers=2, draft_vocab=1024, target_vocab=1024,
    rope_theta=10000.0, dtype="f32", batch=1, prefix=64, topk=4)

LLAMA8B_BF16_B1 = DrafterConfig(
    name="llama8b_bf16_b1", hidden=4096, n_q_heads=32, n_kv_heads=8, head_dim=128,
    intermediate=14336, n_layers=5, draft_vocab=32000, target_vocab=128256,
    rope_theta=500000.0, dtype="bf16", batch=1, prefix=1024, topk=8)

VICUNA13B_BF16_B1 = DrafterConfig(
    name="vicuna13b_bf16_b1", hidden=5120, n_q_heads=40, n_kv_heads=40, head_dim=128,
    intermediate=13824, n_layers=6, draft_vocab=32000, target_vocab=32000,
    rope_theta=10000.0, dtype="bf16", batch=1, prefix=2048, topk=8)

LLAMA70B_BF16_B1 = DrafterConfig(
    name="llama70b_bf16_b1", hidden=8192, n_q_heads=64, n_kv_heads=8, head_dim=128,
    intermediate=28672, n_layers=5, draft_vocab=32000, target_vocab=128256,
    rope_theta=500000.0, dtype="bf16", batch=1, prefix=4096, topk=10)

LLAMA8B_BF16_B32 = LLAMA8B_BF16_B1.with_(
    name="llama8b_bf16_b32", batch=32, prefix=(256, 8192), n_layers=7, topk=8)

NAMED = {c.name: c for c in (TINY_F32_B1, LLAMA8B_BF16_B1, VICUNA13B_BF16_B1,
                             LLAMA70B_BF16_B1, LLAMA8B_BF16_B32)}

# Small shapes that still span several GEMM tiles, ragged attention chunks and
# ragged batches; the oracle finishes them in well under a second.
SMALL_GQA_BF16 = DrafterConfig(
    name="small_gqa_bf16_b3", hidden=512, n_q_heads=8, n_kv_heads=2, head_dim=64,
    intermediate=1376, n_layers=3, draft_vocab=2000, target_vocab=5003,
    rope_theta=500000.0, dtype="bf16", batch=3, prefix=(0, 700), topk=5)

SMALL_GQA_F32 = SMALL_GQA_BF16.with_(name="small_gqa_f32_b3", dtype="f32")

SMALL_MHA_BF16_D128 = DrafterConfig(
    name="small_mha_bf16_d128", hidden=384, n_q_heads=3, n_kv_heads=3, head_dim=128,
    intermediate=1024, n_layers=4, draft_vocab=1040, target_vocab=1040,
    rope_theta=10000.0, dtype="bf16", batch=2, prefix=(1, 300), topk=3)


# Grouped-query layouts the small shapes above do not reach: 8 query heads per
# KV head (the 70B-shaped grouping, head dim 128) and 2 per KV head.
SMALL_GQA8_BF16_D128 = DrafterConfig(
    name="small_gqa8_bf16_d128", hidden=512, n_q_heads=16, n_kv_heads=2, head_dim=128,
    intermediate=1088, n_layers=3, draft_vocab=1504, target_vocab=3001,
    rope_theta=500000.0, dtype="bf16", batch=3, prefix=(0, 700), topk=4)

SMALL_GQA2_BF16 = DrafterConfig(
    name="small_gqa2_bf16", hidden=256, n_q_heads=8, n_kv_heads=4, head_dim=64,
    intermediate=704, n_layers=3, draft_vocab=1024, target_vocab=2048,
    rope_theta=10000.0, dtype="bf16", batch=2, prefix=(1, 400), topk=4)

SMALL_GQA2_F32 = SMALL_GQA2_BF16.with_(name="small_gqa2_f32", dtype="f32")


# Batch-1 shapes whose widths are multiples of 512 (d, 3d, 2d, H_q * D, I), as
# the persistent batch-1 pass needs: GQA with head dim 64, 8 query heads per KV
# head with head dim 128, and multi-head attention with head dim 128 and the
# deepest cascade the persistent pass takes (8 layers).
SMALL_PASS_GQA = DrafterConfig(
    name="small_pass_gqa", hidden=512, n_q_heads=8, n_kv_heads=2, head_dim=64,
    intermediate=1536, n_layers=3, draft_vocab=2000, target_vocab=5003,
    rope_theta=500000.0, dtype="bf16", batch=1, prefix=700, topk=5)

SMALL_PASS_GQA8 = DrafterConfig(
    name="small_pass_gqa8", hidden=1024, n_q_heads=16, n_kv_heads=2, head_dim=128,
    intermediate=2048, n_layers=4, draft_vocab=3008, target_vocab=7001,
    rope_theta=500000.0, dtype="bf16", batch=1, prefix=300, topk=8)

SMALL_PASS_MHA_N8 = DrafterConfig(
    name="small_pass_mha_n8", hidden=1024, n_q_heads=8, n_kv_heads=8, head_dim=128,
    intermediate=2560, n_layers=8, draft_vocab=1504, target_vocab=1504,
    rope_theta=10000.0, dtype="bf16", batch=1, prefix=129, topk=3)


def prefix_range(cfg: DrafterConfig) -> Tuple[int, int]:
    if isinstance(cfg.prefix, int):
        return cfg.prefix, cfg.prefix
    lo, hi = cfg.prefix
    return int(lo), int(hi)
