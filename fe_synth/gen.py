"""Seeded synthetic inputs for the drafter.

Both the GPU path and the CPU oracle consume the very same host arrays made
here; this module holds none of the drafter's arithmetic.

Definition of the streams (so that any consumer can regenerate them):
  * every tensor has a name; a float tensor of n elements is cut into blocks of
    BLOCK = 2**22 elements, and block j is drawn with
    numpy.random.Generator(PCG64(SeedSequence([seed, crc32(name), j]))).standard_normal(float32);
  * the block is scaled (and shifted) in float32: weights, embedding and LM
    head use 0.02*z, RMSNorm gains 1 + 0.02*z, features and prefix K/V use z;
  * bf16 storage rounds that float32 value to nearest-even bf16 and keeps the
    16-bit pattern (numpy uint16);
  * integer draws use one Generator(PCG64(SeedSequence([seed, crc32(name)]))).

Distributions stand in for the paper's benchmarks (MT-Bench, HumanEval, GSM8K,
Alpaca, CNN/DM and the ShareGPT/UltraChat training data), none of which a
drafter pass needs: only shapes, lengths and value scales matter here.
"""
from __future__ import annotations

import dataclasses
import os
import zlib
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional

import numpy as np

from .configs import DrafterConfig, prefix_range

BLOCK = 1 << 22


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _ss(seed: int, name: str, *extra: int) -> np.random.SeedSequence:
    return np.random.SeedSequence([int(seed), zlib.crc32(name.encode()), *extra])


def float_tensor(name: str, shape, seed: int, dtype: str, scale: float = 1.0,
                 shift: float = 0.0) -> np.ndarray:
    """shift + scale * N(0,1), drawn block-wise in float32; bf16 -> uint16 bit patterns."""
    shape = tuple(int(s) for s in shape)
    n = int(np.prod(shape)) if shape else 1
    out = np.empty(n, dtype=np.uint16 if dtype == "bf16" else np.float32)
    sc, sh = np.float32(scale), np.float32(shift)

    def fill(j: int) -> None:
        lo, hi = j * BLOCK, min(n, (j + 1) * BLOCK)
        rng = np.random.Generator(np.random.PCG64(_ss(seed, name, j)))
        z = rng.standard_normal(hi - lo, dtype=np.float32)
        if scale != 1.0:
            z *= sc
        if shift != 0.0:
            z += sh
        if dtype == "bf16":
            b = z.view(np.uint32)
            b += np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
            b >>= np.uint32(16)
            out[lo:hi] = b
        else:
            out[lo:hi] = z

    nblk = (n + BLOCK - 1) // BLOCK
    if nblk <= 1:
        for j in range(nblk):
            fill(j)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(nblk)))
    return out.reshape(shape)


def int_rng(name: str, seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(_ss(seed, name)))


@dataclasses.dataclass
class LayerWeights:
    attn_norm: np.ndarray
    wq: np.ndarray
    wk: np.ndarray
    wv: np.ndarray
    wo: np.ndarray
    mlp_norm: np.ndarray
    w_gate: np.ndarray
    w_up: np.ndarray
    w_down: np.ndarray

    FIELDS = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")


@dataclasses.dataclass
class Weights:
    w_fuse: np.ndarray      # [d, 3d]
    w_in: np.ndarray        # [d, 2d]
    embed: np.ndarray       # [V_t, d]
    final_norm: np.ndarray  # [d]
    lm_head: np.ndarray     # [V, d]
    d2t: np.ndarray         # int32 [V], draft id -> target id
    layers: List[LayerWeights]


@dataclasses.dataclass
class Inputs:
    features: np.ndarray      # [B, 3d]: l_t, m_t, h_t of the target
    next_tokens: np.ndarray   # int32 [B]: token t+1 (target vocabulary)
    prefix_lens: np.ndarray   # int32 [B]
    kcache: List[np.ndarray]  # per layer [sum P_b, H_kv, D], already rotated
    vcache: List[np.ndarray]  # per layer [sum P_b, H_kv, D]

    @property
    def cu_prefix(self) -> np.ndarray:
        cu = np.zeros(len(self.prefix_lens) + 1, dtype=np.int32)
        cu[1:] = np.cumsum(self.prefix_lens)
        return cu


def make_weights(cfg: DrafterConfig, seed: int = 0) -> Weights:
    d, I, D = cfg.hidden, cfg.intermediate, cfg.head_dim
    qd, kvd = cfg.n_q_heads * D, cfg.n_kv_heads * D
    dt = cfg.dtype

    def lin(name, shape):
        return float_tensor(name, shape, seed, dt, scale=0.02)

    def gain(name):
        return float_tensor(name, (d,), seed, dt, scale=0.02, shift=1.0)

    layers = []
    for i in range(cfg.n_layers):
        p = f"layer{i}."
        layers.append(LayerWeights(
            attn_norm=gain(p + "attn_norm"), wq=lin(p + "wq", (qd, d)),
            wk=lin(p + "wk", (kvd, d)), wv=lin(p + "wv", (kvd, d)),
            wo=lin(p + "wo", (d, qd)), mlp_norm=gain(p + "mlp_norm"),
            w_gate=lin(p + "w_gate", (I, d)), w_up=lin(p + "w_up", (I, d)),
            w_down=lin(p + "w_down", (d, I))))
    if cfg.draft_vocab == cfg.target_vocab:
        d2t = np.arange(cfg.draft_vocab, dtype=np.int32)
    else:
        rng = int_rng("d2t", seed)
        d2t = np.sort(rng.choice(cfg.target_vocab, size=cfg.draft_vocab,
                                 replace=False)).astype(np.int32)
    return Weights(
        w_fuse=lin("w_fuse", (d, cfg.n_feat_levels * d)), w_in=lin("w_in", (d, 2 * d)),
        embed=lin("embed", (cfg.target_vocab, d)), final_norm=gain("final_norm"),
        lm_head=lin("lm_head", (cfg.draft_vocab, d)), d2t=d2t, layers=layers)


def make_prefix_lens(cfg: DrafterConfig, seed: int = 0) -> np.ndarray:
    lo, hi = prefix_range(cfg)
    if lo == hi:
        return np.full(cfg.batch, lo, dtype=np.int32)
    return int_rng("prefix_lens", seed).integers(lo, hi + 1, size=cfg.batch).astype(np.int32)


def make_inputs(cfg: DrafterConfig, seed: int = 0,
                prefix_lens: Optional[np.ndarray] = None) -> Inputs:
    B = cfg.batch
    if prefix_lens is None:
        prefix_lens = make_prefix_lens(cfg, seed)
    prefix_lens = np.asarray(prefix_lens, dtype=np.int32)
    total = int(prefix_lens.sum())
    kv_shape = (total, cfg.n_kv_heads, cfg.head_dim)
    kc = [float_tensor(f"layer{i}.kcache", kv_shape, seed, cfg.dtype) for i in range(cfg.n_layers)]
    vc = [float_tensor(f"layer{i}.vcache", kv_shape, seed, cfg.dtype) for i in range(cfg.n_layers)]
    feats = float_tensor("features", (B, cfg.n_feat_levels * cfg.hidden), seed, cfg.dtype)
    toks = int_rng("next_tokens", seed).integers(0, cfg.target_vocab, size=B).astype(np.int32)
    return Inputs(features=feats, next_tokens=toks, prefix_lens=prefix_lens, kcache=kc, vcache=vc)


def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of stored values (bf16 bit patterns or float32) to float64."""
    if dtype == "bf16":
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


@dataclasses.dataclass
class UpdateRows:
    """Verified positions whose drafter-cache rows are to be written: row m has
    the target's features at position positions[m], the token after it, and
    the cache row dst_rows[m] it goes to (caches of cache_rows rows)."""
    features: np.ndarray   # [M, 3d]
    tokens: np.ndarray     # int32 [M]
    positions: np.ndarray  # int32 [M]
    dst_rows: np.ndarray   # int32 [M]
    cache_rows: int


def make_update_rows(cfg: DrafterConfig, accepted: np.ndarray, prefix_lens: np.ndarray,
                     capacity: int, seed: int = 0) -> UpdateRows:
    """Sequence b appends accepted[b] positions P_b .. P_b + accepted[b] - 1 to
    its cache, which owns rows b*capacity .. (b+1)*capacity - 1 (row = position)."""
    accepted = np.asarray(accepted, dtype=np.int32)
    prefix_lens = np.asarray(prefix_lens, dtype=np.int32)
    assert np.all(prefix_lens + accepted <= capacity)
    b_of = np.repeat(np.arange(len(accepted), dtype=np.int64), accepted)
    j = np.concatenate([np.arange(a, dtype=np.int64) for a in accepted]) if len(accepted) else \
        np.zeros(0, np.int64)
    pos = (prefix_lens[b_of] + j).astype(np.int32)
    dst = (b_of * capacity + pos).astype(np.int32)
    M = len(pos)
    feats = float_tensor("update.features", (M, cfg.n_feat_levels * cfg.hidden), seed, cfg.dtype)
    toks = int_rng("update.tokens", seed).integers(0, cfg.target_vocab, size=M).astype(np.int32)
    return UpdateRows(features=feats, tokens=toks, positions=pos, dst_rows=dst,
                      cache_rows=int(len(accepted) * capacity))


def make_uniforms(shape, seed: int = 0, name: str = "uniforms") -> np.ndarray:
    """float32 uniforms in the open interval (0, 1): (j + 0.5) / 2^23 for a
    23-bit integer j drawn uniformly, exact in float32 (the noise of
    stochastic drafting; the extremes are 2^-24 and 1 - 2^-24)."""
    rng = int_rng(name, seed)
    j = rng.integers(0, 1 << 23, size=tuple(int(s) for s in shape), dtype=np.int64)
    return ((j.astype(np.float64) + 0.5) / float(1 << 23)).astype(np.float32)
