"""Seeded synthetic inputs for the encoder-stage workloads.

This module is shared by the tests, the smoke check and the benchmark.  It
draws random numbers and rounds them to the storage type of a stage; it holds
none of the encoder layer's arithmetic.  Both the CPU oracle and the HIP
library receive exactly the arrays produced here.

Workload shapes follow the paper's BERT experiments (§VI-B: 16 heads,
batch 32) with hidden size, FFN width, sequence length and padding
distribution fixed by the five stage presets below.  The paper trains on MNLI;
no dataset is used here: the synthetic tensors only stand in for its shapes.

Random draws use numpy's PCG64 (``numpy.random.default_rng(seed)``):
  * weights ~ N(0, 0.02), biases 0, LayerNorm gamma 1 and beta 0;
  * x ~ N(0, 1) of shape [B, S, h], dy ~ N(0, 1) of the same shape;
  * per-sequence valid lengths uniform over the integers [lo, hi];
    key positions at or past the length are masked.
``perturb=True`` replaces the zero biases / unit gammas by random values so
that a dropped bias or a swapped gamma/beta cannot hide behind the default
initialisation.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

# Parameter order of one encoder layer (row-major, torch Linear layout
# [out_features, in_features] for the matrices).
PARAM_NAMES = ("W_qkv", "b_qkv", "W_o", "b_o", "g1", "be1",
               "W_1", "b_1", "W_2", "b_2", "g2", "be2")


def param_shapes(h: int, f: int) -> Dict[str, tuple]:
    return {
        "W_qkv": (3 * h, h), "b_qkv": (3 * h,),
        "W_o": (h, h), "b_o": (h,),
        "g1": (h,), "be1": (h,),
        "W_1": (f, h), "b_1": (f,),
        "W_2": (h, f), "b_2": (h,),
        "g2": (h,), "be2": (h,),
    }


MATRICES = ("W_qkv", "W_o", "W_1", "W_2")


@dataclasses.dataclass(frozen=True)
class StageConfig:
    name: str
    L: int
    hidden: int
    heads: int
    ffn: int
    batch: int
    seq: int
    len_lo: Optional[int]  # None: no padding (every length == seq)
    len_hi: Optional[int]
    dtype: str  # "f32" or "bf16"
    seed: int

    @property
    def tokens(self) -> int:
        return self.batch * self.seq

    def with_(self, **kw) -> "StageConfig":
        return dataclasses.replace(self, **kw)


CONFIGS: Dict[str, StageConfig] = {
    # 2 layers, h128/2 heads/f512, B2 x S32, lengths in [16, 32], fp32.
    "tiny": StageConfig("tiny", 2, 128, 2, 512, 2, 32, 16, 32, "f32", 0),
    # 3 layers of a BERT-base-shaped model, B16 x S128, lengths in [64, 128].
    "bert_base_3": StageConfig("bert_base_3", 3, 768, 12, 3072, 16, 128, 64, 128, "bf16", 1),
    # 8 layers (the larger share of a faster device), B32 x S512, lengths in [256, 512].
    "bert_base_8_uneven": StageConfig("bert_base_8_uneven", 8, 768, 12, 3072, 32, 512, 256, 512, "bf16", 2),
    # 4 BERT-large-shaped layers, B32 x S512, no padding.
    "bert_large_4": StageConfig("bert_large_4", 4, 1024, 16, 4096, 32, 512, None, None, "bf16", 3),
    # Depth sweep at B8 x S512, lengths in [128, 512]; L is set per run.
    "deep_sweep": StageConfig("deep_sweep", 1, 1024, 16, 4096, 8, 512, 128, 512, "bf16", 4),
}

DEEP_SWEEP_DEPTHS = (1, 5, 10, 20, 40)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 (ties to even); returned as float32."""
    a32 = np.ascontiguousarray(a, dtype=np.float32)
    u = a32.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32)
    # NaN stays NaN (never produced by the generators here).
    return np.where(np.isnan(a32), a32, out)


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) of values that are already bf16-exact."""
    a32 = np.ascontiguousarray(a, dtype=np.float32)
    return (a32.view(np.uint32) >> 16).astype(np.uint16)


def from_bf16_bits(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def round_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    """Round to the stage storage type; the result is float64 and exact."""
    if dtype == "bf16":
        return round_bf16(a).astype(np.float64)
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    raise ValueError(dtype)


def make_lengths(cfg: StageConfig, rng: np.random.Generator) -> np.ndarray:
    if cfg.len_lo is None:
        return np.full(cfg.batch, cfg.seq, dtype=np.int64)
    return rng.integers(cfg.len_lo, cfg.len_hi, size=cfg.batch, endpoint=True).astype(np.int64)


def key_mask(lengths: np.ndarray, seq: int) -> np.ndarray:
    """[B, S] uint8, 1 where key position s < length (attend), 0 past it."""
    return (np.arange(seq)[None, :] < np.asarray(lengths)[:, None]).astype(np.uint8)


def make_inputs(cfg: StageConfig, seed: Optional[int] = None) -> Dict[str, np.ndarray]:
    """x, dy (float64 holding storage-exact values), lengths and key mask."""
    rng = np.random.default_rng(cfg.seed if seed is None else seed)
    B, S, h = cfg.batch, cfg.seq, cfg.hidden
    lengths = make_lengths(cfg, rng)
    x = round_storage(rng.standard_normal((B, S, h), dtype=np.float32), cfg.dtype)
    dy = round_storage(rng.standard_normal((B, S, h), dtype=np.float32), cfg.dtype)
    return {"x": x, "dy": dy, "lengths": lengths, "mask": key_mask(lengths, S)}


def make_params(cfg: StageConfig, seed: Optional[int] = None,
                perturb: bool = False) -> List[Dict[str, np.ndarray]]:
    """Per-layer parameters as float64 arrays holding storage-exact values.

    Matrices are rounded to the stage dtype; biases, gammas and betas are
    float32 on both paths."""
    rng = np.random.default_rng((cfg.seed if seed is None else seed) + 7919)
    shapes = param_shapes(cfg.hidden, cfg.ffn)
    layers = []
    for _ in range(cfg.L):
        p = {}
        for name in PARAM_NAMES:
            shp = shapes[name]
            if name in MATRICES:
                v = round_storage(0.02 * rng.standard_normal(shp, dtype=np.float32), cfg.dtype)
            elif name.startswith("g"):
                v = np.ones(shp) if not perturb else \
                    1.0 + 0.25 * rng.standard_normal(shp, dtype=np.float32)
            else:
                v = np.zeros(shp) if not perturb else \
                    0.25 * rng.standard_normal(shp, dtype=np.float32)
            p[name] = np.asarray(v, dtype=np.float32).astype(np.float64) \
                if name not in MATRICES else v
        layers.append(p)
    return layers


def flops_per_step(cfg: StageConfig, lengths: Optional[np.ndarray] = None) -> float:
    """Algorithmic fwd+bwd FLOPs of one stage step.

    Per token per layer: 3 * [2 * (4 h^2 + 2 h f) + 4 h S_k], S_k the number of
    valid keys of the token's sequence; the factor 3 counts the forward pass
    plus the two backward contractions of every product."""
    h, f = cfg.hidden, cfg.ffn
    if lengths is None:
        keys = np.full(cfg.batch, cfg.seq, dtype=np.float64)
    else:
        keys = np.asarray(lengths, dtype=np.float64)
    per_seq = cfg.seq * 3.0 * (2.0 * (4 * h * h + 2 * h * f) + 4.0 * h * keys)
    return float(per_seq.sum() * cfg.L)
