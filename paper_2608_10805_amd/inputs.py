"""Seeded synthetic inputs for WTConv tests and benchmarks.

This module only draws random numbers and rounds them to a storage type; it
holds none of the operator's arithmetic, so both the GPU path's tests and the
CPU oracle can take their inputs from it.

Recipe (the same for every workload):
  * numpy.random.default_rng(seed), draws in this order:
      x ~ N(0, 1)                [B, C, H, W]
      base_w ~ U(-0.2, 0.2)      [C, k, k]
      base_scale ~ U(0.5, 1.5)   [C]
      for l = 1..L:
        level_w[l] ~ U(-0.2, 0.2)      [4C, k, k]
        level_scale[l] ~ U(0.05, 0.2)  [4C]
      dy ~ N(0, 1)               [B, C, H, W]   (only when requested)
  * float64 draws are rounded to float32 (round to nearest even); the
    activations x and dy are then rounded to the storage dtype (bf16 / fp16,
    round to nearest even). Parameters stay float32.
  * Every array is returned as float32 holding exactly the values the GPU
    receives, so the float64 oracle can be fed the same numbers.
"""
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returned as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32)
    nan = np.isnan(a)
    if nan.any():
        out = out.copy()
        out[nan] = np.nan
    return out


def round_to_fp16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest IEEE half (ties to even); returned as float32."""
    return np.asarray(a, dtype=np.float32).astype(np.float16).astype(np.float32)


def round_to(a: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32)
    if dtype == "bf16":
        return round_to_bf16(a)
    if dtype == "f16":
        return round_to_fp16(a)
    raise ValueError(f"unknown dtype {dtype!r}")


@dataclass
class Workload:
    """One operator configuration: shape, kernel size, levels and storage dtype."""
    name: str
    B: int
    C: int
    H: int
    W: int
    k: int = 5
    L: int = 1
    dtype: str = "f32"
    backward: bool = False

    @property
    def N(self) -> int:
        return self.B * self.C * self.H * self.W


@dataclass
class Inputs:
    x: np.ndarray
    base_w: np.ndarray
    base_scale: np.ndarray
    level_w: List[np.ndarray] = field(default_factory=list)
    level_scale: List[np.ndarray] = field(default_factory=list)
    dy: Optional[np.ndarray] = None


def make_inputs(B: int, C: int, H: int, W: int, k: int, L: int, dtype: str = "f32",
                seed: int = 0, with_dy: bool = True) -> Inputs:
    """Draw one seeded input set following the recipe in the module docstring."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((B, C, H, W))
    base_w = rng.uniform(-0.2, 0.2, (C, k, k))
    base_scale = rng.uniform(0.5, 1.5, (C,))
    level_w, level_scale = [], []
    for _ in range(L):
        level_w.append(rng.uniform(-0.2, 0.2, (4 * C, k, k)).astype(np.float32))
        level_scale.append(rng.uniform(0.05, 0.2, (4 * C,)).astype(np.float32))
    dy = rng.standard_normal((B, C, H, W)) if with_dy else None
    return Inputs(
        x=round_to(x.astype(np.float32), dtype),
        base_w=base_w.astype(np.float32),
        base_scale=base_scale.astype(np.float32),
        level_w=level_w,
        level_scale=level_scale,
        dy=None if dy is None else round_to(dy.astype(np.float32), dtype),
    )


def make_bias(C: int, seed: int = 0) -> np.ndarray:
    """Seeded base bias for runs that use one (the benchmark workloads have none):
    numpy.random.default_rng([seed, 1]), b0 ~ U(-0.5, 0.5) [C], rounded to float32."""
    return np.random.default_rng([seed, 1]).uniform(-0.5, 0.5, (C,)).astype(np.float32)


# Named workloads. ConvNeXt-T stage shapes follow from 224x224 inputs
# (56, 28, 14, 7 pixels at C = 96, 192, 384, 768).
WORKLOADS: Dict[str, Workload] = {
    "small_b2_c16_32_k5_l1": Workload("small_b2_c16_32_k5_l1", 2, 16, 32, 32, 5, 1, "f32", False),
    "convnext_s1_b64_c96_56_k5_l3": Workload("convnext_s1_b64_c96_56_k5_l3", 64, 96, 56, 56, 5, 3, "f32", True),
    "convnext_s2_b64_c192_28_k5": Workload("convnext_s2_b64_c192_28_k5", 64, 192, 28, 28, 5, 1, "f32", True),
    "convnext_s1_b128_c96_56_k5_l5_bf16": Workload("convnext_s1_b128_c96_56_k5_l5_bf16", 128, 96, 56, 56, 5, 5,
                                                   "bf16", True),
}


def sweep_shapes():
    """(B, C, H, W) shapes of the fwd+bwd sweep: ConvNeXt-T stages at B=128, an odd
    non-square shape and a large-plane shape."""
    return [(128, 96, 56, 56), (128, 192, 28, 28), (128, 384, 14, 14), (128, 768, 7, 7),
            (32, 128, 63, 95), (16, 64, 224, 224)]
