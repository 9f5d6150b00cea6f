"""Seeded synthetic weight tensors shaped like the paper's workloads.

This module only draws random numbers and casts them to BF16 bit patterns; it
holds none of EntroPack's arithmetic, so both the oracle-side tests and the
GPU-side benchmark can use it.  The paper's model weights (Z-Image-Turbo,
Qwen3.8-27B, MiniMax-H3; Section 4.1) are not available; these tensors stand
in for them with the shapes of a 27B-class LLM MLP and of a
diffusion-transformer block stack whose MLP shape equals the paper's reference
layer (10240 x 3840, Appendix A evaluation details).

Recipe per tensor, in draw order from one ``numpy.random.Generator`` (PCG64):
  1. row standard deviations ``sigma_r = exp(mu + s * N(0,1))`` (R draws);
  2. the R x C body, Gaussian or Student-t(5) scaled to unit variance, times
     ``sigma_r``;
  3. outlier positions ``rng.choice(N, k, replace=False)`` with
     ``k = round(rate * N)``, multiplied by a factor;
  4. float64 -> float32 (round to nearest even) -> BF16 (round to nearest
     even), returned as uint16 bit patterns.
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to BF16 (nearest, ties to even); return uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass(frozen=True)
class TensorSpec:
    name: str
    rows: int
    cols: int


def draw_tensor(rng: np.random.Generator, rows: int, cols: int, *, body: str,
                log_mu: float, log_sigma: float, outlier_rate: float = 0.0,
                outlier_factor: float = 1.0) -> np.ndarray:
    """One BF16 weight matrix (uint16 bits, shape rows x cols)."""
    sig = np.exp(log_mu + log_sigma * rng.standard_normal(rows))
    if body == "gauss":
        w = rng.standard_normal((rows, cols))
    elif body == "t5":
        w = rng.standard_t(5, size=(rows, cols)) / math.sqrt(5.0 / 3.0)
    else:
        raise ValueError(body)
    w *= sig[:, None]
    n = rows * cols
    k = int(round(outlier_rate * n))
    if k:
        pos = rng.choice(n, size=k, replace=False)
        w.reshape(-1)[pos] *= outlier_factor
    return f32_to_bf16_bits(w.astype(np.float32))


# ---- the five workloads -------------------------------------------------------

CFG1 = dict(body="gauss", log_mu=math.log(0.02), log_sigma=0.5, outlier_rate=0.001,
            outlier_factor=10.0)
CFG2 = dict(body="t5", log_mu=math.log(0.015), log_sigma=0.4)
CFG3 = dict(body="gauss", log_mu=math.log(0.01), log_sigma=0.5, outlier_rate=0.0005,
            outlier_factor=8.0)

DIT_SHAPES = [("q", 3840, 3840), ("k", 3840, 3840), ("v", 3840, 3840), ("o", 3840, 3840),
              ("mlp_in", 10240, 3840), ("mlp_out", 3840, 10240)]
LLM_SHAPES = [("gate", 17408, 5120), ("up", 17408, 5120), ("down", 5120, 17408)]


def single_linear() -> np.ndarray:
    """256 x 512 BF16, Gaussian rows with lognormal(ln 0.02, 0.5) std, 0.1 % x10 outliers, seed 0."""
    return draw_tensor(np.random.default_rng(0), 256, 512, **CFG1)


def attention_projection() -> np.ndarray:
    """3072 x 3072 BF16, Student-t(5) rows with lognormal(ln 0.015, 0.4) std, seed 1."""
    return draw_tensor(np.random.default_rng(1), 3072, 3072, **CFG2)


def llm_mlp(names=("gate", "up", "down")) -> dict:
    """27B-class MLP: gate/up 17408 x 5120, down 5120 x 17408, seed 2 (drawn in that order)."""
    rng = np.random.default_rng(2)
    out = {}
    for name, r, c in LLM_SHAPES:
        w = draw_tensor(rng, r, c, **CFG3)
        if name in names:
            out[name] = w
        if all(n in out for n in names):
            break
    return out


def llm_activations() -> np.ndarray:
    """INT8 activations 8192 x 17408, uniform on [-127, 127], seed 3."""
    return np.random.default_rng(3).integers(-127, 128, (8192, 17408), dtype=np.int8)


def dit_block(b: int) -> list:
    """Block b of the 30-block diffusion-transformer stack: [(name, bits)] in layer order."""
    rng = np.random.default_rng([4, b])
    return [(f"blocks.{b}.{name}", draw_tensor(rng, r, c, **CFG2)) for name, r, c in DIT_SHAPES]


def dit_stack(n_blocks: int = 30, workers: int = 8) -> list:
    """All layers of the first n_blocks blocks, in order (blocks drawn in parallel threads)."""
    with ThreadPoolExecutor(max_workers=max(1, workers)) as ex:
        blocks = list(ex.map(dit_block, range(n_blocks)))
    return [layer for blk in blocks for layer in blk]


def ragged_tensor(seed: int, rows: int, cols: int, scale: float = 0.02) -> np.ndarray:
    """Small Gaussian BF16 tensor of arbitrary shape for edge-case tests."""
    return draw_tensor(np.random.default_rng(seed), rows, cols, body="gauss",
                       log_mu=math.log(scale), log_sigma=0.3)
