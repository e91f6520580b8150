"""Seeded synthetic workloads for the sparse SwiGLU FFN decode step.

This module only draws random numbers and casts them to the model dtype. It
holds none of the method's arithmetic (no quantisation, selection or FFN
math), so both the HIP path's tests/bench and the CPU oracle can take their
inputs from here without sharing any computation.

Shapes and value distributions stand in for the paper's decode workloads:
the paper measures real checkpoints (Qwen3-8B FFN is 4096 x 12288, Sec. 5 and
App. A.5) that are not available here, so the weights are i.i.d. Gaussian and
the FFN inputs heavy-tailed (Laplace with outlier channels, or Student-t), in
line with the Gaussian-to-Laplacian activation shapes the paper reports in
App. A.2.

Layout: every weight matrix is produced channel-major, ``[d_ff][d_model]``
row-major, i.e. ``gate_proj.weight``, ``up_proj.weight`` and
``down_proj.weight.T`` in ``nn.Linear`` terms.  Entries are i.i.d., so drawing
directly in this layout is the same distribution as drawing the paper's
``W_gate in R^{d_model x d_ff}`` and transposing.

Random streams per config (numpy PCG64): weight matrix m (0 = W_gate,
1 = W_up, 2 = W_down) is drawn in chunks of 2048 channel rows, chunk c from
``default_rng([seed, m, c]).standard_normal(float32) * sigma`` (independent
streams, so chunks are drawn in parallel); the outlier channel indices
(``choice(d, n_out, replace=False)``) and then the x vectors come from
``default_rng([seed, 3])``.  fp32 values are cast to bf16/fp16 with
round-to-nearest-even.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import List, Optional, Tuple

import numpy as np

DT_F16 = 0
DT_BF16 = 1
DTYPE_NAMES = {DT_F16: "f16", DT_BF16: "bf16"}

# Channel rows of a weight matrix drawn from one child stream.
_CHUNK_ROWS = 2048
_THREADS = max(1, min(16, os.cpu_count() or 1))


def frac_to_k(frac: float, n: int) -> int:
    """Integer count kept for a kept-fraction ``frac`` of ``n`` entries."""
    return int(math.floor(frac * n + 0.5))


@dataclasses.dataclass(frozen=True)
class FFNConfig:
    """One synthetic decode-FFN workload."""
    name: str
    d_model: int
    d_ff: int
    dtype: int                 # DT_F16 or DT_BF16
    sigma_w: float
    seed: int
    x_kind: str                # "laplace" or "student_t"
    n_outliers: int
    outlier_scale: float
    qbits: int                 # 8 or 4
    group: int                 # quantisation group along d_model
    in_frac: float             # kept fraction of input channels (Stage 1)
    ff_frac: float             # kept fraction of intermediate channels (Stage 2)
    batch: int = 1
    n_vectors: int = 1
    t_nu: float = 3.0

    @property
    def k_in(self) -> int:
        return frac_to_k(self.in_frac, self.d_model)

    @property
    def k_ff(self) -> int:
        return frac_to_k(self.ff_frac, self.d_ff)

    def with_(self, **kw) -> "FFNConfig":
        return dataclasses.replace(self, **kw)


# The five synthetic workloads.  "ffn sparsity" s2 = 1 - ff_frac.
CONFIGS = {
    # 1024x3072 fp16, int8 per-output-channel proxy (group = d_model).
    "c1_1024x3072_f16": FFNConfig("c1_1024x3072_f16", 1024, 3072, DT_F16, 0.02, 0,
                                  "laplace", 4, 20.0, 8, 1024, 0.5, 0.5,
                                  n_vectors=100),
    # Qwen3-8B FFN shape, int4 group-128 proxy, 70% FFN sparsity.
    "c2_4096x12288_bf16": FFNConfig("c2_4096x12288_bf16", 4096, 12288, DT_BF16, 0.02, 1,
                                    "laplace", 16, 30.0, 4, 128, 0.5, 0.3,
                                    n_vectors=1000),
    # Llama3-8B FFN shape, Student-t inputs; batch and sparsity are swept.
    "c3_4096x14336_bf16": FFNConfig("c3_4096x14336_bf16", 4096, 14336, DT_BF16, 0.02, 2,
                                    "student_t", 0, 1.0, 4, 128, 0.5, 0.3,
                                    n_vectors=100),
    # 8192x28672 FFN, int4 group-128 proxy, 40% inputs / 30% channels kept.
    "c4_8192x28672_bf16": FFNConfig("c4_8192x28672_bf16", 8192, 28672, DT_BF16, 0.015, 3,
                                    "laplace", 32, 40.0, 4, 128, 0.4, 0.3,
                                    n_vectors=1000),
}

# 36-layer stack of Qwen3-8B-shaped FFNs, x_{l+1} = RMSNorm(x_l + FFN_l(x_l)).
STACK_LAYERS = 36
STACK_BASE = CONFIGS["c2_4096x12288_bf16"].with_(name="c5_stack36_4096x12288_bf16",
                                                  n_vectors=100)
C3_FFN_SPARSITIES = (0.0, 0.5, 0.7, 0.9)
C3_BATCHES = (1, 4, 16)


def stack_layer_config(layer: int) -> FFNConfig:
    """Layer ``layer`` of the 36-layer stack: independent weights, seed 4+layer."""
    return STACK_BASE.with_(seed=4 + layer, name=f"c5_layer{layer}")


# ----------------------------------------------------------------------------
# Casting fp32 -> 16-bit patterns (round to nearest even)
# ----------------------------------------------------------------------------

def f32_to_bf16_bits_ref(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round-to-nearest-even (finite inputs)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round-to-nearest-even.  Uses torch's cast
    (multi-threaded); the tests check it against f32_to_bf16_bits_ref."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def f32_to_f16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> fp16 bit patterns (numpy's cast is round-to-nearest-even)."""
    return np.ascontiguousarray(a, dtype=np.float32).astype(np.float16).view(np.uint16)


def to_bits(a: np.ndarray, dtype: int) -> np.ndarray:
    return f32_to_bf16_bits(a) if dtype == DT_BF16 else f32_to_f16_bits(a)


def bits_to_f32(bits: np.ndarray, dtype: int) -> np.ndarray:
    """16-bit patterns -> fp32 values (exact)."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    if dtype == DT_BF16:
        return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)
    return bits.view(np.float16).astype(np.float32)


# ----------------------------------------------------------------------------
# Generators
# ----------------------------------------------------------------------------

def _draw_matrix(seed: int, m: int, rows: int, cols: int, sigma: float,
                 dtype: int) -> np.ndarray:
    out = np.empty((rows, cols), dtype=np.uint16)

    def chunk(c: int) -> None:
        r0 = c * _CHUNK_ROWS
        r1 = min(rows, r0 + _CHUNK_ROWS)
        blk = np.random.default_rng([seed, m, c]).standard_normal((r1 - r0, cols),
                                                                 dtype=np.float32)
        blk *= np.float32(sigma)
        out[r0:r1] = to_bits(blk, dtype)

    n = (rows + _CHUNK_ROWS - 1) // _CHUNK_ROWS
    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(chunk, range(n)))
    return out


@dataclasses.dataclass
class Workload:
    cfg: FFNConfig
    w_gate: np.ndarray         # uint16 [d_ff][d_model]
    w_up: np.ndarray           # uint16 [d_ff][d_model]
    w_down: np.ndarray         # uint16 [d_ff][d_model]
    outliers: np.ndarray       # int64 [n_outliers]
    rng: np.random.Generator   # positioned after the weights/outliers

    def x_vectors(self, n: int, batch: Optional[int] = None) -> np.ndarray:
        """Draw ``n`` decode inputs, uint16 [n][batch][d_model]."""
        return draw_x(self.rng, self.cfg, n, batch or self.cfg.batch, self.outliers)


def draw_x(rng: np.random.Generator, cfg: FFNConfig, n: int, batch: int,
           outliers: np.ndarray) -> np.ndarray:
    shape = (n, batch, cfg.d_model)
    if cfg.x_kind == "laplace":
        x = rng.laplace(0.0, 1.0, size=shape).astype(np.float32)
    elif cfg.x_kind == "student_t":
        x = rng.standard_t(cfg.t_nu, size=shape).astype(np.float32)
    else:
        raise ValueError(cfg.x_kind)
    if len(outliers):
        x[..., outliers] *= np.float32(cfg.outlier_scale)
    return to_bits(x, cfg.dtype)


def make_workload(cfg: FFNConfig, weights: bool = True) -> Workload:
    """Weights and outlier channels for ``cfg`` in the documented draw order."""
    f, d = cfg.d_ff, cfg.d_model
    if weights:
        wg = _draw_matrix(cfg.seed, 0, f, d, cfg.sigma_w, cfg.dtype)
        wu = _draw_matrix(cfg.seed, 1, f, d, cfg.sigma_w, cfg.dtype)
        wd = _draw_matrix(cfg.seed, 2, f, d, cfg.sigma_w, cfg.dtype)
    else:
        wg = wu = wd = None
    rng = np.random.default_rng([cfg.seed, 3])
    out = (rng.choice(d, cfg.n_outliers, replace=False).astype(np.int64)
           if cfg.n_outliers else np.zeros(0, np.int64))
    return Workload(cfg, wg, wu, wd, out, rng)


def reservoir_draws(seed: int):
    """Uniform 64-bit random numbers for the calibration reservoirs (one per
    offered sample), from a seeded stream: returns draw(n) -> uint64 [n]."""
    rng = np.random.default_rng([seed, 7])

    def draw(n: int) -> np.ndarray:
        return rng.integers(0, np.iinfo(np.uint64).max, size=n, dtype=np.uint64,
                            endpoint=True)
    return draw


def small_config(name: str = "tiny", d: int = 256, f: int = 384, dtype: int = DT_BF16,
                 qbits: int = 4, group: int = 128, in_frac: float = 0.5,
                 ff_frac: float = 0.3, batch: int = 1, seed: int = 11,
                 x_kind: str = "laplace", n_outliers: int = 3,
                 outlier_scale: float = 20.0, sigma_w: float = 0.05) -> FFNConfig:
    """A reduced-size config with the same recipe, for tests the oracle
    finishes in seconds (several tiles plus a ragged tail)."""
    return FFNConfig(name, d, f, dtype, sigma_w, seed, x_kind, n_outliers, outlier_scale,
                     qbits, group, in_frac, ff_frac, batch=batch, n_vectors=4)
