"""Threshold calibration of the threshold-mode decode step (App. A.7, Alg. 1).

Layers are calibrated in depth order.  Each layer sees its calibration inputs
as produced by the earlier layers running with their final thresholds.  A
layer's tau_x is the empirical quantile, at target sparsity s1, of a bounded
sample of |x| over the calibration tokens.  tau_s is the quantile at s2 of
|s~|, the proxy intermediate of each token computed on its input mask m_x.
The forward passes run on the GPU through libprox, one token per call so
every token gets its own masks.  The bounded samples (Algorithm R) and their
quantiles are libprox's host calls.
"""
from __future__ import annotations

import ctypes
import math
from typing import Callable, List, Sequence, Tuple

import numpy as np
import torch

from . import prox

Draw = Callable[[int], np.ndarray]   # n -> n uniform uint64 random numbers


class Reservoir:
    """A bounded sample of at most `cap` float32 values (App. A.7)."""

    def __init__(self, cap: int):
        self.cap = int(cap)
        self.buf = np.zeros(self.cap, np.float32)
        self.seen = ctypes.c_uint64(0)

    def add(self, values: np.ndarray, draws: np.ndarray) -> None:
        v = np.ascontiguousarray(values, dtype=np.float32).ravel()
        r = np.ascontiguousarray(draws, dtype=np.uint64).ravel()
        if r.size != v.size:
            raise ValueError("one draw per value")
        prox._check(prox.lib().prox_reservoir_add(
            self.buf.ctypes.data, self.cap, ctypes.byref(self.seen), v.ctypes.data, v.size,
            r.ctypes.data), "prox_reservoir_add")

    def sample(self) -> np.ndarray:
        return self.buf[:min(self.cap, self.seen.value)]


def quantile_threshold(samples: np.ndarray, sparsity: float) -> float:
    """The sample value at ascending position min(n - 1, floor(sparsity n))."""
    v = np.ascontiguousarray(samples, dtype=np.float32)
    tau = ctypes.c_float()
    prox._check(prox.lib().prox_quantile_threshold(v.ctypes.data, v.size, float(sparsity),
                                                   ctypes.byref(tau)), "prox_quantile_threshold")
    return float(tau.value)


def proxy_magnitudes(w: prox.Weights, p: prox.Proxy, x: torch.Tensor, tau_x: float,
                     scores: torch.Tensor, ws: torch.Tensor) -> np.ndarray:
    """|s~| of one token (x: [1][d]) on its input mask |x| >= tau_x: the
    proxy scores of a one-row call (no channel kept: tau_s = +inf)."""
    prox.ffn_sparse_tau(w, p, x, tau_x, math.inf, scores=scores, ws=ws)
    return scores.cpu().numpy()


def layer_forward(w: prox.Weights, p: prox.Proxy, xs: torch.Tensor, tau_x: float, tau_s: float,
                  ws: torch.Tensor, eps: float = 1e-6) -> torch.Tensor:
    """x' = RMSNorm(x + FFN(x)) for each token row of xs, with the threshold
    rule applied per token."""
    out = torch.empty_like(xs)
    for t in range(xs.shape[0]):
        y, _, _ = prox.ffn_sparse_tau(w, p, xs[t:t + 1], tau_x, tau_s, ws=ws)
        prox.add_rmsnorm(xs[t:t + 1], y, eps, out=out[t:t + 1])
    return out


def calibrate_stack(layers: Sequence[Tuple[prox.Weights, prox.Proxy]], tokens: torch.Tensor,
                    s1: float, s2: float, cap: int, draw: Draw,
                    eps: float = 1e-6) -> List[Tuple[float, float]]:
    """Alg. 1 on calibration tokens ([T][d] device tensor of the weights'
    dtype).  Returns [(tau_x, tau_s)] per layer.  Random draws are consumed
    per token, |x| first (d per token), then |s~| (d_ff per token)."""
    xs = tokens.contiguous()
    T = xs.shape[0]
    taus = []
    for w, p in layers:
        ws = prox.new_workspace(w.d_model, w.d_ff, 1, xs.device)
        res_x = Reservoir(cap)
        mags = xs.float().abs().cpu().numpy()
        for t in range(T):
            res_x.add(mags[t], draw(w.d_model))
        tau_x = quantile_threshold(res_x.sample(), s1)
        res_s = Reservoir(cap)
        scores = torch.empty(w.d_ff, dtype=torch.float32, device=xs.device)
        for t in range(T):
            res_s.add(proxy_magnitudes(w, p, xs[t:t + 1], tau_x, scores, ws), draw(w.d_ff))
        tau_s = quantile_threshold(res_s.sample(), s2)
        taus.append((tau_x, tau_s))
        xs = layer_forward(w, p, xs, tau_x, tau_s, ws, eps)
    return taus
