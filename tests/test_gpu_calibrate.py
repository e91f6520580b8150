"""Sequential threshold calibration (App. A.7, Alg. 1) run on the GPU path:
libprox's threshold-mode kernels produce the signals, its host calls keep the
bounded samples and take the quantiles.

Checks:
  * the calibrated thresholds are the order statistics of the signals that
    each layer sees when the finished stack runs on the calibration tokens
    (the property that makes the calibration sequential; with every sample
    kept it must hold exactly);
  * layer 0 (identical inputs and random draws on both sides): tau_x equals
    the oracle's bit for bit, tau_s agrees to the proxy-score tolerance, with
    and without a reservoir smaller than the sample stream.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2607_27591_amd import calibrate as C
from paper_2607_27591_amd import prox
from paper_2607_27591_amd import workloads as W

from gpu_cases import SCORE_TOL, log, make_case

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def stack():
    cases = []
    for l in range(3):
        cfg = W.small_config(d=256, f=384, seed=60 + l, sigma_w=0.05, n_outliers=2)
        cases.append(make_case(cfg))
    tokens = cases[0].wl.x_vectors(8, 1)[:, 0, :]
    log("[calib] 3-layer 256x384 stack, 8 tokens")
    yield cases, tokens
    del cases
    torch.cuda.empty_cache()


def _oracle_layers(cases):
    return [dict(w_gate=c.wl.w_gate, w_up=c.wl.w_up, w_down=c.wl.w_down, codes_g=c.codes_g,
                 scales_g=c.scales_g, codes_u=c.codes_u, scales_u=c.scales_u,
                 group=c.cfg.group) for c in cases]


def _order_statistic(v, tau, s):
    pos = min(v.size - 1, math.floor(s * v.size))
    return (v < tau).sum() <= pos < (v <= tau).sum()


def test_gpu_calibration_is_sequential(stack):
    cases, tokens = stack
    s1, s2 = 0.5, 0.7
    layers = [(c.w, c.proxy) for c in cases]
    x0 = prox.from_bits(tokens, cases[0].cfg.dtype)
    taus = C.calibrate_stack(layers, x0, s1, s2, 10 ** 6, W.reservoir_draws(9))
    log(f"    taus {taus}")
    xs = x0
    for l, ((w, p), (tx, ts)) in enumerate(zip(layers, taus)):
        ws = prox.new_workspace(w.d_model, w.d_ff, 1)
        scores = torch.empty(w.d_ff, dtype=torch.float32, device="cuda")
        mx = xs.float().abs().cpu().numpy().ravel()
        sv = np.concatenate([C.proxy_magnitudes(w, p, xs[t:t + 1], tx, scores, ws)
                             for t in range(xs.shape[0])])
        assert _order_statistic(mx, np.float32(tx), s1), f"layer {l}: tau_x"
        assert _order_statistic(sv, np.float32(ts), s2), f"layer {l}: tau_s"
        xs = C.layer_forward(w, p, xs, tx, ts, ws)


@pytest.mark.parametrize("cap", [10 ** 6, 1000])
def test_gpu_calibration_layer0_matches_oracle(stack, cap):
    cases, tokens = stack
    s1, s2 = 0.6, 0.7
    c = cases[0]
    taus = C.calibrate_stack([(c.w, c.proxy)], prox.from_bits(tokens, c.cfg.dtype), s1, s2, cap,
                             W.reservoir_draws(11))
    ref = oracle.calibrate_stack(tokens, c.cfg.dtype, _oracle_layers(cases[:1]), s1, s2, cap,
                                 W.reservoir_draws(11))
    log(f"[calib layer 0] cap={cap} gpu {taus[0]} oracle {ref[0]}")
    assert taus[0][0] == ref[0][0]
    assert abs(taus[0][1] - ref[0][1]) <= SCORE_TOL * ref[0][1]
