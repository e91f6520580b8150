"""Pins of the oracle's GeGLU variant (gate activation GELU(z) = z Phi(z) in
place of SiLU; the gated FFN of Sec. 2.1 with another activation)."""
import math

import numpy as np
import pytest
from scipy.special import erf
from scipy.stats import norm

from paper_2607_27591_amd import workloads as W


@pytest.mark.parametrize("z", [-6.0, -3.0, -1.0, -0.25, 0.0, 0.5, 1.0, 2.0, 4.0])
def test_gelu_is_z_times_normal_cdf(oracle_lib, z):
    assert oracle_lib.gate_act(z, oracle_lib.GELU) == pytest.approx(z * norm.cdf(z), rel=1e-14,
                                                                    abs=1e-300)


def test_gelu_odd_part_identity(oracle_lib):
    # Phi(z) + Phi(-z) = 1, so GELU(z) - GELU(-z) = z
    for z in np.linspace(-8, 8, 161):
        g = oracle_lib.gate_act(z, oracle_lib.GELU) - oracle_lib.gate_act(-z, oracle_lib.GELU)
        assert g == pytest.approx(z, abs=1e-14)


def test_silu_unchanged(oracle_lib):
    for z in (-3.0, 0.0, 1.0, 5.0):
        assert oracle_lib.gate_act(z, oracle_lib.SILU) == pytest.approx(z / (1 + math.exp(-z)),
                                                                        rel=1e-15)


def _tiny(seed, B=2, d=96, f=160):
    cfg = W.small_config(d=d, f=f, seed=seed, batch=B, sigma_w=0.05, n_outliers=2, group=32)
    wl = W.make_workload(cfg)
    return cfg, wl, wl.x_vectors(1, B)[0]


def test_dense_geglu_matches_numpy_definition(oracle_lib):
    cfg, wl, x = _tiny(3)
    f64 = lambda b: W.bits_to_f32(b, cfg.dtype).astype(np.float64)
    xf, wg, wu, wd = f64(x), f64(wl.w_gate), f64(wl.w_up), f64(wl.w_down)
    g = xf @ wg.T
    want = ((xf @ wu.T) * (0.5 * g * (1 + erf(g / math.sqrt(2))))) @ wd
    got = oracle_lib.ffn_dense(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down, act=oracle_lib.GELU)
    assert np.abs(got - want).max() <= 1e-12 * np.abs(want).max()
    silu = oracle_lib.ffn_dense(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down)
    assert np.abs(silu - got).max() > 1e-3 * np.abs(want).max()   # the activation matters


def test_geglu_full_channels_equal_dense_bitwise(oracle_lib):
    cfg, wl, x = _tiny(4)
    cg, sg = oracle_lib.quantize(wl.w_gate, cfg.dtype, 4, 32)
    cu, su = oracle_lib.quantize(wl.w_up, cfg.dtype, 4, 32)
    out = oracle_lib.ffn_sparse(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down, 40, cfg.d_ff,
                                codes_g=cg, scales_g=sg, codes_u=cu, scales_u=su, group=32,
                                act=oracle_lib.GELU)
    dense = oracle_lib.ffn_dense(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down, act=oracle_lib.GELU)
    assert np.array_equal(out["y"], dense)


def test_geglu_proxy_score_definition(oracle_lib):
    # Unquantised proxy, every input kept: score_j = max_b |GELU(g_j) u_j|.
    cfg, wl, x = _tiny(5)
    f64 = lambda b: W.bits_to_f32(b, cfg.dtype).astype(np.float64)
    xf, wg, wu = f64(x), f64(wl.w_gate), f64(wl.w_up)
    g, u = xf @ wg.T, xf @ wu.T
    want = np.abs(0.5 * g * (1 + erf(g / math.sqrt(2))) * u).max(axis=0)
    _, _, _, score = oracle_lib.proxy(x, cfg.dtype, np.arange(cfg.d_model, dtype=np.int32),
                                      w_gate=wl.w_gate, w_up=wl.w_up, kind=oracle_lib.PROXY_NONE,
                                      act=oracle_lib.GELU)
    assert np.abs(score - want).max() <= 1e-12 * want.max()
