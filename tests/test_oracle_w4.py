"""Pins of the oracle's Stage 2 on INT4 base weights (W4A16: low-bit weights
combined with the sparse step, which Sec. 5.1 leaves to future work).

  * Weights that are exactly sigma * q (sigma a power of two per group,
    |q| <= 7 with a 7 in every group) come back unchanged from the 4-bit
    quantiser of Sec. 4.3, and the W4 Stage 2 on their codes (group sums of
    x q, scaled once per group) equals the 16-bit Stage 2 on the weights
    themselves (one plain sum of x w).
  * Keeping every input and every channel, the W4 decode step is the W4 dense
    FFN.
  * A hand-sized example with two groups and one channel, in closed form.
"""
import math

import numpy as np
import pytest

from paper_2607_27591_amd import workloads as W


def _exact_w4(rng, f, d, group, dtype):
    """[f][d] weights equal to sigma_{j,g} q_{j,i} exactly, and their (q, sigma)."""
    ng = d // group
    q = rng.integers(-7, 8, size=(f, d))
    for j in range(f):
        for g in range(ng):
            q[j, g * group + rng.integers(group)] = rng.choice([-7, 7])   # amax = 7 sigma
    sigma = 2.0 ** -rng.integers(3, 9, size=(f, ng)).astype(np.float64)
    w = q * np.repeat(sigma, group, axis=1)
    bits = W.to_bits(w.astype(np.float32), dtype)
    assert np.array_equal(W.bits_to_f32(bits, dtype).astype(np.float64), w)
    return bits, q.astype(np.int8), np.float16(sigma).view(np.uint16)


@pytest.mark.parametrize("dtype", [W.DT_BF16, W.DT_F16])
def test_quantiser_recovers_exact_w4_weights(oracle_lib, dtype):
    rng = np.random.default_rng(1)
    bits, q, s = _exact_w4(rng, 24, 384, 128, dtype)
    codes, scales = oracle_lib.quantize(bits, dtype, 4, 128)
    assert np.array_equal(codes, q)
    assert np.array_equal(scales, s)


@pytest.mark.parametrize("dtype,act", [(W.DT_BF16, 0), (W.DT_F16, 0), (W.DT_BF16, 1)])
def test_w4_stage2_equals_16bit_stage2_on_exact_weights(oracle_lib, dtype, act):
    rng = np.random.default_rng(2 + act)
    B, d, f, group = 3, 384, 40, 128
    mats = [_exact_w4(rng, f, d, group, dtype) for _ in range(3)]
    w4 = {"group": group}
    for key, (_, q, s) in zip(("g", "u", "d"), mats):
        w4["codes_" + key], w4["scales_" + key] = q, s
    x = W.to_bits(rng.standard_normal((B, d)).astype(np.float32), dtype)
    ff_idx = np.sort(rng.choice(f, size=17, replace=False)).astype(np.int32)
    s16, y16 = oracle_lib.stage2(x, dtype, mats[0][0], mats[1][0], mats[2][0], ff_idx, act)
    s4, y4 = oracle_lib.stage2_w4(x, dtype, w4, ff_idx, act)
    np.testing.assert_allclose(s4, s16, rtol=1e-12, atol=1e-12 * np.abs(s16).max())
    np.testing.assert_allclose(y4, y16, rtol=1e-12, atol=1e-12 * np.abs(y16).max())


def test_w4_full_keep_is_dense_w4(oracle_lib):
    cfg = W.small_config(d=256, f=96, batch=2, seed=5, sigma_w=0.05)
    wl = W.make_workload(cfg)
    x = wl.x_vectors(1, cfg.batch)[0]
    w4 = oracle_lib.quantize_w4(wl.w_gate, wl.w_up, wl.w_down, cfg.dtype, 128)
    cg, sg = oracle_lib.quantize(wl.w_gate, cfg.dtype, 4, 128)
    cu, su = oracle_lib.quantize(wl.w_up, cfg.dtype, 4, 128)
    out = oracle_lib.ffn_sparse_w4(x, cfg.dtype, w4, cfg.d_model, cfg.d_ff, codes_g=cg,
                                   scales_g=sg, codes_u=cu, scales_u=su, group=128)
    assert np.array_equal(out["y"], oracle_lib.ffn_dense_w4(x, cfg.dtype, w4))


def test_w4_hand_example(oracle_lib):
    # d = 256 in two groups of 128, one channel, x = 1 at input 0 and 2 at 200.
    d, group = 256, 128
    x = np.zeros((1, d), np.float32)
    x[0, 0], x[0, 200] = 1.0, 2.0
    xb = W.to_bits(x, W.DT_BF16)
    z = lambda: np.zeros((1, d), np.int8)
    cg, cu, cd = z(), z(), z()
    cg[0, 0], cg[0, 200] = 3, -2
    cu[0, 0], cu[0, 200] = 1, 4
    cd[0, 5], cd[0, 130] = 7, -1
    f16 = lambda *v: np.float16(v).view(np.uint16).reshape(1, -1)
    w4 = dict(codes_g=cg, scales_g=f16(0.5, 0.25), codes_u=cu, scales_u=f16(1.0, 0.125),
              codes_d=cd, scales_d=f16(0.5, 2.0), group=group)
    s, y = oracle_lib.stage2_w4(xb, W.DT_BF16, w4, np.array([0], np.int32))
    g = 0.5 * 3 * 1.0 + 0.25 * (-2) * 2.0      # 0.5
    u = 1.0 * 1 * 1.0 + 0.125 * 4 * 2.0       # 2.0
    s_ref = g / (1.0 + math.exp(-g)) * u
    assert s[0, 0] == pytest.approx(s_ref, rel=1e-15)
    y_ref = np.zeros(d)
    y_ref[5], y_ref[130] = s_ref * 0.5 * 7, s_ref * 2.0 * -1
    np.testing.assert_allclose(y[0], y_ref, rtol=1e-15, atol=0)
