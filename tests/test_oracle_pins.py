"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these compare the oracle with itself: each check comes from a closed
form, an invariant, a special case that reduces to a library routine, the
paper's printed constants (tests/golden/), or brute force on tiny inputs.
"""
import json
import math
import os

import numpy as np
import pytest

from paper_2607_27591_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        return json.load(fh)


def _as_f64(bits, dtype):
    return W.bits_to_f32(bits, dtype).astype(np.float64)


def _silu(z):
    return z / (1.0 + np.exp(-z))


def _tiny(seed=5, d=64, f=96, B=1, dtype=W.DT_BF16, sigma=0.05, x_kind="laplace"):
    cfg = W.small_config(d=d, f=f, dtype=dtype, seed=seed, batch=B, sigma_w=sigma,
                         x_kind=x_kind, n_outliers=2, group=32)
    wl = W.make_workload(cfg)
    x = wl.x_vectors(1, B)[0]
    return cfg, wl, x


# ---------------------------------------------------------------------------
# Number formats (exact conversions; RNE rounding to fp16)
# ---------------------------------------------------------------------------

def test_half_to_double_exhaustive(oracle_lib):
    """All 65536 patterns of both formats against numpy's fp16 and the bf16
    definition (the top half of a binary32)."""
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    want16 = bits.view(np.float16).astype(np.float64)
    with np.errstate(invalid="ignore"):
        wantbf = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    for dt, want in ((W.DT_F16, want16), (W.DT_BF16, wantbf)):
        got = oracle_lib.halves_to_double(bits, dt)
        nan = np.isnan(want)
        assert np.array_equal(np.isnan(got), nan)
        assert np.array_equal(got[~nan], want[~nan])
        # the scalar entry point agrees with the array one on a spread of patterns
        for b in range(0, 65536, 257):
            g = oracle_lib.half_to_double(b, dt)
            assert (math.isnan(g) and nan[b]) or g == want[b]


def _bf16_rne_exact(v):
    """bfloat16 RNE of a finite double by exact rational arithmetic (bit
    pattern): the quantum of the value's binade (2^-133 below 2^-126), the
    quotient rounded half to even, overflow to infinity at 2^128."""
    from fractions import Fraction
    sign = 0x8000 if math.copysign(1.0, v) < 0 else 0
    a = Fraction(abs(v))
    if a == 0:
        return sign
    e = math.frexp(abs(v))[1] - 1
    e = max(e, -126)
    quantum = Fraction(2) ** (e - 7)
    q = a / quantum
    n = math.floor(q)
    rem = q - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    r = n * quantum
    if r >= Fraction(2) ** 128:
        return sign | 0x7F80
    f32 = np.array(float(r), np.float32)       # exact: r has at most 8 significant bits
    assert Fraction(float(f32)) == r
    return sign | int(f32.view(np.uint32)) >> 16


def test_double_to_bf16_is_rne(oracle_lib):
    """bf16 RNE of the oracle against torch's binary32 -> bfloat16 cast (RNE)
    on binary32 values, including every 97th midpoint between adjacent bf16
    values and their binary32 neighbours; and against exact rational rounding
    on doubles with bits below binary32 precision (where rounding through
    binary32 first would differ)."""
    import torch
    pos = np.arange(0, 0x7F7F, 97, dtype=np.uint32)
    lo = (pos << 16).view(np.float32).astype(np.float64)
    hi = ((pos + 1) << 16).view(np.float32).astype(np.float64)
    mids = ((lo + hi) / 2).astype(np.float32)             # 9 significant bits: exact
    rng = np.random.default_rng(3)
    rnd = (rng.standard_normal(4000) * np.exp(rng.uniform(-90, 80, 4000))).astype(np.float32)
    f32 = np.concatenate([mids, -mids, np.nextafter(mids, np.float32(0)),
                          np.nextafter(mids, np.float32(np.inf)), rnd,
                          np.array([0.0, -0.0, 1.0, 3.0e38, 3.4028235e38, 1e-40, 1e-45,
                                    2.0 ** -126, 2.0 ** -133, 3 * 2.0 ** -134], np.float32)])
    f32 = f32[np.isfinite(f32)]
    want = torch.from_numpy(f32.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = oracle_lib.round_to_dtype(f32.astype(np.float64), W.DT_BF16)
    assert np.array_equal(got, want)
    for v, w_ in zip(f32[::53], want[::53]):
        assert oracle_lib.double_to_bf16(float(v)) == int(w_)
    # doubles that binary32 cannot hold: a midpoint plus or minus 2^-40 of it
    base = mids[::7].astype(np.float64)
    near = np.concatenate([base * (1 + 2.0 ** -40), base * (1 - 2.0 ** -40),
                           rng.standard_normal(500) * np.exp(rng.uniform(-80, 80, 500))])
    got = oracle_lib.round_to_dtype(near, W.DT_BF16)
    for v, g in zip(near, got):
        assert int(g) == _bf16_rne_exact(float(v)), v


def test_double_to_f16_is_ieee_rne(oracle_lib):
    """numpy's float64 -> float16 cast is correctly rounded (ties to even)."""
    rng = np.random.default_rng(1)
    vals = list(rng.standard_normal(3000) * np.exp(rng.uniform(-20, 12, 3000)))
    # Every midpoint between adjacent finite fp16 values, plus neighbours.
    h = np.arange(0, 0x7BFF, 37, dtype=np.uint16).view(np.float16).astype(np.float64)
    h2 = (np.arange(0, 0x7BFF, 37, dtype=np.uint16) + 1).view(np.float16).astype(np.float64)
    mids = (h + h2) / 2
    vals += list(mids) + list(-mids) + list(np.nextafter(mids, 0)) + list(np.nextafter(mids, 1e9))
    vals += [0.0, -0.0, 65504.0, 65519.99, 65520.0, 1e6, 2.0 ** -24, 2.0 ** -25,
             3 * 2.0 ** -26, 2.0 ** -14, 6.1e-5]
    for v in vals:
        with np.errstate(over="ignore"):
            want = int(np.array(v, np.float64).astype(np.float16).view(np.uint16))
        assert oracle_lib.double_to_f16(v) == want, v


# ---------------------------------------------------------------------------
# Step 1: proxy quantisation (Sec. 4.3)
# ---------------------------------------------------------------------------

def test_quant_hand_worked_ties(oracle_lib):
    g = _golden("quant_ties.json")
    w = np.array(g["w"], np.float32)
    bits = W.f32_to_bf16_bits(w).reshape(1, -1)
    assert np.array_equal(W.bits_to_f32(bits, W.DT_BF16).ravel(), w)   # exact in bf16
    codes, scales = oracle_lib.quantize(bits, W.DT_BF16, g["bits"], g["group"])
    assert codes.ravel().tolist() == g["codes"]
    assert scales.view(np.float16).astype(np.float64).ravel().tolist() == [g["sigma"]]


@pytest.mark.parametrize("bits,group,dtype", [(4, 128, W.DT_BF16), (4, 32, W.DT_BF16),
                                              (8, 256, W.DT_F16), (8, 64, W.DT_BF16)])
def test_quant_invariants(oracle_lib, bits, group, dtype):
    rng = np.random.default_rng(bits * 100 + group)
    f, d = 40, 256
    w32 = (rng.standard_normal((f, d)) * 0.02).astype(np.float32)
    w32[3, :group] = 0.0                       # an all-zero group
    w32[5] *= 1e3                              # a large-scale channel
    wb = W.to_bits(w32, dtype)
    wv = W.bits_to_f32(wb, dtype).astype(np.float64)
    codes, scales = oracle_lib.quantize(wb, dtype, bits, group)
    qmax = 2 ** (bits - 1) - 1
    sig = scales.view(np.float16).astype(np.float64)            # [f][d/group]
    sig_full = np.repeat(sig, group, axis=1)
    assert np.abs(codes.astype(int)).max() <= qmax
    # scale = fp16 RNE of the group's amax / qmax (numpy's correctly rounded cast)
    amax = np.abs(wv).reshape(f, d // group, group).max(axis=2)
    assert np.array_equal(scales, (amax / qmax).astype(np.float16).view(np.uint16))
    # zero group -> zero scale, zero codes
    assert scales[3, 0] == 0 and not codes[3, :group].any()
    # reconstruction error at most half a quantum, except where the group
    # amax was clamped after fp16 rounding of the scale pushed it past qmax
    err = np.abs(wv - codes * sig_full)
    unclamped = np.abs(wv) <= qmax * sig_full
    assert (err[unclamped] <= 0.5 * sig_full[unclamped] * (1 + 1e-12)).all()
    assert (err[~unclamped] <= np.abs(wv[~unclamped]) - qmax * sig_full[~unclamped]
            + 0.5 * sig_full[~unclamped] + 1e-300).all()
    # the largest entry of each non-zero group lands on +-qmax (or qmax-1 if the
    # fp16-rounded scale came out above amax/qmax)
    am = np.abs(codes.astype(int)).reshape(f, d // group, group).max(axis=2)
    nz = amax > 0
    assert ((am[nz] == qmax) | (am[nz] == qmax - 1)).all()
    # sign symmetry: quant(-W) = -quant(W), same scales
    neg = W.to_bits(-w32, dtype)
    c2, s2 = oracle_lib.quantize(neg, dtype, bits, group)
    assert np.array_equal(s2, scales) and np.array_equal(c2, -codes)


def test_quant_lossless_grid(oracle_lib):
    """Weights that are already q*sigma with amax = qmax*sigma come back exactly."""
    rng = np.random.default_rng(7)
    f, d, group = 12, 64, 16
    q = rng.integers(-7, 8, size=(f, d))
    q[:, ::group] = 7 * rng.choice([-1, 1], size=(f, d // group))   # amax = 7 sigma
    sig = 2.0 ** rng.integers(-10, -3, size=(f, d // group))
    w = (q * np.repeat(sig, group, axis=1)).astype(np.float32)
    codes, scales = oracle_lib.quantize(W.f32_to_bf16_bits(w), W.DT_BF16, 4, group)
    assert np.array_equal(codes, q)
    assert np.array_equal(scales.view(np.float16).astype(np.float64), sig)


# ---------------------------------------------------------------------------
# Steps 2 and 4: top-k selection (App. A.6), brute force with crafted ties
# ---------------------------------------------------------------------------

def _brute_topk(key, k):
    order = sorted(range(len(key)), key=lambda i: (-key[i], i))
    return sorted(order[:k])


@pytest.mark.parametrize("case", ["dups", "zeros", "allequal", "random", "signs"])
def test_topk_brute_force(oracle_lib, case):
    rng = np.random.default_rng(len(case))
    n = 37
    if case == "dups":
        key = rng.integers(0, 5, n).astype(float)
    elif case == "zeros":
        key = np.where(rng.random(n) < 0.6, 0.0, rng.random(n))
    elif case == "allequal":
        key = np.full(n, 2.5)
    elif case == "signs":
        key = np.abs(rng.choice([-1.0, 1.0], n) * rng.integers(0, 3, n))
    else:
        key = rng.random(n)
    for k in [0, 1, 5, 18, 36, 37]:
        assert oracle_lib.topk(key, k).tolist() == _brute_topk(list(key), k)


def test_select_inputs_brute_force(oracle_lib):
    """a_i = max_b |x_{b,i}|; +0 and -0 tie; ties go to the lower index."""
    rng = np.random.default_rng(3)
    B, d = 3, 29
    vals = rng.choice([-2.0, -1.0, -0.0, 0.0, 1.0, 2.0, 0.5, -0.5], size=(B, d))
    bits = W.f32_to_bf16_bits(vals.astype(np.float32))
    a = np.abs(vals).max(axis=0)
    for k in [1, 4, 10, 28, 29]:
        assert oracle_lib.select_inputs(bits, W.DT_BF16, k).tolist() == _brute_topk(list(a), k)


# ---------------------------------------------------------------------------
# P1: sparsity 0 reproduces the dense FFN (Sec. 2.1), which equals the plain
# matrix definition evaluated by numpy.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,B", [(W.DT_BF16, 1), (W.DT_F16, 3)])
def test_dense_matches_numpy_definition(oracle_lib, dtype, B):
    cfg, wl, x = _tiny(seed=9, B=B, dtype=dtype)
    y = oracle_lib.ffn_dense(x, dtype, wl.w_gate, wl.w_up, wl.w_down)
    xf = _as_f64(x, dtype)
    wg, wu, wd = (_as_f64(m, dtype) for m in (wl.w_gate, wl.w_up, wl.w_down))
    ref = ((xf @ wu.T) * _silu(xf @ wg.T)) @ wd
    assert np.abs(y - ref).max() <= 1e-12 * np.abs(ref).max()


@pytest.mark.parametrize("kind", ["quant", "none"])
@pytest.mark.parametrize("k_in", [1, 20, 64])
def test_full_channels_equal_dense_bitwise(oracle_lib, kind, k_in):
    cfg, wl, x = _tiny(seed=4, B=2)
    cg, sg = oracle_lib.quantize(wl.w_gate, cfg.dtype, 4, 32)
    cu, su = oracle_lib.quantize(wl.w_up, cfg.dtype, 4, 32)
    out = oracle_lib.ffn_sparse(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down, k_in,
                                cfg.d_ff, codes_g=cg, scales_g=sg, codes_u=cu,
                                scales_u=su, group=32,
                                kind=oracle_lib.PROXY_QUANT if kind == "quant"
                                else oracle_lib.PROXY_NONE)
    dense = oracle_lib.ffn_dense(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down)
    assert out["ff_idx"].tolist() == list(range(cfg.d_ff))
    assert np.array_equal(out["y"], dense)


# ---------------------------------------------------------------------------
# P2: fixed point = oracle-s (Sec. 3.1).  With an unquantised proxy and no
# input sparsity, s~ = s, so the mask is the exact top-k of |s|.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("B", [1, 3])
def test_fp_proxy_full_input_is_oracle_s(oracle_lib, B):
    cfg, wl, x = _tiny(seed=21, B=B, d=128, f=200)
    k_ff = 61
    out = oracle_lib.ffn_sparse(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down, cfg.d_model,
                                k_ff, kind=oracle_lib.PROXY_NONE)
    xf = _as_f64(x, cfg.dtype)
    wg, wu = _as_f64(wl.w_gate, cfg.dtype), _as_f64(wl.w_up, cfg.dtype)
    s = (xf @ wu.T) * _silu(xf @ wg.T)
    score = np.abs(s).max(axis=0)
    assert out["ff_idx"].tolist() == _brute_topk(list(score), k_ff)
    assert np.abs(out["score"] - score).max() <= 1e-12 * score.max()
    assert out["in_idx"].tolist() == list(range(cfg.d_model))


# ---------------------------------------------------------------------------
# P3: Stage 2 output is W_down applied to the masked s (Sec. 3.1 weighted sum).
# ---------------------------------------------------------------------------

def test_stage2_is_masked_weighted_sum(oracle_lib):
    cfg, wl, x = _tiny(seed=13, B=2, d=96, f=160)
    rng = np.random.default_rng(2)
    ff = np.sort(rng.choice(cfg.d_ff, 50, replace=False)).astype(np.int32)
    s_got, y = oracle_lib.stage2(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down, ff)
    xf = _as_f64(x, cfg.dtype)
    wg, wu, wd = (_as_f64(m, cfg.dtype) for m in (wl.w_gate, wl.w_up, wl.w_down))
    s = (xf @ wu.T) * _silu(xf @ wg.T)
    m = np.zeros(cfg.d_ff)
    m[ff] = 1.0
    ref = (s * m) @ wd
    assert np.abs(y - ref).max() <= 1e-12 * np.abs(ref).max()
    assert np.abs(s_got - s[:, ff]).max() <= 1e-12 * np.abs(s).max()


# ---------------------------------------------------------------------------
# Step 3 special case: a lossless quantised proxy equals the unquantised proxy,
# which is the input-sparse projection x[I] W[I, :] (Sec. 2.2 Pi_in).
# ---------------------------------------------------------------------------

def test_quant_proxy_lossless_equals_input_sparse_projection(oracle_lib):
    rng = np.random.default_rng(17)
    f, d, group = 50, 64, 16
    mats = []
    for _ in range(2):
        q = rng.integers(-7, 8, size=(f, d))
        q[:, ::group] = 7
        sig = 2.0 ** rng.integers(-9, -4, size=(f, d // group))
        mats.append(W.f32_to_bf16_bits((q * np.repeat(sig, group, axis=1)).astype(np.float32)))
    x = W.f32_to_bf16_bits(rng.laplace(size=(2, d)).astype(np.float32))
    I = np.sort(rng.choice(d, 23, replace=False)).astype(np.int32)
    cg, sg = oracle_lib.quantize(mats[0], W.DT_BF16, 4, group)
    cu, su = oracle_lib.quantize(mats[1], W.DT_BF16, 4, group)
    gq, uq, sq, scq = oracle_lib.proxy(x, W.DT_BF16, I, codes_g=cg, scales_g=sg, codes_u=cu,
                                       scales_u=su, group=group)
    gn, un, sn, scn = oracle_lib.proxy(x, W.DT_BF16, I, w_gate=mats[0], w_up=mats[1],
                                       kind=oracle_lib.PROXY_NONE)
    assert np.array_equal(gq, gn) and np.array_equal(uq, un) and np.array_equal(scq, scn)
    xf = _as_f64(x, W.DT_BF16)
    wgf, wuf = _as_f64(mats[0], W.DT_BF16), _as_f64(mats[1], W.DT_BF16)
    gref = xf[:, I] @ wgf[:, I].T
    uref = xf[:, I] @ wuf[:, I].T
    assert np.abs(gq - gref).max() <= 1e-12 * np.abs(gref).max()
    sref = _silu(gref) * uref
    assert np.abs(scq - np.abs(sref).max(axis=0)).max() <= 1e-12 * np.abs(sref).max()


def test_input_sparse_error_bound(oracle_lib):
    """Sec. 3.2: ||xW - x_sp W||_2 <= ||r||_2 ||W||_2 with the top-|x| input set."""
    cfg, wl, x = _tiny(seed=31, d=128, f=160)
    k = 40
    I = oracle_lib.select_inputs(x, cfg.dtype, k)
    g_t, _, _, _ = oracle_lib.proxy(x, cfg.dtype, I, w_gate=wl.w_gate, w_up=wl.w_up,
                                    kind=oracle_lib.PROXY_NONE)
    xf = _as_f64(x, cfg.dtype)[0]
    wg = _as_f64(wl.w_gate, cfg.dtype)
    g = wg @ xf
    r = xf.copy()
    r[I] = 0.0
    lhs = np.linalg.norm(g - g_t[0])
    assert lhs <= np.linalg.norm(r) * np.linalg.norm(wg, 2) * (1 + 1e-12)
    # and the kept set is the magnitude top-k, which minimises ||r||
    assert np.linalg.norm(r) <= np.sqrt(np.sort(xf ** 2)[: xf.size - k].sum()) * (1 + 1e-12)


# ---------------------------------------------------------------------------
# Statistical pins from App. A.2 at realistic size.
# ---------------------------------------------------------------------------

def _q_gauss(p):
    from scipy.stats import norm
    z = norm.ppf((1 + p) / 2)
    return 1 - p + 2 * z * norm.pdf(z)


def test_app_a2_closed_forms_match_printed_constants():
    g = _golden("paper_constants.json")
    p = 0.7
    a = -math.log(1 - p)
    q_lap = (1 - p) / 2 * (a * a + 2 * a + 2)
    # The paper prints three digits, not always rounded (eta = 0.46550 is
    # printed as 0.465), so agreement is to one unit in the last digit.
    ulp = 10.0 ** -g["printed_digits"]
    assert abs(q_lap - g["q_lap_p07"]["value"]) < ulp
    assert abs(_q_gauss(p) - g["q_gauss_p07"]["value"]) < ulp
    assert abs(math.sqrt(1 - _q_gauss(p)) - g["eta_p07"]["value"]) < ulp
    assert abs(math.sqrt(_q_gauss(p)) - g["corr_p07"]["value"]) < ulp


def test_laplace_energy_kept_by_topk(oracle_lib):
    """P7: top-30% by magnitude keeps q_Lap(0.7) = 0.879 of a Laplace vector's energy."""
    g = _golden("paper_constants.json")
    rng = np.random.default_rng(123)
    n = 28672
    vals = []
    for _ in range(4):
        s = rng.laplace(size=n)
        idx = oracle_lib.topk(np.abs(s), W.frac_to_k(0.3, n))
        vals.append((s[idx] ** 2).sum() / (s ** 2).sum())
    assert abs(np.mean(vals) - g["q_lap_p07"]["value"]) < 0.01


def test_gaussian_input_sparse_projection_stats(oracle_lib):
    """P6: with Gaussian x and weights and 70% input sparsity, the proxy
    correlates with the exact projection at sqrt(q_G(0.7)) = 0.885 and its
    relative RMS error is eta(0.7) = 0.465 (App. A.2)."""
    g = _golden("paper_constants.json")
    rng = np.random.default_rng(99)
    d, f, n_x = 4096, 8192, 6
    w = W.f32_to_bf16_bits((rng.standard_normal((f, d)) * 0.02).astype(np.float32))
    wf = _as_f64(w, W.DT_BF16)
    k = W.frac_to_k(0.3, d)
    corrs, etas = [], []
    for _ in range(n_x):
        x = W.f32_to_bf16_bits(rng.standard_normal((1, d)).astype(np.float32))
        I = oracle_lib.select_inputs(x, W.DT_BF16, k)
        g_t, _, _, _ = oracle_lib.proxy(x, W.DT_BF16, I, w_gate=w, w_up=w,
                                        kind=oracle_lib.PROXY_NONE)
        gx = wf @ _as_f64(x, W.DT_BF16)[0]
        corrs.append(np.corrcoef(gx, g_t[0])[0, 1])
        etas.append(np.sqrt(((gx - g_t[0]) ** 2).sum() / (gx ** 2).sum()))
    assert abs(np.mean(corrs) - g["corr_p07"]["value"]) < 0.01
    assert abs(np.mean(etas) - g["eta_p07"]["value"]) < 0.01


def test_proxy_mask_disagreements_sit_at_the_boundary(oracle_lib):
    """P8 (App. A.2 ranking condition): every channel where the proxy mask and
    the exact top-k disagree has ||s_j| - tau| <= 2 max_j ||s~_j| - |s_j||."""
    cfg = W.small_config(d=512, f=1024, seed=8, sigma_w=0.03, group=128)
    wl = W.make_workload(cfg)
    x = wl.x_vectors(1)[0]
    cg, sg = oracle_lib.quantize(wl.w_gate, cfg.dtype, 4, 128)
    cu, su = oracle_lib.quantize(wl.w_up, cfg.dtype, 4, 128)
    k_in, k_ff = 256, 307
    out = oracle_lib.ffn_sparse(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down, k_in, k_ff,
                                codes_g=cg, scales_g=sg, codes_u=cu, scales_u=su, group=128)
    xf = _as_f64(x, cfg.dtype)
    s = np.abs(((xf @ _as_f64(wl.w_up, cfg.dtype).T)
                * _silu(xf @ _as_f64(wl.w_gate, cfg.dtype).T))[0])
    exact = set(_brute_topk(list(s), k_ff))
    proxy = set(out["ff_idx"].tolist())
    tau = np.sort(s)[::-1][k_ff - 1]
    delta = np.abs(out["score"] - s).max()
    diff = exact ^ proxy
    assert len(diff) > 0            # the quantised, input-sparse proxy is not exact
    for j in diff:
        assert abs(s[j] - tau) <= 2 * delta * (1 + 1e-12)


def test_rmsnorm_definition(oracle_lib):
    rng = np.random.default_rng(4)
    x = W.f32_to_bf16_bits(rng.laplace(size=(2, 64)).astype(np.float32))
    y = W.f32_to_bf16_bits(rng.normal(size=(2, 64)).astype(np.float32))
    out = oracle_lib.add_rmsnorm(x, y, W.DT_BF16, 1e-6)
    r = _as_f64(x, W.DT_BF16) + _as_f64(y, W.DT_BF16)
    # unit gain: each row has mean square ms/(ms+eps) and the direction of r
    ms = (r ** 2).mean(axis=1)
    assert np.allclose((out ** 2).mean(axis=1), ms / (ms + 1e-6), rtol=1e-12)
    assert np.allclose(out * np.sqrt(ms + 1e-6)[:, None], r, rtol=1e-12, atol=0)
