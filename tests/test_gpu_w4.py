"""GPU parity of the INT4 base-weight (W4A16) Stage 2 against the oracle.

Stage 1 is the usual proxy path, so its checks are those of the 16-bit step:
input top-k bit-exact, the channel mask the exact top-k of the GPU's own
scores, the scores within the proxy tolerance.  Stage 2 reads the INT4 copy
of the three matrices (packed bit-exactly like the proxy, checked here), and
y is compared with the oracle's W4 Stage 2 on the GPU's own mask, to the same
2e-2 max-abs-rel bar.  Cases cover bf16 and fp16, SiLU and GeGLU, group 256,
and batches split over several Stage 2 launches (d_model 8192 takes 4 rows
per launch, 16384 takes 2; 24 rows at 8192 take six).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_27591_amd import prox
from paper_2607_27591_amd import workloads as W

from gpu_cases import SCORE_TOL, Y_TOL, check_selection, log, make_case, y_rel_err
from test_gpu_threshold import quantile_taus

pytestmark = pytest.mark.gpu

CASES = {
    "bf16_w4_1024x1600_b1": (W.small_config(d=1024, f=1600, batch=1, seed=71, in_frac=0.4,
                                            ff_frac=0.3, sigma_w=0.02), prox.SILU),
    "f16_w4_512x700_b2": (W.small_config(d=512, f=700, batch=2, seed=72, dtype=W.DT_F16,
                                         ff_frac=0.5), prox.SILU),
    # d / 8 = 80 output columns per thread group: the down projection's
    # thread groups do not line up with waves.
    "bf16_w4_640x900_b1": (W.small_config(d=640, f=900, batch=1, seed=78, in_frac=0.4,
                                          ff_frac=0.3, sigma_w=0.02), prox.SILU),
    # fp16 at one batch row (the one-row gate/up loop with fp16 codes), and
    # d / 8 = 144 columns per down thread group.
    "f16_w4_1152x800_b1": (W.small_config(d=1152, f=800, batch=1, seed=79, dtype=W.DT_F16,
                                          in_frac=0.4, ff_frac=0.3), prox.SILU),
    "bf16_w4_g256_2048x3000_b5": (W.small_config(d=2048, f=3000, batch=5, seed=73, group=256,
                                                 sigma_w=0.02), prox.SILU),
    "bf16_w4_geglu_1024x900_b3": (W.small_config(d=1024, f=900, batch=3, seed=74,
                                                 sigma_w=0.02), prox.GELU),
    "bf16_w4_8192x640_b7": (W.small_config(d=8192, f=640, batch=7, seed=75, in_frac=0.4,
                                           sigma_w=0.01), prox.SILU),
    "bf16_w4_8192x512_b24": (W.small_config(d=8192, f=512, batch=24, seed=77, in_frac=0.4,
                                            sigma_w=0.01), prox.SILU),
    "bf16_w4_16384x320_b3": (W.small_config(d=16384, f=320, batch=3, seed=76, in_frac=0.3,
                                            sigma_w=0.01), prox.SILU),
    # One batch row with the gate/up parts of the one-row loop: four parts of
    # 4096 columns (d 16384) and four uneven ones of 3072 (d 12288).
    "bf16_w4_16384x300_b1": (W.small_config(d=16384, f=300, batch=1, seed=80, in_frac=0.3,
                                            sigma_w=0.01), prox.SILU),
    "bf16_w4_12288x700_b1": (W.small_config(d=12288, f=700, batch=1, seed=81, in_frac=0.4,
                                            sigma_w=0.01), prox.GELU),
    # The largest batch a call takes: eight 8-row Stage 2 launches.
    "bf16_w4_1024x600_b64": (W.small_config(d=1024, f=600, batch=64, seed=82, in_frac=0.4,
                                            sigma_w=0.02), prox.SILU),
}


@pytest.fixture(scope="module", params=sorted(CASES))
def case(request):
    cfg, act = CASES[request.param]
    cfg = cfg.with_(name=request.param)
    log(f"[w4 case] {request.param}: d={cfg.d_model} f={cfg.d_ff} B={cfg.batch} "
        f"group={cfg.group} act={act}")
    c = make_case(cfg, act=act)
    q = prox.pack_w4(c.w, cfg.group)
    w4 = oracle.quantize_w4(c.wl.w_gate, c.wl.w_up, c.wl.w_down, cfg.dtype, cfg.group)
    yield c, q, w4
    del c, q
    torch.cuda.empty_cache()


def _run_w4(c, q, x_bits, k_in, k_ff):
    cfg = c.cfg
    x = prox.from_bits(np.atleast_2d(x_bits), cfg.dtype)
    in_mask = torch.empty(cfg.d_model, dtype=torch.uint8, device="cuda")
    scores = torch.empty(cfg.d_ff, dtype=torch.float32, device="cuda")
    y, mask = prox.ffn_sparse_w4(q, c.proxy, x, k_in, k_ff, in_mask=in_mask, scores=scores)
    torch.cuda.synchronize()
    return prox.to_bits(y), mask.cpu().numpy(), in_mask.cpu().numpy(), scores.cpu().numpy()


def test_w4_pack_bit_exact(case):
    c, q, w4 = case
    for m, key in enumerate(("g", "u", "d")):
        codes, scales = prox.unpack_w4(q, m)
        torch.cuda.synchronize()
        assert np.array_equal(codes.cpu().numpy(), w4["codes_" + key]), f"codes {key}"
        assert np.array_equal(scales.cpu().numpy().view(np.uint16), w4["scales_" + key]), \
            f"scales {key}"


def test_w4_sparse_parity(case):
    c, q, w4 = case
    cfg = c.cfg
    for v, x in enumerate(c.wl.x_vectors(2, cfg.batch)):
        out = _run_w4(c, q, x, cfg.k_in, cfg.k_ff)
        stats = _check_w4(c, w4, x, cfg.k_in, cfg.k_ff, out, f"v{v}")
        log(f"    v{v}: {stats}")


def test_w4_dense_parity_and_full_keep(case):
    c, q, w4 = case
    cfg = c.cfg
    x_bits = c.wl.x_vectors(1, cfg.batch)[0]
    x = prox.from_bits(np.atleast_2d(x_bits), cfg.dtype)
    y_dense = prox.to_bits(prox.ffn_dense_w4(q, x))
    y_ref = oracle.ffn_dense_w4(x_bits, cfg.dtype, w4, c.act)
    err = y_rel_err(y_dense, y_ref, cfg.dtype)
    log(f"    dense W4: y max-abs-rel {err:.2e}")
    assert err <= Y_TOL
    # Keeping every input and channel runs the dense channel split: bitwise.
    y_full, mask, _, _ = _run_w4(c, q, x_bits, cfg.d_model, cfg.d_ff)
    assert mask.all()
    assert np.array_equal(y_full, y_dense)


def _check_w4(c, w4, x_bits, k_in, k_ff, out, tag):
    """The selection bar of the 16-bit step (input top-k exact, the mask the
    top-k of the GPU's scores, scores, mask agreement with the oracle's and
    its band), then y against the oracle's W4 Stage 2 on the GPU's mask."""
    cfg = c.cfg
    y, mask, in_mask, scores = out
    ref = oracle.ffn_sparse_w4(x_bits, cfg.dtype, w4, k_in, k_ff, codes_g=c.codes_g,
                               scales_g=c.scales_g, codes_u=c.codes_u, scales_u=c.scales_u,
                               group=cfg.group, act=c.act)
    stats = check_selection(ref, in_mask, mask, scores, k_ff, tag)
    gpu_sel = np.flatnonzero(mask).astype(np.int32)
    _, y_ref = oracle.stage2_w4(x_bits, cfg.dtype, w4, gpu_sel, c.act)
    err = y_rel_err(y, y_ref, cfg.dtype)
    assert err <= Y_TOL, f"{tag}: y err {err}"
    stats["y_err"] = err
    return stats


def test_w4_extreme_k(case):
    c, q, w4 = case
    cfg = c.cfg
    x = c.wl.x_vectors(1, cfg.batch)[0]
    for k_in, k_ff in [(1, 1), (1, cfg.d_ff), (cfg.d_model, 1), (cfg.d_model // 2 + 1, cfg.d_ff - 1)]:
        log(f"[w4 extreme] {cfg.name} k_in={k_in} k_ff={k_ff}")
        _check_w4(c, w4, x, k_in, k_ff, _run_w4(c, q, x, k_in, k_ff), f"k_in={k_in} k_ff={k_ff}")


def test_w4_zero_input(case):
    # All magnitudes tie at zero: the lowest indices are kept, and y is 0.
    c, q, w4 = case
    cfg = c.cfg
    x = np.zeros((cfg.batch, cfg.d_model), np.uint16)
    k_in, k_ff = min(100, cfg.d_model), min(200, cfg.d_ff)
    y, mask, in_mask, scores = _run_w4(c, q, x, k_in, k_ff)
    assert np.flatnonzero(in_mask).tolist() == list(range(k_in))
    assert np.flatnonzero(mask).tolist() == list(range(k_ff))
    assert not scores.any()
    assert not W.bits_to_f32(y, cfg.dtype).any()


def _check_w4_tau(c, q, w4, x_bits):
    """Thresholds in place of counts (prox_ffn_sparse_tau_w4): the masks follow
    the rule exactly on the GPU's own values, y is the oracle's W4 Stage 2 on
    the GPU's mask."""
    cfg = c.cfg
    tau_x, tau_s = quantile_taus(c, x_bits)
    x = prox.from_bits(np.atleast_2d(x_bits), cfg.dtype)
    in_mask = torch.empty(cfg.d_model, dtype=torch.uint8, device="cuda")
    scores = torch.empty(cfg.d_ff, dtype=torch.float32, device="cuda")
    y, mask, counts = prox.ffn_sparse_tau_w4(q, c.proxy, x, tau_x, tau_s, in_mask=in_mask,
                                             scores=scores)
    torch.cuda.synchronize()
    y, mask, counts = prox.to_bits(y), mask.cpu().numpy(), counts.cpu().numpy().tolist()
    in_mask, scores = in_mask.cpu().numpy(), scores.cpu().numpy()
    ref = oracle.ffn_sparse_tau(x_bits, cfg.dtype, c.wl.w_gate, c.wl.w_up, c.wl.w_down, tau_x,
                                tau_s, codes_g=c.codes_g, scales_g=c.scales_g, codes_u=c.codes_u,
                                scales_u=c.scales_u, group=cfg.group, act=c.act)
    assert np.array_equal(np.flatnonzero(in_mask), ref["in_idx"])
    assert counts[0] == ref["k_in"]
    gpu_sel = np.flatnonzero(scores >= np.float32(tau_s))
    assert np.array_equal(np.flatnonzero(mask), gpu_sel)
    assert counts[1] == gpu_sel.size
    serr = np.abs(scores.astype(np.float64) - ref["score"]).max()
    assert serr <= SCORE_TOL * ref["score"].max()
    _, y_ref = oracle.stage2_w4(x_bits, cfg.dtype, w4, gpu_sel.astype(np.int32), c.act)
    err = y_rel_err(y, y_ref, cfg.dtype)
    log(f"    tau W4: k_in {counts[0]} k_ff {counts[1]} y max-abs-rel {err:.2e}")
    assert err <= Y_TOL


def test_w4_threshold_mode(case):
    c, q, w4 = case
    _check_w4_tau(c, q, w4, c.wl.x_vectors(1, c.cfg.batch)[0])


def test_w4_staged_entry_point(case):
    from test_gpu_parity import check_staged
    c, q, w4 = case
    cfg = c.cfg
    x = prox.from_bits(np.atleast_2d(c.wl.x_vectors(1, cfg.batch)[0]), cfg.dtype)
    log(f"[w4 staged] {cfg.name}")
    check_staged(lambda ev: prox.ffn_sparse_w4(q, c.proxy, x, cfg.k_in, cfg.k_ff, events=ev),
                 cfg.name)


def test_w4_c4_full_size():
    cfg = W.CONFIGS["c4_8192x28672_bf16"]
    log("[w4 full] c4: generating and packing")
    c = make_case(cfg)
    q = prox.pack_w4(c.w, cfg.group)
    w4 = oracle.quantize_w4(c.wl.w_gate, c.wl.w_up, c.wl.w_down, cfg.dtype, cfg.group)
    x = c.wl.x_vectors(1, 1)[0]
    stats = _check_w4(c, w4, x, cfg.k_in, cfg.k_ff, _run_w4(c, q, x, cfg.k_in, cfg.k_ff), "c4 W4")
    log(f"    c4 W4: {stats}")
    log("[w4 full] c4 threshold mode")
    _check_w4_tau(c, q, w4, x)
    del c, q
    torch.cuda.empty_cache()
