"""GPU parity of the threshold-mode decode step (Sec. 4.1 masks with the
layer-wise threshold rule |z| >= tau of App. A.6) against the CPU oracle,
through the C-ABI entry point prox_ffn_sparse_tau.

Bars:
  * input mask: bit-exact (|x| >= tau_x is an exact fp32 comparison);
  * channel mask: exactly {j : gpu score_j >= tau_s}, and against the
    oracle's mask >= 99.9% agreement with every disagreement within 1e-3
    relative of tau_s;
  * proxy scores: |gpu - oracle| <= 1e-4 * max oracle score;
  * realised counts equal the masks' sizes;
  * y: max-abs-rel <= 2e-2 against the oracle on the GPU's mask.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2607_27591_amd import prox
from paper_2607_27591_amd import workloads as W

from gpu_cases import (MASK_AGREE, MASK_BAND, SCORE_TOL, Y_TOL, GpuOut, log, make_case,
                       run_sparse, y_rel_err)
from test_gpu_parity import SMALL

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", params=sorted(SMALL))
def case(request):
    cfg = SMALL[request.param]
    log(f"[tau case] {request.param}")
    c = make_case(cfg)
    yield c
    del c
    torch.cuda.empty_cache()


def run_tau(case, x_bits, tau_x, tau_s, ws=None):
    cfg = case.cfg
    x = prox.from_bits(np.atleast_2d(x_bits), cfg.dtype)
    in_mask = torch.empty(cfg.d_model, dtype=torch.uint8, device="cuda")
    scores = torch.empty(cfg.d_ff, dtype=torch.float32, device="cuda")
    y, mask, counts = prox.ffn_sparse_tau(case.w, case.proxy, x, tau_x, tau_s,
                                          in_mask=in_mask, scores=scores, ws=ws)
    torch.cuda.synchronize()
    return (GpuOut(prox.to_bits(y), mask.cpu().numpy(), in_mask.cpu().numpy(),
                   scores.cpu().numpy()), counts.cpu().numpy().tolist())


def quantile_taus(case, x_bits, s1=0.5, s2=0.7):
    """tau_x at the s1 order statistic of this input's a_i (an exact
    comparison, so ties at tau_x are exercised); tau_s halfway between the
    oracle's proxy scores around the s2 order statistic, so that no channel
    sits within fp32 rounding of it (fp32, as the entry point takes them)."""
    cfg = case.cfg
    a = np.abs(W.bits_to_f32(np.atleast_2d(x_bits), cfg.dtype)).max(axis=0)
    tau_x = float(np.sort(a)[min(a.size - 1, math.floor(s1 * a.size))])
    ref = oracle.ffn_sparse_tau(x_bits, cfg.dtype, case.wl.w_gate, case.wl.w_up, case.wl.w_down,
                                tau_x, math.inf, codes_g=case.codes_g, scales_g=case.scales_g,
                                codes_u=case.codes_u, scales_u=case.scales_u, group=cfg.group)
    sc = np.sort(ref["score"])
    pos = min(sc.size - 1, max(1, math.floor(s2 * sc.size)))
    tau_s = float(np.float32(0.5 * (sc[pos - 1] + sc[pos])))
    return tau_x, tau_s


def check_tau(case, x_bits, tau_x, tau_s, out, counts, tag=""):
    cfg = case.cfg
    x_bits = np.atleast_2d(x_bits)
    ref = oracle.ffn_sparse_tau(x_bits, cfg.dtype, case.wl.w_gate, case.wl.w_up, case.wl.w_down,
                                tau_x, tau_s, codes_g=case.codes_g, scales_g=case.scales_g,
                                codes_u=case.codes_u, scales_u=case.scales_u, group=cfg.group)
    # input mask: exact
    assert np.array_equal(np.flatnonzero(out.in_mask), ref["in_idx"]), f"{tag}: input mask"
    assert counts[0] == ref["k_in"], f"{tag}: k_in {counts[0]} vs {ref['k_in']}"
    # channel mask: the rule on the GPU's own scores, and its count
    gpu_sel = np.flatnonzero(out.scores >= np.float32(tau_s))
    assert np.array_equal(np.flatnonzero(out.mask), gpu_sel), f"{tag}: rule on GPU scores"
    assert counts[1] == int(out.mask.sum()), f"{tag}: k_ff count"
    # proxy scores
    smax = ref["score"].max()
    serr = np.abs(out.scores.astype(np.float64) - ref["score"]).max()
    assert serr <= SCORE_TOL * max(smax, 1e-30), f"{tag}: score err {serr}"
    # mask agreement with the oracle, disagreements at the threshold
    ref_mask = np.zeros(cfg.d_ff, np.uint8)
    ref_mask[ref["ff_idx"]] = 1
    diff = np.flatnonzero(ref_mask != out.mask)
    agree = 1.0 - diff.size / cfg.d_ff
    assert agree >= MASK_AGREE or diff.size == 0, f"{tag}: mask agreement {agree}"
    assert all(abs(ref["score"][j] - tau_s) <= MASK_BAND * max(tau_s, 1e-30) for j in diff), \
        f"{tag}: disagreement away from tau_s"
    # y on the GPU's mask
    gpu_ff = np.flatnonzero(out.mask).astype(np.int32)
    if gpu_ff.size == 0:
        assert not W.bits_to_f32(out.y, cfg.dtype).any(), f"{tag}: y must be 0"
        return {"k_in": counts[0], "k_ff": counts[1], "y_err": 0.0}
    _, y_ref = oracle.stage2(x_bits, cfg.dtype, case.wl.w_gate, case.wl.w_up, case.wl.w_down,
                             gpu_ff)
    yerr = y_rel_err(out.y, y_ref, cfg.dtype)
    assert yerr <= Y_TOL, f"{tag}: y max-abs-rel {yerr}"
    return {"k_in": counts[0], "k_ff": counts[1], "mask_agree": agree, "y_err": yerr}


def test_tau_parity(case):
    cfg = case.cfg
    xs = case.wl.x_vectors(2, cfg.batch)
    for v in range(2):
        for s1, s2 in ((0.5, 0.7), (0.2, 0.9)):
            tau_x, tau_s = quantile_taus(case, xs[v], s1, s2)
            log(f"[tau] {cfg.name} v{v} s1={s1} s2={s2} tau_x={tau_x:.4g} tau_s={tau_s:.4g}")
            out, counts = run_tau(case, xs[v], tau_x, tau_s)
            log(f"    {check_tau(case, xs[v], tau_x, tau_s, out, counts, tag=cfg.name)}")


def test_tau_zero_is_the_dense_ffn_bitwise(case):
    # Magnitudes are >= 0: tau = 0 keeps every input and channel, and the
    # channel split then matches the dense launch exactly.
    cfg = case.cfg
    x_bits = case.wl.x_vectors(1, cfg.batch)[0]
    log(f"[tau 0] {cfg.name}")
    out, counts = run_tau(case, x_bits, 0.0, 0.0)
    assert counts == [cfg.d_model, cfg.d_ff]
    assert out.in_mask.all() and out.mask.all()
    y_dense = prox.to_bits(prox.ffn_dense(case.w, prox.from_bits(np.atleast_2d(x_bits), cfg.dtype)))
    torch.cuda.synchronize()
    assert np.array_equal(out.y, y_dense)


def test_tau_infinite_keeps_nothing(case):
    cfg = case.cfg
    x_bits = case.wl.x_vectors(1, cfg.batch)[0]
    log(f"[tau inf] {cfg.name}")
    out, counts = run_tau(case, x_bits, math.inf, 1e-30)
    assert counts == [0, 0]
    assert not out.in_mask.any() and not out.mask.any() and not out.scores.any()
    assert not W.bits_to_f32(out.y, cfg.dtype).any()
    # no inputs: every score is 0, so tau_s = 0 keeps every channel
    out, counts = run_tau(case, x_bits, math.inf, 0.0)
    assert counts == [0, cfg.d_ff]


def _untied_k(desc, k):
    """The count nearest k whose k-th largest value differs from the next."""
    n = desc.size
    for dk in range(n):
        for kk in (k - dk, k + dk):
            if 1 <= kk <= n and (kk == n or desc[kk] != desc[kk - 1]):
                return kk
    return n


def test_tau_at_topk_values_matches_topk_bitwise(case):
    # Thresholds at the k-th largest a_i and the k-th largest GPU score pick
    # the same sets as the top-k entry point, so everything after matches.
    cfg = case.cfg
    x_bits = case.wl.x_vectors(1, cfg.batch)[0]
    a = np.abs(W.bits_to_f32(np.atleast_2d(x_bits), cfg.dtype)).max(axis=0)
    a_desc = np.sort(a)[::-1]
    k_in = _untied_k(a_desc, cfg.k_in)   # bf16 magnitudes tie often: move off a tie
    top = run_sparse(case, x_bits, k_in, cfg.k_ff)
    sc = np.sort(top.scores)[::-1]
    k_ff = _untied_k(sc, cfg.k_ff)
    if k_ff != cfg.k_ff:
        top = run_sparse(case, x_bits, k_in, k_ff)
    log(f"[tau=topk] {cfg.name} k_in={k_in} k_ff={k_ff}")
    out, counts = run_tau(case, x_bits, float(a_desc[k_in - 1]), float(sc[k_ff - 1]))
    assert counts[0] == k_in
    assert np.array_equal(out.in_mask, top.in_mask)
    fmt, d = case.proxy.fmt, cfg.d_model
    if (prox.stage1_mfma_rows(d, fmt, cfg.group, cfg.batch, k_in) > 0) != \
            (prox.stage1_mfma_rows(d, fmt, cfg.group, cfg.batch, d) > 0):
        # The threshold call's list (sized for every input) does not fit the
        # matrix-core kernel that the top-k call takes: same proxy, another
        # fp32 summation order, so the scores agree to the score tolerance
        # and only channels that close to tau_s may change sides.
        serr = np.abs(out.scores.astype(np.float64) - top.scores).max()
        assert serr <= SCORE_TOL * top.scores.max()
        assert counts[1] == int(out.mask.sum())
        band = np.abs(top.scores.astype(np.float64) - sc[k_ff - 1]) <= serr
        assert abs(counts[1] - k_ff) <= int(band.sum())
        return
    assert counts[1] == k_ff
    assert np.array_equal(out.scores.view(np.uint32), top.scores.view(np.uint32))
    assert np.array_equal(out.mask, top.mask)
    assert np.array_equal(out.y, top.y)


def test_tau_workspace_reuse_and_determinism():
    cfg = W.small_config(d=512, f=1100, batch=2, seed=23)
    c = make_case(cfg)
    ws = prox.new_workspace(cfg.d_model, cfg.d_ff, 16)
    for B in (1, 16, 3, 1):
        x_bits = c.wl.x_vectors(1, B)[0]
        tau_x, tau_s = quantile_taus(c, x_bits)
        log(f"[tau ws] B={B}")
        a, ca = run_tau(c, x_bits, tau_x, tau_s, ws=ws)
        b, cb = run_tau(c, x_bits, tau_x, tau_s, ws=ws)
        assert ca == cb and np.array_equal(a.y, b.y) and np.array_equal(a.mask, b.mask)
        check_tau(c, x_bits, tau_x, tau_s, a, ca, tag=f"B={B}")


@pytest.mark.slow
def test_tau_c4_full_size():
    # The 8192 x 28672 workload with thresholds at this input's 60% / 70%
    # order statistics (about the 40% / 30% kept fractions of the top-k runs).
    cfg = W.CONFIGS["c4_8192x28672_bf16"]
    log("[tau full] c4: generating and packing")
    c = make_case(cfg)
    x_bits = c.wl.x_vectors(1, 1)[0]
    tau_x, tau_s = quantile_taus(c, x_bits, 0.6, 0.7)
    out, counts = run_tau(c, x_bits, tau_x, tau_s)
    log(f"    {check_tau(c, x_bits, tau_x, tau_s, out, counts, tag='c4 tau')}")
    del c
    torch.cuda.empty_cache()
