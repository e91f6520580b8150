"""Shared helpers of the GPU parity tests: run the HIP path through the C-ABI
binding and check it against the CPU oracle on the same seeded inputs.

Parity bars (the sparse decode step's contract):
  * input top-k indices: bit-exact (ties to the lower index);
  * channel selection on the GPU's own scores: bit-exact top-k of those scores;
  * proxy scores: |gpu - oracle| <= 1e-4 * max oracle score;
  * channel mask vs the oracle's: >= 99.9% of channels agree, and every
    disagreement lies within 1e-3 relative of the oracle's k-th score;
  * y: per batch row, max|y_gpu - y_oracle| / max|y_oracle| <= 2e-2, the
    oracle evaluated on the GPU's mask.
"""
from __future__ import annotations

import dataclasses
import sys
from typing import Optional

import numpy as np
import torch

import oracle
from paper_2607_27591_amd import prox
from paper_2607_27591_amd import workloads as W

SCORE_TOL = 1e-4
MASK_AGREE = 0.999
MASK_BAND = 1e-3
Y_TOL = 2e-2


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


@dataclasses.dataclass
class Case:
    cfg: W.FFNConfig
    wl: W.Workload
    w: prox.Weights
    proxy: prox.Proxy
    codes_g: np.ndarray
    scales_g: np.ndarray
    codes_u: np.ndarray
    scales_u: np.ndarray
    act: int = prox.SILU


def make_case(cfg: W.FFNConfig, device="cuda", act: int = prox.SILU) -> Case:
    wl = W.make_workload(cfg)
    w = prox.Weights(*(prox.from_bits(m, cfg.dtype, device) for m in (wl.w_gate, wl.w_up, wl.w_down)),
                     act=act)
    fmt = prox.INT4 if cfg.qbits == 4 else prox.INT8
    p = prox.pack_proxy(w, fmt, cfg.group)
    cg, sg = oracle.quantize(wl.w_gate, cfg.dtype, cfg.qbits, cfg.group)
    cu, su = oracle.quantize(wl.w_up, cfg.dtype, cfg.qbits, cfg.group)
    return Case(cfg, wl, w, p, cg, sg, cu, su, act)


def check_pack(case: Case) -> None:
    cfg = case.cfg
    cg, sg, cu, su = prox.unpack_proxy(case.proxy, cfg.d_model, cfg.d_ff)
    torch.cuda.synchronize()
    assert np.array_equal(cg.cpu().numpy(), case.codes_g), "gate codes differ"
    assert np.array_equal(cu.cpu().numpy(), case.codes_u), "up codes differ"
    assert np.array_equal(sg.cpu().numpy().view(np.uint16), case.scales_g), "gate scales differ"
    assert np.array_equal(su.cpu().numpy().view(np.uint16), case.scales_u), "up scales differ"


@dataclasses.dataclass
class GpuOut:
    y: np.ndarray        # uint16 [B][d]
    mask: np.ndarray     # uint8 [f]
    in_mask: np.ndarray  # uint8 [d]
    scores: np.ndarray   # float32 [f]


def run_sparse(case: Case, x_bits: np.ndarray, k_in: int, k_ff: int,
               ws: Optional[torch.Tensor] = None) -> GpuOut:
    cfg = case.cfg
    x = prox.from_bits(np.atleast_2d(x_bits), cfg.dtype)
    in_mask = torch.empty(cfg.d_model, dtype=torch.uint8, device="cuda")
    scores = torch.empty(cfg.d_ff, dtype=torch.float32, device="cuda")
    y, mask = prox.ffn_sparse(case.w, case.proxy, x, k_in, k_ff, in_mask=in_mask, scores=scores,
                              ws=ws)
    torch.cuda.synchronize()
    return GpuOut(prox.to_bits(y), mask.cpu().numpy(), in_mask.cpu().numpy(),
                  scores.cpu().numpy())


def y_rel_err(y_bits: np.ndarray, y_ref: np.ndarray, dtype: int) -> float:
    y = W.bits_to_f32(y_bits, dtype).astype(np.float64).reshape(y_ref.shape)
    worst = 0.0
    for b in range(y_ref.shape[0]):
        den = np.abs(y_ref[b]).max()
        num = np.abs(y[b] - y_ref[b]).max()
        worst = max(worst, num / den if den > 0 else num)
    return worst


def check_selection(ref: dict, in_mask: np.ndarray, mask: np.ndarray, scores: np.ndarray,
                    k_ff: int, tag: str = "") -> dict:
    """Steps (a)-(d) of the parity bar, against the oracle's run `ref` (its
    in_idx, score and ff_idx): input top-k bit-exact, the channel mask the
    exact top-k of the GPU's own scores, scores to SCORE_TOL of the largest,
    and the mask agreeing with the oracle's on MASK_AGREE of the channels with
    every disagreement inside the MASK_BAND of the oracle's k-th score."""
    f = mask.size
    # (a) input top-k, bit-exact
    assert np.array_equal(np.flatnonzero(in_mask), ref["in_idx"]), f"{tag}: input top-k"
    # (b) channel selection is the exact top-k of the GPU's own scores
    gpu_sel = oracle.topk(scores.astype(np.float64), k_ff)
    assert np.array_equal(np.flatnonzero(mask), gpu_sel), f"{tag}: select on GPU scores"
    assert int(mask.sum()) == k_ff
    # (c) proxy scores
    smax = ref["score"].max()
    serr = np.abs(scores.astype(np.float64) - ref["score"]).max()
    assert serr <= SCORE_TOL * max(smax, 1e-30), f"{tag}: score err {serr} vs max {smax}"
    # (d) mask agreement with the oracle's selection
    ref_mask = np.zeros(f, np.uint8)
    ref_mask[ref["ff_idx"]] = 1
    diff = np.flatnonzero(ref_mask != mask)
    agree = 1.0 - diff.size / f
    tau = np.sort(ref["score"])[::-1][k_ff - 1]
    band_ok = all(abs(ref["score"][j] - tau) <= MASK_BAND * tau for j in diff)
    assert agree >= MASK_AGREE or diff.size == 0, f"{tag}: mask agreement {agree}"
    assert band_ok, f"{tag}: mask disagreement outside the 1e-3 band"
    return {"score_err_rel": serr / max(smax, 1e-30), "mask_agree": agree,
            "mask_diff": int(diff.size)}


def check_sparse(case: Case, x_bits: np.ndarray, k_in: int, k_ff: int, out: GpuOut,
                 tag: str = "") -> dict:
    cfg = case.cfg
    x_bits = np.atleast_2d(x_bits)
    ref = oracle.ffn_sparse(x_bits, cfg.dtype, case.wl.w_gate, case.wl.w_up, case.wl.w_down,
                            k_in, k_ff, codes_g=case.codes_g, scales_g=case.scales_g,
                            codes_u=case.codes_u, scales_u=case.scales_u, group=cfg.group,
                            act=case.act)
    stats = check_selection(ref, out.in_mask, out.mask, out.scores, k_ff, tag)
    # (e) y against the oracle on the GPU's mask
    gpu_ff = np.flatnonzero(out.mask).astype(np.int32)
    _, y_ref = oracle.stage2(x_bits, cfg.dtype, case.wl.w_gate, case.wl.w_up, case.wl.w_down,
                             gpu_ff, act=case.act)
    yerr = y_rel_err(out.y, y_ref, cfg.dtype)
    assert yerr <= Y_TOL, f"{tag}: y max-abs-rel {yerr}"
    stats["y_err"] = yerr
    return stats
