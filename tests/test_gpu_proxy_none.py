"""GPU parity of the unquantised 16-bit proxy (PROX_Q_NONE: W~ = W, the
proxy ablation; also the reference of the proxy-cost ratio alpha, Sec. 4.2)
against the oracle's unquantised proxy, and the paper's fixed point: with no
input sparsity the proxy intermediate is the exact s, so the channel mask is
the exact top-k of |s| (Sec. 3.1 oracle-s)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_27591_amd import prox
from paper_2607_27591_amd import workloads as W

from gpu_cases import (MASK_AGREE, MASK_BAND, SCORE_TOL, Y_TOL, log, run_sparse, y_rel_err)

pytestmark = pytest.mark.gpu

CASES = {
    "bf16_none_512x700_b2": W.small_config(d=512, f=700, batch=2, seed=31),
    "f16_none_384x520_b1": W.small_config(d=384, f=520, batch=1, seed=32, dtype=W.DT_F16),
    "bf16_none_2048x3000_b4": W.small_config(d=2048, f=3000, batch=4, seed=33, sigma_w=0.02),
    "bf16_none_8192x640_b1": W.small_config(d=8192, f=640, batch=1, seed=34, sigma_w=0.01),
}


class _Case:
    def __init__(self, cfg):
        self.cfg = cfg
        self.wl = W.make_workload(cfg)
        self.w = prox.Weights(*(prox.from_bits(m, cfg.dtype) for m in
                                (self.wl.w_gate, self.wl.w_up, self.wl.w_down)))
        self.proxy = prox.pack_proxy(self.w, prox.NONE)


@pytest.fixture(scope="module", params=sorted(CASES))
def case(request):
    log(f"[none case] {request.param}")
    c = _Case(CASES[request.param])
    yield c
    del c
    torch.cuda.empty_cache()


def _check(c, x, k_in, k_ff, tag):
    cfg = c.cfg
    out = run_sparse(c, x, k_in, k_ff)
    ref = oracle.ffn_sparse(x, cfg.dtype, c.wl.w_gate, c.wl.w_up, c.wl.w_down, k_in, k_ff,
                            kind=oracle.PROXY_NONE)
    assert np.array_equal(np.flatnonzero(out.in_mask), ref["in_idx"]), f"{tag}: input top-k"
    assert np.array_equal(np.flatnonzero(out.mask),
                          oracle.topk(out.scores.astype(np.float64), k_ff)), f"{tag}: selection"
    smax = ref["score"].max()
    serr = np.abs(out.scores.astype(np.float64) - ref["score"]).max()
    assert serr <= SCORE_TOL * smax, f"{tag}: score err {serr / smax}"
    ref_mask = np.zeros(cfg.d_ff, np.uint8)
    ref_mask[ref["ff_idx"]] = 1
    diff = np.flatnonzero(ref_mask != out.mask)
    kth = np.sort(ref["score"])[::-1][k_ff - 1]
    assert 1 - diff.size / cfg.d_ff >= MASK_AGREE or diff.size == 0, f"{tag}: mask agreement"
    assert all(abs(ref["score"][j] - kth) <= MASK_BAND * kth for j in diff), f"{tag}: band"
    _, y_ref = oracle.stage2(x, cfg.dtype, c.wl.w_gate, c.wl.w_up, c.wl.w_down,
                             np.flatnonzero(out.mask).astype(np.int32))
    assert y_rel_err(out.y, y_ref, cfg.dtype) <= Y_TOL, f"{tag}: y"
    return out, ref


def test_none_proxy_parity(case):
    cfg = case.cfg
    for v, x in enumerate(case.wl.x_vectors(2, cfg.batch)):
        log(f"[none] {cfg.name} v{v}")
        _check(case, x, cfg.k_in, cfg.k_ff, f"{cfg.name}/{v}")


def test_none_proxy_full_input_is_oracle_s(case):
    # k_in = d and W~ = W: the score is max_b |s_{b,j}| of the exact FFN, so
    # the mask must be (to the fp32 band) the exact top-k of |s|.
    cfg = case.cfg
    x = case.wl.x_vectors(1, cfg.batch)[0]
    out, _ = _check(case, x, cfg.d_model, cfg.k_ff, f"{cfg.name}/full")
    s, _ = oracle.stage2(x, cfg.dtype, case.wl.w_gate, case.wl.w_up, case.wl.w_down,
                         np.arange(cfg.d_ff, dtype=np.int32))
    exact = np.abs(s).max(axis=0)
    assert np.abs(out.scores - exact).max() <= SCORE_TOL * exact.max()
    top = oracle.topk(exact, cfg.k_ff)
    kth = np.sort(exact)[::-1][cfg.k_ff - 1]
    diff = np.setxor1d(np.flatnonzero(out.mask), top)
    assert all(abs(exact[j] - kth) <= MASK_BAND * kth for j in diff)
