"""The entry point that allocates nothing (prox_ffn_sparse_noalloc), called
through the C-ABI, against prox_ffn_sparse with a caller workspace: two calls
in a row, the second with a smaller input, each bitwise equal to the
workspace call (same kernels, deterministic) and within the oracle's parity
bar."""
import numpy as np
import pytest
import torch

from paper_2607_27591_amd import prox
from paper_2607_27591_amd import workloads as W

from gpu_cases import check_sparse, log, make_case, run_sparse

pytestmark = pytest.mark.gpu


def _noalloc(case, x_bits, k_in, k_ff):
    cfg = case.cfg
    x = prox.from_bits(np.atleast_2d(x_bits), cfg.dtype)
    in_mask = torch.empty(cfg.d_model, dtype=torch.uint8, device="cuda")
    scores = torch.empty(cfg.d_ff, dtype=torch.float32, device="cuda")
    y, mask = prox.ffn_sparse_noalloc(case.w, case.proxy, x, k_in, k_ff, in_mask=in_mask,
                                      scores=scores)
    torch.cuda.synchronize()
    return prox.to_bits(y), mask.cpu().numpy(), in_mask.cpu().numpy(), scores.cpu().numpy()


def _same(a, b, tag):
    y, mask, in_mask, scores = a
    assert np.array_equal(y, b.y), f"{tag}: y"
    assert np.array_equal(mask, b.mask), f"{tag}: mask"
    assert np.array_equal(in_mask, b.in_mask), f"{tag}: in_mask"
    assert np.array_equal(scores.view(np.uint32), b.scores.view(np.uint32)), f"{tag}: scores"


def test_noalloc_matches_workspace_call_twice():
    # 8192 x 28672 (the headline shape) at batch 2, then batch 1 on the same
    # scratch; then a smaller FFN on the same scratch.
    big = make_case(W.CONFIGS["c4_8192x28672_bf16"])
    cfg = big.cfg
    assert prox.workspace_bytes(cfg.d_model, cfg.d_ff, 2) <= prox.noalloc_max_bytes()
    for n, B in enumerate((2, 1)):
        x = big.wl.x_vectors(1, B)[0]
        log(f"[noalloc] call {n}: {cfg.name} batch {B}")
        got = _noalloc(big, x, cfg.k_in, cfg.k_ff)
        ref = run_sparse(big, x, cfg.k_in, cfg.k_ff)
        _same(got, ref, f"call {n}")
        log(f"    {check_sparse(big, x, cfg.k_in, cfg.k_ff, ref, tag=f'noalloc {n}')}")
    del big
    torch.cuda.empty_cache()
    small = make_case(W.small_config(d=1024, f=1600, batch=1, seed=31, in_frac=0.4,
                                     sigma_w=0.02))
    cfg = small.cfg
    x = small.wl.x_vectors(1, 1)[0]
    log("[noalloc] call 2: 1024 x 1600 batch 1")
    got = _noalloc(small, x, cfg.k_in, cfg.k_ff)
    ref = run_sparse(small, x, cfg.k_in, cfg.k_ff)
    _same(got, ref, "call 2")
    check_sparse(small, x, cfg.k_in, cfg.k_ff, ref, tag="noalloc 2")
