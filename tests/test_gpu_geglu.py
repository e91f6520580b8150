"""GPU parity of the GeGLU variant (gate activation GELU(z) = z Phi(z) in
both stages) against the oracle, with the bars of the SwiGLU tests."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_27591_amd import prox
from paper_2607_27591_amd import workloads as W

from gpu_cases import Y_TOL, check_sparse, log, make_case, run_sparse, y_rel_err

pytestmark = pytest.mark.gpu

CASES = {
    "bf16_i4_geglu_1024x1600_b1": W.small_config(d=1024, f=1600, batch=1, seed=41, sigma_w=0.02),
    "f16_i8_geglu_512x700_b2": W.small_config(d=512, f=700, batch=2, seed=42, dtype=W.DT_F16,
                                              qbits=8, group=512),
    "bf16_i4_geglu_2048x3000_b4": W.small_config(d=2048, f=3000, batch=4, seed=43, sigma_w=0.02),
    "bf16_i4_geglu_256x640_b16": W.small_config(d=256, f=640, batch=16, seed=44),
    "bf16_i4_geglu_4096x900_b16": W.small_config(d=4096, f=900, batch=16, seed=45,
                                                 sigma_w=0.02),
}


@pytest.fixture(scope="module", params=sorted(CASES))
def case(request):
    log(f"[geglu case] {request.param}")
    c = make_case(CASES[request.param], act=prox.GELU)
    yield c
    del c
    torch.cuda.empty_cache()


def test_geglu_sparse_parity(case):
    cfg = case.cfg
    for v, x in enumerate(case.wl.x_vectors(2, cfg.batch)):
        out = run_sparse(case, x, cfg.k_in, cfg.k_ff)
        log(f"    {check_sparse(case, x, cfg.k_in, cfg.k_ff, out, tag=f'{cfg.name}/{v}')}")


def test_geglu_dense_parity_and_full_sparse_equals_dense(case):
    cfg = case.cfg
    x = case.wl.x_vectors(1, cfg.batch)[0]
    xt = prox.from_bits(np.atleast_2d(x), cfg.dtype)
    y = prox.to_bits(prox.ffn_dense(case.w, xt))
    torch.cuda.synchronize()
    ref = oracle.ffn_dense(x, cfg.dtype, case.wl.w_gate, case.wl.w_up, case.wl.w_down,
                           act=oracle.GELU)
    assert y_rel_err(y, ref, cfg.dtype) <= Y_TOL
    out = run_sparse(case, x, cfg.k_in, cfg.d_ff)   # every channel kept
    assert np.array_equal(out.y, y)


def test_geglu_differs_from_swiglu(case):
    # the activation reaches both stages: scores and y change with it
    cfg = case.cfg
    x = case.wl.x_vectors(1, cfg.batch)[0]
    a = run_sparse(case, x, cfg.k_in, cfg.k_ff)
    silu = prox.Weights(case.w.w_gate, case.w.w_up, case.w.w_down)
    sc = torch.empty(cfg.d_ff, dtype=torch.float32, device="cuda")
    prox.ffn_sparse(silu, case.proxy, prox.from_bits(np.atleast_2d(x), cfg.dtype), cfg.k_in,
                    cfg.k_ff, scores=sc)
    torch.cuda.synchronize()
    assert not np.array_equal(a.scores, sc.cpu().numpy())
