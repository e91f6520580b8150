"""GPU parity at the full sizes of the synthetic workloads, in the launch
configuration the benchmark times (the same prox_ffn_sparse call).  The CPU
oracle is fast enough to evaluate every output at these sizes."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_27591_amd import prox
from paper_2607_27591_amd import workloads as W

from gpu_cases import Y_TOL, check_pack, check_sparse, log, make_case, run_sparse, y_rel_err

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _ties(case, batch, tag):
    """All-tied and equal-magnitude inputs at full size: every selection
    breaks its ties by the lower index (App. A.6), here with d_ff score keys
    per call (above 16384 the channel top-k takes its 12-bit first pass)."""
    cfg = case.cfg
    k_in, k_ff = cfg.k_in, cfg.k_ff
    x = np.zeros((batch, cfg.d_model), np.uint16)
    x[batch - 1, 1::2] = 0x8000   # -0 ties with +0
    log(f"[full] {tag} zero input B={batch}")
    out = run_sparse(case, x, k_in, k_ff)
    assert np.flatnonzero(out.in_mask).tolist() == list(range(k_in))
    assert np.flatnonzero(out.mask).tolist() == list(range(k_ff))
    assert not out.scores.any()
    assert not W.bits_to_f32(out.y, cfg.dtype).any()
    rng = np.random.default_rng(7)
    v = rng.choice([-0.75, 0.75], size=(batch, cfg.d_model)).astype(np.float32)
    v[:, k_in + 5:] = 0.125       # the cut falls inside a run of equal magnitudes
    xe = W.to_bits(v, cfg.dtype)
    log(f"[full] {tag} equal magnitudes B={batch}")
    out = run_sparse(case, xe, k_in, k_ff)
    assert np.flatnonzero(out.in_mask).tolist() == list(range(k_in))
    log(f"    {check_sparse(case, xe, k_in, k_ff, out, tag=f'{tag} equal magnitudes')}")


def _full(name, n_vectors, dense=True):
    cfg = W.CONFIGS[name]
    log(f"[full] {name}: generating and packing")
    case = make_case(cfg)
    check_pack(case)
    xs = case.wl.x_vectors(n_vectors, cfg.batch)
    for n, x in enumerate(xs):
        log(f"[full] {name} vector {n}")
        out = run_sparse(case, x, cfg.k_in, cfg.k_ff)
        log(f"    {check_sparse(case, x, cfg.k_in, cfg.k_ff, out, tag=f'{name}/{n}')}")
    _ties(case, cfg.batch, name)
    if dense:
        log(f"[full] {name} dense")
        y = prox.ffn_dense(case.w, prox.from_bits(xs[0], cfg.dtype))
        torch.cuda.synchronize()
        ref = oracle.ffn_dense(xs[0], cfg.dtype, case.wl.w_gate, case.wl.w_up, case.wl.w_down)
        err = y_rel_err(prox.to_bits(y), ref, cfg.dtype)
        log(f"    dense y err {err:.3e}")
        assert err <= Y_TOL
    del case
    torch.cuda.empty_cache()


def test_c1_1024x3072_f16_int8():
    _full("c1_1024x3072_f16", 8)


def test_c2_4096x12288_bf16():
    _full("c2_4096x12288_bf16", 4)


def test_c4_8192x28672_bf16():
    _full("c4_8192x28672_bf16", 3)


@pytest.mark.parametrize("batch", [1, 6])
def test_c2_per_row_int4_proxy(batch):
    """The paper's own proxy format, symmetric INT4 with one scale per output
    channel (group = d_model), at the Qwen3-8B FFN shape: batch 1 on the
    dot-product Stage 1, batch 6 on the matrix-core Stage 1."""
    cfg = W.CONFIGS["c2_4096x12288_bf16"].with_(group=4096, batch=batch,
                                                 name=f"c2_per_row_int4_b{batch}")
    mfma = prox.stage1_mfma_rows(cfg.d_model, prox.INT4, cfg.group, batch, cfg.k_in)
    assert (mfma > 0) == (batch >= 3), mfma
    log(f"[full] {cfg.name}: generating and packing")
    case = make_case(cfg)
    check_pack(case)
    for n, x in enumerate(case.wl.x_vectors(2, batch)):
        out = run_sparse(case, x, cfg.k_in, cfg.k_ff)
        log(f"    {check_sparse(case, x, cfg.k_in, cfg.k_ff, out, tag=f'{cfg.name}/{n}')}")
    del case
    torch.cuda.empty_cache()


def test_max_dff_matrix_core_stage2():
    """d_ff 65536 with 9 batch rows on the matrix-core Stage 2: 64 score keys
    per thread in its selection, 1024 channels per down group (the down
    kernel's largest LDS), and the dense FFN over every channel; full keep
    equals dense bitwise."""
    cfg = W.small_config(d=4096, f=65536, batch=9, seed=20, in_frac=0.5, ff_frac=0.2,
                         sigma_w=0.02)
    assert prox.stage2_rows(cfg.d_model, cfg.d_ff, False, cfg.batch) == 16
    log("[full] 4096x65536 b9: generating and packing")
    case = make_case(cfg)
    x = case.wl.x_vectors(1, cfg.batch)[0]
    out = run_sparse(case, x, cfg.k_in, cfg.k_ff)
    log(f"    {check_sparse(case, x, cfg.k_in, cfg.k_ff, out, tag='4096x65536 b9')}")
    y = prox.to_bits(prox.ffn_dense(case.w, prox.from_bits(x, cfg.dtype)))
    torch.cuda.synchronize()
    ref = oracle.ffn_dense(x, cfg.dtype, case.wl.w_gate, case.wl.w_up, case.wl.w_down)
    err = y_rel_err(y, ref, cfg.dtype)
    log(f"    dense y err {err:.3e}")
    assert err <= Y_TOL
    full = run_sparse(case, x, cfg.d_model, cfg.d_ff)
    assert full.mask.all() and np.array_equal(full.y, y)
    del case
    torch.cuda.empty_cache()


def test_max_shape_d16384_f65536():
    """Both maxima in one call at batch 1: d_model 16384 (16 input rows per
    thread in the proxy's selection) with d_ff 65536 (64 score keys per
    thread in Stage 2's). Packing, sparse and dense parity, full keep equal
    to dense bitwise, then the INT4 base-weight Stage 2 at the same shape."""
    from test_gpu_w4 import _check_w4, _run_w4
    cfg = W.small_config(d=16384, f=65536, batch=1, seed=26, in_frac=0.4, ff_frac=0.3,
                         sigma_w=0.01)
    log("[full] 16384x65536 b1: generating and packing")
    case = make_case(cfg)
    check_pack(case)
    x = case.wl.x_vectors(1, 1)[0]
    out = run_sparse(case, x, cfg.k_in, cfg.k_ff)
    log(f"    {check_sparse(case, x, cfg.k_in, cfg.k_ff, out, tag='16384x65536')}")
    y = prox.to_bits(prox.ffn_dense(case.w, prox.from_bits(x, cfg.dtype)))
    torch.cuda.synchronize()
    ref = oracle.ffn_dense(x, cfg.dtype, case.wl.w_gate, case.wl.w_up, case.wl.w_down)
    err = y_rel_err(y, ref, cfg.dtype)
    log(f"    dense y err {err:.3e}")
    assert err <= Y_TOL
    full = run_sparse(case, x, cfg.d_model, cfg.d_ff)
    assert full.mask.all() and np.array_equal(full.y, y)
    log("[full] 16384x65536 b1: INT4 base weights")
    q = prox.pack_w4(case.w, cfg.group)
    w4 = oracle.quantize_w4(case.wl.w_gate, case.wl.w_up, case.wl.w_down, cfg.dtype, cfg.group)
    stats = _check_w4(case, w4, x, cfg.k_in, cfg.k_ff, _run_w4(case, q, x, cfg.k_in, cfg.k_ff),
                      "16384x65536 W4")
    log(f"    W4: {stats}")
    del case, q, w4
    torch.cuda.empty_cache()


@pytest.fixture(scope="module")
def c3_case():
    cfg = W.CONFIGS["c3_4096x14336_bf16"]
    log("[full] c3: generating and packing")
    c = make_case(cfg)
    yield c
    del c
    torch.cuda.empty_cache()


@pytest.mark.parametrize("batch,sparsity", [(1, 0.0), (1, 0.5), (1, 0.7), (1, 0.9),
                                            (4, 0.0), (4, 0.5), (4, 0.7), (4, 0.9),
                                            (5, 0.7), (8, 0.7),
                                            (16, 0.0), (16, 0.5), (16, 0.7), (16, 0.9)])
def test_c3_batch_sparsity_sweep(c3_case, batch, sparsity):
    cfg = c3_case.cfg
    k_ff = W.frac_to_k(1.0 - sparsity, cfg.d_ff)
    x = c3_case.wl.x_vectors(1, batch)[0]
    log(f"[full] c3 B={batch} sparsity={sparsity} k_ff={k_ff}")
    out = run_sparse(c3_case, x, cfg.k_in, k_ff)
    log(f"    {check_sparse(c3_case, x, cfg.k_in, k_ff, out, tag=f'c3 B={batch} s={sparsity}')}")


@pytest.mark.parametrize("batch", [1, 4, 16])
def test_c3_threshold_mode(c3_case, batch):
    """The threshold rule at full size on each Stage 1 and Stage 2 path: its
    kept-row list holds up to d rows, so the matrix-core Stage 1 takes 8 rows
    per launch here (two launches at 16 rows)."""
    from test_gpu_threshold import check_tau, quantile_taus, run_tau
    x = c3_case.wl.x_vectors(1, batch)[0]
    tau_x, tau_s = quantile_taus(c3_case, x)
    log(f"[full] c3 threshold mode B={batch}")
    out, counts = run_tau(c3_case, x, tau_x, tau_s)
    log(f"    {check_tau(c3_case, x, tau_x, tau_s, out, counts, tag=f'c3 tau B={batch}')}")


@pytest.mark.parametrize("batch", [4, 16])
def test_c3_ties(c3_case, batch):
    """Ties on the dot-product (4 rows) and matrix-core (16 rows) paths."""
    _ties(c3_case, batch, f"c3 B={batch}")


def test_c5_stack_teacher_forced():
    """First layers of the 36-layer stack, each checked on the GPU's own input
    x_l (masks may legitimately diverge over many layers), then the residual
    RMSNorm x_{l+1} = RMSNorm(x_l + y_l) checked against the oracle."""
    base = W.stack_layer_config(0)
    x_bits = W.make_workload(base, weights=False).x_vectors(1, 1)[0]
    x = prox.from_bits(x_bits, base.dtype)
    for layer in range(3):
        cfg = W.stack_layer_config(layer)
        log(f"[full] c5 layer {layer}")
        case = make_case(cfg)
        xb = prox.to_bits(x)
        out = run_sparse(case, xb, cfg.k_in, cfg.k_ff)
        check_sparse(case, xb, cfg.k_in, cfg.k_ff, out, tag=f"c5 layer {layer}")
        y = prox.from_bits(out.y, cfg.dtype)
        x_next = prox.add_rmsnorm(x, y, 1e-6)
        torch.cuda.synchronize()
        ref = oracle.add_rmsnorm(xb, out.y, cfg.dtype, 1e-6)
        got = W.bits_to_f32(prox.to_bits(x_next), cfg.dtype).astype(np.float64)
        assert (np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-6).all()
        x = x_next
        del case
        torch.cuda.empty_cache()
