"""GPU parity of the HIP path against the CPU oracle at reduced sizes that
still span several tiles and a ragged tail, plus the method's edge cases.
All calls go through the C-ABI (libprox.so) via the ctypes binding."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_27591_amd import prox
from paper_2607_27591_amd import workloads as W

from gpu_cases import (Y_TOL, check_pack, check_sparse, log, make_case, run_sparse,
                       y_rel_err)

pytestmark = pytest.mark.gpu

SMALL = {
    "bf16_i4_256x384_b1": W.small_config(d=256, f=384, batch=1, seed=1),
    "bf16_i4_1024x1600_b1": W.small_config(d=1024, f=1600, batch=1, seed=2, in_frac=0.4,
                                           ff_frac=0.3, sigma_w=0.02, n_outliers=8),
    "bf16_i4_g256_512x1000_b5": W.small_config(d=512, f=1000, batch=5, seed=3, group=256),
    "f16_i8_pc_512x700_b2": W.small_config(d=512, f=700, batch=2, seed=4, dtype=W.DT_F16,
                                           qbits=8, group=512, ff_frac=0.5),
    "f16_i4_384x520_b1": W.small_config(d=384, f=520, batch=1, seed=5, dtype=W.DT_F16),
    "bf16_i4_256x640_b16": W.small_config(d=256, f=640, batch=16, seed=6, x_kind="student_t",
                                          n_outliers=0),
    "bf16_i4_128x64_b1": W.small_config(d=128, f=64, batch=1, seed=7),
    "bf16_i8_g128_640x513_b3": W.small_config(d=640, f=513, batch=3, seed=8, qbits=8),
    "bf16_i4_2048x3000_b4": W.small_config(d=2048, f=3000, batch=4, seed=9, in_frac=0.4,
                                           sigma_w=0.02),
    # Five or more rows run on the matrix-core proxy: fp16 codes, and a 4096-wide
    # input whose threshold-mode list allows only 8 rows per launch (two
    # launches, the second accumulating into the scores).
    "f16_i4_768x900_b7": W.small_config(d=768, f=900, batch=7, seed=13, dtype=W.DT_F16),
    "bf16_i4_4096x1500_b12": W.small_config(d=4096, f=1500, batch=12, seed=14, in_frac=0.7,
                                            sigma_w=0.02),
    # Batches past one launch's rows: 40 rows on the matrix cores (16 + 16 + 8
    # per Stage 1 launch, five 8-row Stage 2 launches), and 20 INT8 rows on the
    # dot-product kernel (five 4-row Stage 1 launches).
    "bf16_i4_1024x1600_b40": W.small_config(d=1024, f=1600, batch=40, seed=16, in_frac=0.4,
                                            sigma_w=0.02),
    "f16_i8_512x700_b20": W.small_config(d=512, f=700, batch=20, seed=17, dtype=W.DT_F16,
                                         qbits=8, group=512, ff_frac=0.5),
    # d_model 16384 on the matrix cores: 16 input rows per thread, 8 batch
    # rows per launch.
    "bf16_i4_16384x320_b6": W.small_config(d=16384, f=320, batch=6, seed=15, in_frac=0.3,
                                           sigma_w=0.01),
    # More than eight rows of 16-bit weights at d_model >= 4096 run Stage 2 on
    # the matrix cores: 9 fp16 rows in one chunk, and 33 rows as chunks of 16,
    # 16 and 1 sharing one kept list.
    "f16_i4_4096x1000_b9": W.small_config(d=4096, f=1000, batch=9, seed=18, dtype=W.DT_F16,
                                          in_frac=0.5, sigma_w=0.02),
    "bf16_i4_8192x700_b33": W.small_config(d=8192, f=700, batch=33, seed=19, in_frac=0.4,
                                           sigma_w=0.01),
    # The paper's per-row INT4 proxy (one scale per output channel, group =
    # d_model): batch 1 on the dot-product Stage 1, batch 6 on the matrix cores.
    "bf16_i4_perrow_1024x1600_b1": W.small_config(d=1024, f=1600, batch=1, seed=21, group=1024,
                                                  in_frac=0.4, sigma_w=0.02, n_outliers=8),
    "bf16_i4_perrow_2048x1200_b6": W.small_config(d=2048, f=1200, batch=6, seed=22, group=2048,
                                                  in_frac=0.4, sigma_w=0.02),
    # Maximum sizes: d_model 16384 (16 input rows per thread, 1 batch row
    # per proxy launch) and d_ff 65536 (64 score rows per thread).
    "bf16_i4_16384x320_b3": W.small_config(d=16384, f=320, batch=3, seed=10, in_frac=0.3,
                                           sigma_w=0.01),
    "f16_i4_128x65536_b2": W.small_config(d=128, f=65536, batch=2, seed=12, dtype=W.DT_F16,
                                          ff_frac=0.2),
    # The largest batch a call takes (64 rows): four 16-row launches of each
    # matrix-core stage, and sixteen 4-row Stage 1 plus eight 8-row Stage 2
    # launches of the dot-product kernels.
    "bf16_i4_4096x1000_b64": W.small_config(d=4096, f=1000, batch=64, seed=24, in_frac=0.4,
                                            sigma_w=0.02),
    "f16_i8_512x700_b64": W.small_config(d=512, f=700, batch=64, seed=25, dtype=W.DT_F16,
                                         qbits=8, group=512, ff_frac=0.5),
}


@pytest.fixture(scope="module", params=sorted(SMALL))
def case(request):
    cfg = SMALL[request.param]
    log(f"[case] {request.param}: d={cfg.d_model} f={cfg.d_ff} B={cfg.batch} "
        f"q{cfg.qbits} g{cfg.group} dtype={W.DTYPE_NAMES[cfg.dtype]}")
    c = make_case(cfg)
    yield c
    del c
    torch.cuda.empty_cache()


def test_pack_bit_exact(case):
    log(f"[pack] {case.cfg.name}")
    check_pack(case)


def test_sparse_parity(case):
    cfg = case.cfg
    xs = case.wl.x_vectors(3, cfg.batch)
    for n, x in enumerate(xs):
        log(f"[sparse] {cfg.name} vector {n} k_in={cfg.k_in} k_ff={cfg.k_ff}")
        out = run_sparse(case, x, cfg.k_in, cfg.k_ff)
        stats = check_sparse(case, x, cfg.k_in, cfg.k_ff, out, tag=f"{cfg.name}/{n}")
        log(f"    {stats}")


def test_dense_parity(case):
    cfg = case.cfg
    x = case.wl.x_vectors(1, cfg.batch)[0]
    log(f"[dense] {cfg.name}")
    y = prox.ffn_dense(case.w, prox.from_bits(x, cfg.dtype))
    torch.cuda.synchronize()
    ref = oracle.ffn_dense(x, cfg.dtype, case.wl.w_gate, case.wl.w_up, case.wl.w_down)
    err = y_rel_err(prox.to_bits(y), ref, cfg.dtype)
    log(f"    y err {err:.3e}")
    assert err <= Y_TOL


def test_no_sparsity_equals_dense(case):
    """k_in = d and k_ff = d_ff: the sparse step runs the dense kernels over
    every channel in the same order, so y is bitwise the dense y."""
    cfg = case.cfg
    x = case.wl.x_vectors(1, cfg.batch)[0]
    log(f"[k_ff=f] {cfg.name}")
    out = run_sparse(case, x, cfg.d_model, cfg.d_ff)
    y = prox.ffn_dense(case.w, prox.from_bits(x, cfg.dtype))
    torch.cuda.synchronize()
    assert out.mask.all() and out.in_mask.all()
    assert np.array_equal(out.y, prox.to_bits(y))


def test_extreme_k(case):
    cfg = case.cfg
    x = case.wl.x_vectors(1, cfg.batch)[0]
    for k_in, k_ff in [(1, 1), (1, cfg.d_ff), (cfg.d_model, 1), (cfg.d_model // 2 + 1, cfg.d_ff - 1)]:
        log(f"[extreme] {cfg.name} k_in={k_in} k_ff={k_ff}")
        out = run_sparse(case, x, k_in, k_ff)
        check_sparse(case, x, k_in, k_ff, out, tag=f"{cfg.name} k_in={k_in} k_ff={k_ff}")


def test_deterministic(case):
    cfg = case.cfg
    x = case.wl.x_vectors(1, cfg.batch)[0]
    log(f"[determinism] {cfg.name}")
    a = run_sparse(case, x, cfg.k_in, cfg.k_ff)
    b = run_sparse(case, x, cfg.k_in, cfg.k_ff)
    assert np.array_equal(a.y, b.y) and np.array_equal(a.mask, b.mask)
    assert np.array_equal(a.scores.view(np.uint32), b.scores.view(np.uint32))


def _stage_events():
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(prox.SPARSE_STAGES + 1)]
    for e in ev:
        e.record()   # an event must exist before the library records it
    return ev


def check_staged(run, tag):
    """The entry point with events between its stages (how the benchmark times
    it) against the same call without: the same bits, and events that complete
    in stage order."""
    y0, m0 = run(None)
    ev = _stage_events()
    y1, m1 = run(ev)
    torch.cuda.synchronize()
    assert torch.equal(y0, y1) and torch.equal(m0, m1), f"{tag}: staged call differs"
    t = [ev[0].elapsed_time(e) for e in ev[1:]]
    assert all(v >= 0.0 for v in t) and t == sorted(t), f"{tag}: stage events {t}"


def test_staged_entry_point(case):
    cfg = case.cfg
    x = prox.from_bits(np.atleast_2d(case.wl.x_vectors(1, cfg.batch)[0]), cfg.dtype)
    log(f"[staged] {cfg.name}")
    check_staged(lambda ev: prox.ffn_sparse(case.w, case.proxy, x, cfg.k_in, cfg.k_ff, events=ev),
                 cfg.name)


# ---------------------------------------------------------------------------
# Degenerate inputs: ties everywhere
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def tie_case():
    cfg = W.small_config(d=512, f=1100, batch=2, seed=21)
    log("[case] ties 512x1100 B=2")
    c = make_case(cfg)
    yield c
    del c


def test_zero_input(tie_case):
    cfg = tie_case.cfg
    x = np.zeros((cfg.batch, cfg.d_model), np.uint16)
    x[1, ::3] = 0x8000    # -0 ties with +0
    log("[ties] zero input")
    out = run_sparse(tie_case, x, 100, 200)
    assert np.flatnonzero(out.in_mask).tolist() == list(range(100))
    assert np.flatnonzero(out.mask).tolist() == list(range(200))
    assert not out.scores.any()
    assert not W.bits_to_f32(out.y, cfg.dtype).any()
    check_sparse(tie_case, x, 100, 200, out, tag="zero")


def test_equal_magnitudes(tie_case):
    cfg = tie_case.cfg
    rng = np.random.default_rng(0)
    v = rng.choice([-1.5, 1.5], size=(cfg.batch, cfg.d_model)).astype(np.float32)
    v[0, 300:] = 0.25   # lower magnitudes after index 300 on both rows
    v[1, 300:] = -0.25
    x = W.to_bits(v, cfg.dtype)
    for k_in in (1, 150, 300, 301, 511):
        log(f"[ties] equal magnitudes k_in={k_in}")
        out = run_sparse(tie_case, x, k_in, 77)
        check_sparse(tie_case, x, k_in, 77, out, tag=f"equal k_in={k_in}")
        assert np.flatnonzero(out.in_mask).tolist() == list(range(k_in))


def test_workspace_reuse_across_batches(tie_case):
    cfg = tie_case.cfg
    ws = prox.new_workspace(cfg.d_model, cfg.d_ff, 16)
    for B in (1, 4, 16, 2):
        x = tie_case.wl.x_vectors(1, B)[0]
        log(f"[ws reuse] B={B}")
        out = run_sparse(tie_case, x, 200, 300, ws=ws)
        check_sparse(tie_case, x, 200, 300, out, tag=f"ws B={B}")


def test_add_rmsnorm():
    rng = np.random.default_rng(5)
    for dtype in (W.DT_BF16, W.DT_F16):
        for B, d in [(1, 4096), (3, 1000), (16, 8192)]:
            x = W.to_bits(rng.laplace(size=(B, d)).astype(np.float32), dtype)
            y = W.to_bits(rng.normal(size=(B, d)).astype(np.float32), dtype)
            log(f"[rmsnorm] dtype={dtype} B={B} d={d}")
            out = prox.add_rmsnorm(prox.from_bits(x, dtype), prox.from_bits(y, dtype), 1e-6)
            torch.cuda.synchronize()
            ref = oracle.add_rmsnorm(x, y, dtype, 1e-6)
            got = W.bits_to_f32(prox.to_bits(out), dtype).astype(np.float64)
            ulp = 2.0 ** -8 if dtype == W.DT_BF16 else 2.0 ** -11
            assert (np.abs(got - ref) <= ulp * np.abs(ref) + 1e-6).all()
