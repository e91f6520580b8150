"""The seeded input generators: reproducible, RNE casts, config arithmetic."""
import numpy as np
import torch

from paper_2607_27591_amd import workloads as W


def test_draw_recipe_is_reproducible(monkeypatch):
    cfg = W.small_config(d=64, f=300, seed=3)
    monkeypatch.setattr(W, "_CHUNK_ROWS", 7)
    a = W.make_workload(cfg)
    # chunk c of matrix m comes from default_rng([seed, m, c])
    wu = np.concatenate([np.random.default_rng([cfg.seed, 1, c]).standard_normal(
        (min(7, cfg.d_ff - 7 * c), cfg.d_model), dtype=np.float32) for c in range(43)])
    wu *= np.float32(cfg.sigma_w)
    assert np.array_equal(a.w_up, W.f32_to_bf16_bits_ref(wu))
    b = W.make_workload(cfg)
    assert np.array_equal(a.w_down, b.w_down)
    assert np.array_equal(a.x_vectors(3), b.x_vectors(3))


def test_bf16_and_f16_casts_are_rne():
    rng = np.random.default_rng(0)
    v = (rng.standard_normal(100000) * np.exp(rng.uniform(-10, 10, 100000))).astype(np.float32)
    want = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(W.f32_to_bf16_bits_ref(v), want)
    assert np.array_equal(W.f32_to_bf16_bits(v), want)
    want16 = torch.from_numpy(v).to(torch.float16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(W.f32_to_f16_bits(v), want16)
    assert np.array_equal(W.bits_to_f32(W.f32_to_bf16_bits(v), W.DT_BF16),
                          torch.from_numpy(v).to(torch.bfloat16).float().numpy())


def test_config_counts():
    c4 = W.CONFIGS["c4_8192x28672_bf16"]
    assert (c4.k_in, c4.k_ff) == (3277, 8602)
    c2 = W.CONFIGS["c2_4096x12288_bf16"]
    assert (c2.k_in, c2.k_ff) == (2048, 3686)
    c1 = W.CONFIGS["c1_1024x3072_f16"]
    assert (c1.k_in, c1.k_ff, c1.group, c1.qbits) == (512, 1536, 1024, 8)
    c3 = W.CONFIGS["c3_4096x14336_bf16"]
    assert [W.frac_to_k(1 - s, c3.d_ff) for s in W.C3_FFN_SPARSITIES] == [14336, 7168, 4301, 1434]
    assert W.stack_layer_config(35).seed == 39


def test_outliers_scaled():
    cfg = W.small_config(d=128, f=64, n_outliers=5, outlier_scale=50.0)
    wl = W.make_workload(cfg)
    x = W.bits_to_f32(wl.x_vectors(200), cfg.dtype)
    mag = np.abs(x).mean(axis=(0, 1))
    assert len(set(wl.outliers.tolist())) == 5
    assert mag[wl.outliers].min() > 10 * np.median(mag)
