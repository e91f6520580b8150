"""Pins of the oracle's threshold mode (Sec. 4.1 masks with layer-wise
thresholds, App. A.6) and of its calibration (App. A.7, Alg. 1).

Each check comes from brute force on tiny inputs, a special case that reduces
to another definition (the top-k reading, the dense FFN, a library sort), a
hand-worked example (tests/golden/), or a property that a plausible mistake
breaks (demonstrated below by planting the mistake in a copy).
"""
import json
import math
import os

import numpy as np
import pytest

from paper_2607_27591_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _tiny(seed=5, d=64, f=96, B=1, dtype=W.DT_BF16, sigma=0.05):
    cfg = W.small_config(d=d, f=f, dtype=dtype, seed=seed, batch=B, sigma_w=sigma,
                         n_outliers=2, group=32)
    wl = W.make_workload(cfg)
    return cfg, wl, wl.x_vectors(1, B)[0]


def _layer(oracle_lib, cfg, wl):
    cg, sg = oracle_lib.quantize(wl.w_gate, cfg.dtype, 4, cfg.group)
    cu, su = oracle_lib.quantize(wl.w_up, cfg.dtype, 4, cfg.group)
    return dict(w_gate=wl.w_gate, w_up=wl.w_up, w_down=wl.w_down, codes_g=cg, scales_g=sg,
                codes_u=cu, scales_u=su, group=cfg.group)


# ---------------------------------------------------------------------------
# The rule |z| >= tau
# ---------------------------------------------------------------------------

def test_threshold_rule_brute_force(oracle_lib):
    rng = np.random.default_rng(0)
    for trial in range(50):
        n = int(rng.integers(1, 40))
        key = rng.integers(0, 6, n).astype(np.float64)   # many ties
        tau = float(rng.integers(0, 7))
        want = [i for i in range(n) if key[i] >= tau]
        assert oracle_lib.select_threshold(key, tau).tolist() == want


def test_threshold_keeps_values_equal_to_tau(oracle_lib):
    # App. A.6 uses >=: an entry exactly at the threshold is kept, so all
    # tied entries go in together (a top-k of 1 would keep only index 0).
    assert oracle_lib.select_threshold([3.0, 1.0, 3.0, 2.0], 3.0).tolist() == [0, 2]
    assert oracle_lib.topk([3.0, 1.0, 3.0, 2.0], 1).tolist() == [0]


def test_threshold_at_kth_value_is_topk(oracle_lib):
    # With distinct keys, tau = the k-th largest key selects exactly the top k.
    rng = np.random.default_rng(1)
    for k in (1, 7, 30, 64):
        key = rng.permutation(64).astype(np.float64) * 0.25
        tau = np.sort(key)[::-1][k - 1]
        assert oracle_lib.select_threshold(key, tau).tolist() == oracle_lib.topk(key, k).tolist()


def test_inputs_tau_brute_force_batch(oracle_lib):
    cfg, wl, x = _tiny(seed=3, B=3)
    a = np.abs(W.bits_to_f32(x, cfg.dtype).astype(np.float64)).max(axis=0)
    for tau in (0.0, 0.5, 1.0, 2.5, float(a.max()), float(a.max()) * 2):
        want = [i for i in range(cfg.d_model) if a[i] >= tau]
        assert oracle_lib.select_inputs_tau(x, cfg.dtype, tau).tolist() == want


def test_tau_zero_is_dense_bitwise(oracle_lib):
    # Magnitudes are >= 0, so tau_x = tau_s = 0 keeps every input and channel:
    # the step is the dense FFN, summed in the same order.
    cfg, wl, x = _tiny(seed=4, B=2)
    L = _layer(oracle_lib, cfg, wl)
    r = oracle_lib.ffn_sparse_tau(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down, 0.0, 0.0,
                                  codes_g=L["codes_g"], scales_g=L["scales_g"],
                                  codes_u=L["codes_u"], scales_u=L["scales_u"], group=cfg.group)
    assert r["k_in"] == cfg.d_model and r["k_ff"] == cfg.d_ff
    assert np.array_equal(r["y"], oracle_lib.ffn_dense(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down))


def test_tau_infinite_keeps_nothing(oracle_lib):
    cfg, wl, x = _tiny(seed=6)
    L = _layer(oracle_lib, cfg, wl)
    kw = dict(codes_g=L["codes_g"], scales_g=L["scales_g"], codes_u=L["codes_u"],
              scales_u=L["scales_u"], group=cfg.group)
    r = oracle_lib.ffn_sparse_tau(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down, math.inf, 1e-30, **kw)
    assert r["k_in"] == 0 and r["k_ff"] == 0 and not r["score"].any() and not r["y"].any()
    # No inputs: every proxy score is 0, so tau_s = 0 still keeps every channel.
    r = oracle_lib.ffn_sparse_tau(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down, math.inf, 0.0, **kw)
    assert r["k_ff"] == cfg.d_ff
    assert np.array_equal(r["y"], oracle_lib.ffn_dense(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down))


@pytest.mark.parametrize("B", [1, 3])
def test_tau_at_matched_values_reproduces_topk_step(oracle_lib, B):
    # Choose tau_x, tau_s as the k-th largest a_i and proxy score: the
    # threshold step must then pick the same sets and give the same y as the
    # top-k step (both reading the same Sec. 4.1 masks).
    cfg, wl, x = _tiny(seed=8, B=B, d=128, f=160)
    L = _layer(oracle_lib, cfg, wl)
    kw = dict(codes_g=L["codes_g"], scales_g=L["scales_g"], codes_u=L["codes_u"],
              scales_u=L["scales_u"], group=cfg.group)
    a = np.abs(W.bits_to_f32(x, cfg.dtype).astype(np.float64)).reshape(B, -1).max(axis=0)
    k_in = 50
    order = np.lexsort((np.arange(a.size), -a))
    tau_x = a[order[k_in - 1]]
    if a[order[k_in]] == tau_x:   # the k-th value is tied: the sets differ by design
        pytest.skip("tie at the input boundary")
    top = oracle_lib.ffn_sparse(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down, k_in, 40, **kw)
    s_sorted = np.sort(top["score"])[::-1]
    tau_s = s_sorted[39]
    assert s_sorted[40] < tau_s
    r = oracle_lib.ffn_sparse_tau(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down, tau_x, tau_s, **kw)
    assert r["in_idx"].tolist() == top["in_idx"].tolist()
    assert r["ff_idx"].tolist() == top["ff_idx"].tolist()
    assert np.array_equal(r["y"], top["y"])


# ---------------------------------------------------------------------------
# Calibration pieces: the bounded sample and its quantile
# ---------------------------------------------------------------------------

def test_reservoir_hand_worked(oracle_lib):
    g = json.load(open(os.path.join(GOLDEN, "reservoir_example.json")))
    res = oracle_lib.Reservoir(g["cap"])
    res.add(g["values"][:3], np.array(g["draws"][:3], np.uint64))   # two calls: the
    res.add(g["values"][3:], np.array(g["draws"][3:], np.uint64))   # stream continues
    assert res.sample().tolist() == g["reservoir_final"]


def test_reservoir_under_capacity_keeps_everything(oracle_lib):
    v = np.arange(100.0)
    res = oracle_lib.Reservoir(1000)
    res.add(v, W.reservoir_draws(1)(100))
    assert res.sample().tolist() == v.tolist()


def test_reservoir_inclusion_is_uniform(oracle_lib):
    # Algorithm R keeps each of n items with probability cap / n.
    n, cap, trials = 40, 10, 4000
    draw = W.reservoir_draws(3)
    hits = np.zeros(n)
    for _ in range(trials):
        res = oracle_lib.Reservoir(cap)
        res.add(np.arange(float(n)), draw(n))
        hits[res.sample().astype(int)] += 1
    p = hits / trials
    sd = math.sqrt(0.25 * 0.75 / trials)
    assert np.abs(p - cap / n).max() < 5 * sd


@pytest.mark.parametrize("s", [0.0, 0.1, 0.3, 0.5, 0.7, 0.9, 0.999])
def test_quantile_threshold_order_statistic(oracle_lib, s):
    rng = np.random.default_rng(int(s * 1000))
    for trial in range(20):
        n = int(rng.integers(1, 300))
        v = rng.integers(0, 25, n).astype(np.float64)   # ties
        tau = oracle_lib.quantile_threshold(v, s)
        pos = min(n - 1, math.floor(s * n))
        assert tau == np.sort(v)[pos]
        # order-statistic property: at most pos samples lie strictly below
        # tau, and more than pos lie at or below it
        assert (v < tau).sum() <= pos < (v <= tau).sum()


def test_quantile_threshold_hits_target_sparsity(oracle_lib):
    # Distinct samples: the rule |z| >= tau then drops exactly floor(s n).
    v = np.random.default_rng(5).permutation(1000).astype(np.float64)
    for s in (0.4, 0.6, 0.7):
        tau = oracle_lib.quantile_threshold(v, s)
        assert (v < tau).sum() == math.floor(s * 1000)


# ---------------------------------------------------------------------------
# Alg. 1: sequential calibration
# ---------------------------------------------------------------------------

def _stack(oracle_lib, L=3, d=128, f=192):
    layers, cfgs = [], []
    for l in range(L):
        cfg = W.small_config(d=d, f=f, seed=40 + l, sigma_w=0.05, n_outliers=2, group=32)
        wl = W.make_workload(cfg)
        layers.append(_layer(oracle_lib, cfg, wl))
        cfgs.append((cfg, wl))
    tokens = cfgs[0][1].x_vectors(12, 1)[:, 0, :]
    return cfgs[0][0].dtype, layers, tokens


def _quantile_property(oracle_lib, tokens, dtype, layers, taus, s1, s2):
    """Run the finalised sparse stack on the calibration tokens and check, at
    every layer, that its thresholds are the order statistics of the signals
    that layer actually sees."""
    xs = tokens
    for layer, (tau_x, tau_s) in zip(layers, taus):
        mx = np.abs(oracle_lib.halves_to_double(xs, dtype)).ravel()
        sv = []
        nxt = []
        for t in range(xs.shape[0]):
            in_idx = oracle_lib.select_inputs_tau(xs[t], dtype, tau_x)
            _, _, st, _ = oracle_lib.proxy(xs[t], dtype, in_idx, codes_g=layer["codes_g"],
                                           scales_g=layer["scales_g"], codes_u=layer["codes_u"],
                                           scales_u=layer["scales_u"], group=layer["group"])
            sv.append(np.abs(st[0]))
            nxt.append(oracle_lib.stack_layer_tau(xs[t], dtype, layer, tau_x, tau_s)[0][0])
        sv = np.concatenate(sv)
        for v, tau, s in ((mx, tau_x, s1), (sv, tau_s, s2)):
            pos = min(v.size - 1, math.floor(s * v.size))
            if not ((v < tau).sum() <= pos < (v <= tau).sum()):
                return False
        xs = np.stack(nxt)
    return True


def test_calibration_is_sequential(oracle_lib):
    dtype, layers, tokens = _stack(oracle_lib)
    s1, s2 = 0.5, 0.7
    cap = 10 ** 6   # every sample kept: the quantiles are exact
    taus = oracle_lib.calibrate_stack(tokens, dtype, layers, s1, s2, cap, W.reservoir_draws(2))
    assert all(tx > 0 and ts > 0 for tx, ts in taus)
    assert _quantile_property(oracle_lib, tokens, dtype, layers, taus, s1, s2)


def test_planted_dense_calibration_breaks_the_pin(oracle_lib):
    # The mistake Alg. 1 exists to avoid: collecting each layer's inputs
    # through DENSE earlier layers.  Those thresholds are order statistics of
    # the wrong signals, and the pin above notices.
    dtype, layers, tokens = _stack(oracle_lib)
    s1, s2 = 0.5, 0.7
    xs, taus = tokens, []
    for layer in layers:
        mx = np.abs(oracle_lib.halves_to_double(xs, dtype)).ravel()
        tau_x = oracle_lib.quantile_threshold(mx, s1)
        sv = []
        for t in range(xs.shape[0]):
            in_idx = oracle_lib.select_inputs_tau(xs[t], dtype, tau_x)
            _, _, st, _ = oracle_lib.proxy(xs[t], dtype, in_idx, codes_g=layer["codes_g"],
                                           scales_g=layer["scales_g"], codes_u=layer["codes_u"],
                                           scales_u=layer["scales_u"], group=layer["group"])
            sv.append(np.abs(st[0]))
        taus.append((tau_x, oracle_lib.quantile_threshold(np.concatenate(sv), s2)))
        # planted: the next layer's inputs come from the dense layer
        xs = np.stack([oracle_lib.round_to_dtype(oracle_lib.add_rmsnorm(
            xs[t], oracle_lib.round_to_dtype(oracle_lib.ffn_dense(
                xs[t], dtype, layer["w_gate"], layer["w_up"], layer["w_down"]), dtype),
            dtype), dtype)[0] for t in range(xs.shape[0])])
    assert not _quantile_property(oracle_lib, tokens, dtype, layers, taus, s1, s2)
