#!/usr/bin/env python3
"""Benchmark of the Prox sparse SwiGLU FFN decode step on one MI355X.

Default workload: the 8192 x 28672 bf16 FFN at batch 1 with an int4
group-128 proxy, 40% of inputs and 30% of intermediate channels kept (70%
FFN sparsity).  One step = one prox_ffn_sparse call (input top-k, proxy
GEMV + score, channel top-k, gate/up, down) on a fresh decode vector, with
weights, proxy and inputs already resident in HBM.

Timing: every timed call is bracketed by HIP events on the stream the
library launches on; before each call a 1 GiB buffer is read (outside the
events) so neither the L2s nor the 256 MB last-level cache hold weights
("cold").  A back-to-back ("warm") figure is reported as secondary.  The
dense HIP FFN is timed the same way.  Achieved bandwidth is computed from
the bytes the sparse step has to move (algorithmic bytes), not from counters.

Prints ONE JSON line.
"""
import argparse
import hashlib
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "sparse FFN µs/call + achieved HBM GB/s at 70% sparsity, batch 1 (vs dense)"
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E peak
ALPHA = 1.0 / 3.0              # proxy cost ratio used by the paper's cost model
FLUSH_BYTES = 1 << 30


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="c4_8192x28672_bf16",
                    help="c1_1024x3072_f16 | c2_4096x12288_bf16 | c3_4096x14336_bf16 | "
                         "c4_8192x28672_bf16 | c5_stack36")
    ap.add_argument("--batch", type=int, default=None, help="batch rows (c3 sweeps 1/4/16)")
    ap.add_argument("--ffn-sparsity", type=float, default=None,
                    help="override the kept-channel fraction as 1 - sparsity")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-tau", action="store_true", help="skip the threshold-mode leg")
    ap.add_argument("--no-w4", action="store_true", help="skip the INT4 base-weight (W4A16) leg")
    ap.add_argument("--alpha", action="store_true",
                    help="measure the proxy-cost ratio alpha (quantised over 16-bit proxy)")
    ap.add_argument("--calib-tokens", type=int, default=32,
                    help="held-out synthetic vectors for the threshold calibration")
    ap.add_argument("--cpu-budget-s", type=float, default=10.0,
                    help="seconds of sparse oracle calls (the dense oracle gets half)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other workloads (c1, c2, c3 batch 1/4/16, c5 stack)")
    ap.add_argument("--config-steps", type=int, default=20,
                    help="timed calls per workload in the configs object")
    ap.add_argument("--warm", action="store_true", help="headline from back-to-back calls")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only copy a MIB-sized buffer 5 times (reference kernel of known "
                         "traffic for scaling HBM counters) and exit")
    return ap.parse_args()


def algorithmic_bytes(cfg, B, k_in, k_ff):
    """Bytes the sparse step must move: x, the selected proxy rows, the
    touched scale groups, the kept gate/up/down rows, and y."""
    e, d, f = 2, cfg.d_model, cfg.d_ff
    ng = d // cfg.group
    return {
        "x": B * d * e,
        "proxy_codes": 2 * k_in * f * cfg.qbits // 8,
        "proxy_scales": 2 * ng * f * 2,
        "gate_up_rows": 2 * k_ff * d * e,
        "down_rows": k_ff * d * e,
        "y": B * d * e,
    }


def w4_bytes(cfg, B, k_in, k_ff):
    """Bytes of the sparse step with Stage 2 on INT4 base weights: Stage 1 as
    algorithmic_bytes, then the kept channels' codes (d / 2 bytes per row)
    and scales (d / group fp16 per row) of the three matrices."""
    ab = algorithmic_bytes(cfg, B, k_in, k_ff)
    d, ng = cfg.d_model, cfg.d_model // cfg.group
    row = d // 2 + ng * 2
    return {"x": ab["x"], "proxy_codes": ab["proxy_codes"], "proxy_scales": ab["proxy_scales"],
            "gate_up_rows": 2 * k_ff * row, "down_rows": k_ff * row, "y": ab["y"]}


def dense_bytes(cfg, B):
    e, d, f = 2, cfg.d_model, cfg.d_ff
    return 3 * d * f * e + 2 * B * d * e


def src_hash(*names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2607_27591_amd", "csrc", n), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, kernel_src):
    """HBM bytes per launch of the dominant kernel from the committed
    rocprofv3 PMC summary, if it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"pmc_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"traffic_json:\s*(\{.*\})", text)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("source_hash") != kernel_src:
        return None
    return rec.get("hbm_bytes_per_launch")


def pct(v, q):
    v = sorted(v)
    return v[min(len(v) - 1, max(0, int(round(q * (len(v) - 1)))))]


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: --gpus {args.gpus} is not supported "
              "(libprox runs the sparse decode step on a single GPU; sharding along d_ff "
              "is a design note, not code)",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2607_27591_amd import prox
    from paper_2607_27591_amd import workloads as W

    prox.lib()   # fails loudly if libprox.so is missing
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)

    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.ones(n // 8, dtype=torch.int64, device=dev)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes_read": n, "calibrate_copy_bytes_written": n,
                          "launches": 5}), flush=True)
        return

    if args.workload.startswith("c5"):
        return bench_stack(args, np, torch, prox, W, dev)
    if args.alpha:
        return bench_alpha(args, np, torch, prox, W, dev)

    cfg = W.CONFIGS[args.workload]
    B = args.batch or cfg.batch
    k_in = cfg.k_in
    k_ff = cfg.k_ff if args.ffn_sparsity is None else W.frac_to_k(1 - args.ffn_sparsity, cfg.d_ff)
    t_gen = time.perf_counter()
    wl = W.make_workload(cfg)
    n_x = min(args.warmup + args.steps, max(cfg.n_vectors, 1))
    xs_np = wl.x_vectors(n_x, B)
    w = prox.Weights(*(prox.from_bits(m, cfg.dtype, dev) for m in (wl.w_gate, wl.w_up, wl.w_down)))
    proxy = prox.pack_proxy(w, prox.INT4 if cfg.qbits == 4 else prox.INT8, cfg.group)
    xs = prox.from_bits(xs_np.reshape(n_x, B * cfg.d_model), cfg.dtype, dev).view(n_x, B, cfg.d_model)
    ws = prox.new_workspace(cfg.d_model, cfg.d_ff, B, dev)
    y = torch.empty((B, cfg.d_model), dtype=w.dtype, device=dev)
    mask = torch.empty(cfg.d_ff, dtype=torch.uint8, device=dev)
    # Cache eviction by reading 1 GiB (more than the L2s and the 256 MB
    # last-level cache): a written buffer would leave dirty lines whose
    # write-back competes with the timed call's reads (measured to halve the
    # next kernel's bandwidth), which a decode step after weight-reading
    # layers does not see.
    flush = torch.ones(FLUSH_BYTES // 8, dtype=torch.int64, device=dev)
    sink = torch.zeros((), dtype=torch.int64, device=dev)
    torch.cuda.synchronize()
    gen_s = time.perf_counter() - t_gen

    def sparse(i, events=None):
        prox.ffn_sparse(w, proxy, xs[i % n_x], k_in, k_ff, y=y, mask=mask, ws=ws, events=events)

    def dense(i):
        prox.ffn_dense(w, xs[i % n_x], y=y, ws=ws)

    def timed(fn, n, cold=True, staged=False):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(n)]
        stage = None
        if staged:
            stage = [[torch.cuda.Event(enable_timing=True) for _ in range(prox.SPARSE_STAGES + 1)]
                     for _ in range(n)]
            for row in stage:
                for ev in row:
                    ev.record()   # create the HIP events before handing them over
        for i in range(n):
            if cold:
                torch.sum(flush, 0, out=sink)
            evs[i][0].record()
            if staged:
                fn(i, stage[i])
            else:
                fn(i)
            evs[i][1].record()
        torch.cuda.synchronize()
        us = [a.elapsed_time(b) * 1e3 for a, b in evs]
        st = None
        if staged:
            st = [[row[s].elapsed_time(row[s + 1]) * 1e3 for s in range(prox.SPARSE_STAGES)]
                  for row in stage]
        return us, st

    # ---- warmup ----
    for i in range(args.warmup):
        sparse(i)
        if not args.no_dense:
            dense(i)
    torch.cuda.synchronize()

    # ---- timed region: K sparse steps ----
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    cold_us, _ = timed(sparse, args.steps, cold=not args.warm)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3

    # Per-stage durations of the same kernels (staged entry point).
    _, stage_rows = timed(sparse, args.steps, cold=not args.warm, staged=True)
    stage_names = prox.stage_names()
    stage_us = {n: statistics.mean(r[s] for r in stage_rows) for s, n in enumerate(stage_names)}

    # Back-to-back calls between two events.
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(args.steps):
        sparse(i)
    e1.record()
    torch.cuda.synchronize()
    warm_us = e0.elapsed_time(e1) * 1e3 / args.steps

    dense_us = None
    if not args.no_dense:
        dus, _ = timed(dense, args.steps, cold=not args.warm)
        dense_us = statistics.median(dus)

    ab = algorithmic_bytes(cfg, B, k_in, k_ff)
    total_bytes = sum(ab.values())
    med = statistics.median(cold_us)
    mean = statistics.mean(cold_us)
    gbs = total_bytes / (med * 1e-6) / 1e9   # every rate and ratio below uses the median

    # Dominant kernel: the fused Stage 2 kernel (three kept rows of d
    # elements per kept channel, plus the f proxy scores it ranks).
    s2_bytes = ab["gate_up_rows"] + ab["down_rows"] + 4 * cfg.d_ff
    s2_us = stage_us["stage2_select_gate_up_down"]
    s2_gbs = s2_bytes / (s2_us * 1e-6) / 1e9
    traffic = measured_traffic(args.workload, src_hash("stage2.hip", "common.hpp", "layout.hpp",
                                                       "topk.hpp"))
    roofline = {"bound": "hbm", "kernel": "stage2_kernel (channel top-k, gate/up, down)",
                "achieved": round(s2_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(s2_gbs / PEAK_HBM_GBS, 4), "traffic": traffic,
                "algorithmic_bytes_per_launch": s2_bytes, "avg_launch_us": round(s2_us, 2)}

    w4 = None
    if not args.no_w4:
        w4 = w4_leg(args, cfg, w, proxy, xs, n_x, B, ws, y, mask, k_in, k_ff, timed, prox)

    tau = None
    if not args.no_tau:
        tau = threshold_leg(args, cfg, wl, w, proxy, xs, n_x, B, ws, y, mask, flush, sink,
                            k_in, k_ff, dense_us, np, torch, prox, W, dev)

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(args, cfg, wl, xs_np, B, k_in, k_ff, total_bytes)

    torch_dense = None
    if not args.no_dense:
        torch_dense = torch_dense_leg(args, w, xs, n_x, flush, sink, torch)

    configs = None
    if not args.no_configs and args.batch is None and args.ffn_sparsity is None:
        del w, proxy, flush
        torch.cuda.empty_cache()
        configs = config_legs(args, np, torch, prox, W, dev)

    s1 = 1 - k_in / cfg.d_model
    s2 = 1 - k_ff / cfg.d_ff
    out = {
        "metric": METRIC,
        "value": round(gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(mean / 1e3, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": W.DTYPE_NAMES[cfg.dtype],
        "data": "synthetic: seeded i.i.d. Gaussian weights, heavy-tailed x (no checkpoint)",
        "config": {"workload": f"{cfg.name}_b{B}", "d_model": cfg.d_model, "d_ff": cfg.d_ff,
                   "batch": B, "k_in": k_in, "k_ff": k_ff,
                   "proxy": f"int{cfg.qbits} group {cfg.group} fp16 scales",
                   "ffn_sparsity_s2": round(s2, 4), "input_sparsity_s1": round(s1, 4),
                   "paper_effective_sparsity_e": round(s2 - 2 * ALPHA * (1 - s1) / 3, 4)},
        "us_per_call": {"mean": round(mean, 2), "median": round(med, 2),
                        "p10": round(pct(cold_us, 0.1), 2), "p90": round(pct(cold_us, 0.9), 2),
                        "warm_back_to_back": round(warm_us, 2),
                        "protocol": "warm" if args.warm else "cold (1 GiB read between calls evicts the caches)"},
        "statistic": "median of per-call HIP-event times (value, hbm_frac, tokens_per_s, speedup_vs_dense); ms_per_step is the mean",
        "tokens_per_s": round(1e6 / med, 1),
        "hbm_frac": round(gbs / PEAK_HBM_GBS, 4),
        "algorithmic_bytes": total_bytes,
        "stage_us": {k: round(v, 2) for k, v in stage_us.items()},
        "dense_us_per_call": None if dense_us is None else round(dense_us, 2),
        "dense_gbs": None if dense_us is None else round(dense_bytes(cfg, B) / (dense_us * 1e-6) / 1e9, 1),
        "speedup_vs_dense": None if dense_us is None else round(dense_us / med, 3),
        "wall_ms_timed_region": round(wall_ms, 2),
        "setup_s": round(gen_s, 2),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "threshold_mode": tau,
        "w4a16": w4,
        "torch_dense": torch_dense,
        "configs": configs,
    }
    print(json.dumps(out), flush=True)


def w4_leg(args, cfg, w, proxy, xs, n_x, B, ws, y, mask, k_in, k_ff, timed, prox):
    """The same workload with Stage 2 on INT4 base weights (W4A16, the
    combination Sec. 5.1 leaves to future work), and the dense FFN on the
    same INT4 weights as its baseline; same cold protocol and decode vectors."""
    q = prox.pack_w4(w, cfg.group)
    if prox.workspace_bytes(cfg.d_model, cfg.d_ff, B, w4=True) > ws.numel():
        ws = prox.new_workspace(cfg.d_model, cfg.d_ff, B, ws.device, w4=True)

    def sparse(i, events=None):
        prox.ffn_sparse_w4(q, proxy, xs[i % n_x], k_in, k_ff, y=y, mask=mask, ws=ws,
                           events=events)

    def dense(i):
        prox.ffn_dense_w4(q, xs[i % n_x], y=y, ws=ws)

    for i in range(args.warmup):
        sparse(i)
        dense(i)
    us, _ = timed(sparse, args.steps, cold=not args.warm)
    _, st = timed(sparse, args.steps, cold=not args.warm, staged=True)
    dus, _ = timed(dense, args.steps, cold=not args.warm)
    del q
    names = prox.stage_names()
    stage_us = {n: statistics.mean(r[s] for r in st) for s, n in enumerate(names)}
    ab = w4_bytes(cfg, B, k_in, k_ff)
    mean, med, dmed = statistics.mean(us), statistics.median(us), statistics.median(dus)
    d, f, ng = cfg.d_model, cfg.d_ff, cfg.d_model // cfg.group
    dense_b = 3 * f * (d // 2 + ng * 2) + 2 * B * d * 2
    s2_bytes = ab["gate_up_rows"] + ab["down_rows"] + 4 * f
    s2_us = stage_us["stage2_select_gate_up_down"]
    return {"weights": f"int4 group {cfg.group} fp16 scales, all three matrices",
            "us_per_call": {"mean": round(mean, 2), "median": round(med, 2),
                            "p10": round(pct(us, 0.1), 2), "p90": round(pct(us, 0.9), 2)},
            "algorithmic_bytes": sum(ab.values()),
            "algorithmic_gbs": round(sum(ab.values()) / (mean * 1e-6) / 1e9, 1),
            "stage_us": {k: round(v, 2) for k, v in stage_us.items()},
            "stage2_gbs": round(s2_bytes / (s2_us * 1e-6) / 1e9, 1),
            "dense_w4_us_per_call": round(dmed, 2),
            "dense_w4_gbs": round(dense_b / (dmed * 1e-6) / 1e9, 1),
            "speedup_vs_dense_w4": round(dmed / med, 3)}


def threshold_leg(args, cfg, wl, w, proxy, xs, n_x, B, ws, y, mask, flush, sink, k_in, k_ff,
                  dense_us, np, torch, prox, W, dev):
    """The paper's threshold rule on the same workload: tau_x, tau_s from the
    sequential calibration (one layer here) on held-out synthetic vectors at
    the top-k leg's sparsities, then the same cold protocol on the same
    decode vectors.  Counts are data-dependent, so bytes use each call's own
    realised k_in, k_ff."""
    from paper_2607_27591_amd import calibrate as C
    s1, s2 = 1 - k_in / cfg.d_model, 1 - k_ff / cfg.d_ff
    cal_np = wl.x_vectors(args.calib_tokens, 1)[:, 0, :]
    cal = prox.from_bits(cal_np, cfg.dtype, dev)
    t0 = time.perf_counter()
    (tau_x, tau_s), = C.calibrate_stack([(w, proxy)], cal, s1, s2, 200000,
                                        W.reservoir_draws(cfg.seed))
    cal_s = time.perf_counter() - t0
    counts = torch.zeros((args.steps, 2), dtype=torch.int32, device=dev)

    def call(i):
        prox.ffn_sparse_tau(w, proxy, xs[i % n_x], tau_x, tau_s, y=y, mask=mask,
                            counts=counts[i % args.steps], ws=ws)

    for i in range(args.warmup):
        call(i)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    for i in range(args.steps):
        if not args.warm:
            torch.sum(flush, 0, out=sink)
        evs[i][0].record()
        call(i)
        evs[i][1].record()
    torch.cuda.synchronize()
    us = [a.elapsed_time(b) * 1e3 for a, b in evs]
    cnt = counts.cpu().numpy()
    byts = [sum(algorithmic_bytes(cfg, B, int(a), int(b)).values()) for a, b in cnt]
    mean = statistics.mean(us)
    return {"rule": "keep |x| >= tau_x and score >= tau_s (layer-wise thresholds)",
            "tau_x": tau_x, "tau_s": tau_s,
            "calibration": f"Alg. 1 on {args.calib_tokens} held-out synthetic vectors, "
                           f"reservoir 200000, targets s1={s1:.4f} s2={s2:.4f}, {cal_s:.1f} s",
            "us_per_call": {"mean": round(mean, 2), "median": round(statistics.median(us), 2),
                            "p10": round(pct(us, 0.1), 2), "p90": round(pct(us, 0.9), 2)},
            "k_in": {"mean": round(float(cnt[:, 0].mean()), 1), "min": int(cnt[:, 0].min()),
                     "max": int(cnt[:, 0].max())},
            "k_ff": {"mean": round(float(cnt[:, 1].mean()), 1), "min": int(cnt[:, 1].min()),
                     "max": int(cnt[:, 1].max())},
            "algorithmic_gbs": round(statistics.mean(byts) / (mean * 1e-6) / 1e9, 1),
            "speedup_vs_dense": None if dense_us is None
            else round(dense_us / statistics.median(us), 3)}


def bench_alpha(args, np, torch, prox, W, dev):
    """Sec. 4.2 proxy-cost ratio alpha on this GPU: the Stage 1 time with the
    workload's quantised proxy over the time with the unquantised 16-bit
    proxy (PROX_Q_NONE), at the same input sparsity, cold.  Stage 1 is the
    proxy kernel between the staged entry point's events.  Its input
    selection is the same for both formats."""
    cfg = W.CONFIGS[args.workload]
    wl = W.make_workload(cfg)
    w = prox.Weights(*(prox.from_bits(m, cfg.dtype, dev) for m in (wl.w_gate, wl.w_up, wl.w_down)))
    fmt = prox.INT4 if cfg.qbits == 4 else prox.INT8
    proxies = {"quant": prox.pack_proxy(w, fmt, cfg.group), "none": prox.pack_proxy(w, prox.NONE)}
    n_x = 8
    xs = prox.from_bits(wl.x_vectors(n_x, 1)[:, 0, :], cfg.dtype, dev)
    ws = prox.new_workspace(cfg.d_model, cfg.d_ff, 1, dev)
    y = torch.empty((1, cfg.d_model), dtype=w.dtype, device=dev)
    mask = torch.empty(cfg.d_ff, dtype=torch.uint8, device=dev)
    flush = torch.ones(FLUSH_BYTES // 8, dtype=torch.int64, device=dev)
    sink = torch.zeros((), dtype=torch.int64, device=dev)
    rows = []
    for s1 in (0.0, 0.1, 0.55, 0.7):
        k_in = max(1, W.frac_to_k(1.0 - s1, cfg.d_model))
        med = {}
        for name, p in proxies.items():
            stage = [[torch.cuda.Event(enable_timing=True) for _ in range(prox.SPARSE_STAGES + 1)]
                     for _ in range(args.steps)]
            for row in stage:
                for ev in row:
                    ev.record()
            for i in range(args.warmup):
                prox.ffn_sparse(w, p, xs[i % n_x], k_in, cfg.k_ff, y=y, mask=mask, ws=ws)
            torch.cuda.synchronize()
            for i in range(args.steps):
                torch.sum(flush, 0, out=sink)
                prox.ffn_sparse(w, p, xs[i % n_x], k_in, cfg.k_ff, y=y, mask=mask, ws=ws,
                                events=stage[i])
            torch.cuda.synchronize()
            med[name] = statistics.median(r[0].elapsed_time(r[1]) * 1e3 for r in stage)
        rows.append({"input_sparsity": s1, "k_in": k_in, "quant_us": round(med["quant"], 2),
                     "none_us": round(med["none"], 2),
                     "alpha": round(med["quant"] / med["none"], 3)})
    alphas = [r["alpha"] for r in rows]
    out = {"metric": "proxy-cost ratio alpha (Stage 1 time, quantised over 16-bit proxy)",
           "value": round(statistics.mean(alphas), 3), "unit": "ratio", "n_gpus": 1,
           "higher_is_better": False, "config": {"workload": cfg.name,
           "proxy": f"int{cfg.qbits} group {cfg.group} vs unquantised {W.DTYPE_NAMES[cfg.dtype]}"},
           "rows": rows, "protocol": "cold, median of the staged proxy-stage time",
           "paper_alpha": 1.0 / 3.0}
    print(json.dumps(out), flush=True)


def cpu_baseline(args, cfg, wl, xs_np, B, k_in, k_ff, total_bytes):
    """The CPU oracle as it stands, timed on this host on a bounded sample of
    the same workload (proxy quantised once beforehand, untimed): sparse calls
    for the budget, then dense calls for half of it."""
    import oracle
    cg, sg = oracle.quantize(wl.w_gate, cfg.dtype, cfg.qbits, cfg.group)
    cu, su = oracle.quantize(wl.w_up, cfg.dtype, cfg.qbits, cfg.group)

    def run(fn, budget):
        n = 0
        t0 = time.perf_counter()
        while (time.perf_counter() - t0) < budget:   # decode vectors in turn
            fn(xs_np[n % len(xs_np)])
            n += 1
        return (time.perf_counter() - t0) / max(n, 1), n, time.perf_counter() - t0

    dt, n, spent = run(lambda x: oracle.ffn_sparse(x, cfg.dtype, wl.w_gate, wl.w_up, wl.w_down,
                                                   k_in, k_ff, codes_g=cg, scales_g=sg,
                                                   codes_u=cu, scales_u=su, group=cfg.group),
                       args.cpu_budget_s)
    ddt, dn, dspent = run(lambda x: oracle.ffn_dense(x, cfg.dtype, wl.w_gate, wl.w_up,
                                                     wl.w_down), args.cpu_budget_s / 2)
    return {"value": round(total_bytes / dt / 1e9, 3), "unit": "GB/s", "cores": oracle.max_threads(),
            "nproc": os.cpu_count(), "kind": "oracle", "us_per_call": round(dt * 1e6, 1),
            "dense_us_per_call": round(ddt * 1e6, 1),
            "sample": f"{n} sparse decode calls ({spent:.1f} s) and {dn} dense calls "
                      f"({dspent:.1f} s) of {cfg.name} at batch {B} over the bench's decode "
                      f"vectors (fp64 C oracle, OpenMP; proxy quantised beforehand)"}


def torch_dense_leg(args, w, xs, n_x, flush, sink, torch):
    """A dense FFN through torch (hipBLASLt GEMVs: F.linear for gate and up,
    SiLU product, matmul for down), timed like the HIP dense FFN: a check that
    the dense baseline of the speedup is competitive."""
    import torch.nn.functional as F

    def call(i):
        x = xs[i % n_x]
        h = F.silu(F.linear(x, w.w_gate)) * F.linear(x, w.w_up)
        return torch.matmul(h, w.w_down)

    for i in range(args.warmup):
        call(i)
    us = []
    for i in range(args.steps):
        torch.sum(flush, 0, out=sink)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        call(i)
        b.record()
        us.append((a, b))
    torch.cuda.synchronize()
    v = [a.elapsed_time(b) * 1e3 for a, b in us]
    return {"us_per_call": round(statistics.median(v), 2),
            "what": "torch bf16 F.linear(x, W_gate), F.linear(x, W_up), SiLU product, "
                    "matmul with W_down; cold, median"}


def timed_calls(fn, n, flush, sink, torch, cold=True):
    """Per-call HIP-event times (µs) of n calls, each after a 1 GiB cache flush."""
    evs = []
    for i in range(n):
        if cold:
            torch.sum(flush, 0, out=sink)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        fn(i)
        b.record()
        evs.append((a, b))
    torch.cuda.synchronize()
    return [a.elapsed_time(b) * 1e3 for a, b in evs]


def config_legs(args, np, torch, prox, W, dev):
    """The other synthetic workloads, each timed cold like the headline (median
    of --config-steps calls) next to the dense HIP FFN: C1, C2, C3 at 70% FFN
    sparsity and batch 1, 4, 16, and the 36-layer C5 stack per token."""
    flush = torch.ones(FLUSH_BYTES // 8, dtype=torch.int64, device=dev)
    sink = torch.zeros((), dtype=torch.int64, device=dev)
    n = args.config_steps
    out = {}
    runs = [("c1_1024x3072_f16", 1), ("c2_4096x12288_bf16", 1), ("c3_4096x14336_bf16", 1),
            ("c3_4096x14336_bf16", 4), ("c3_4096x14336_bf16", 16)]
    loaded = {}
    for name, B in runs:
        cfg = W.CONFIGS[name]
        if name not in loaded:
            loaded.clear()
            torch.cuda.empty_cache()
            wl = W.make_workload(cfg)
            w = prox.Weights(*(prox.from_bits(m, cfg.dtype, dev)
                               for m in (wl.w_gate, wl.w_up, wl.w_down)))
            p = prox.pack_proxy(w, prox.INT4 if cfg.qbits == 4 else prox.INT8, cfg.group)
            loaded[name] = (wl, w, p)
        wl, w, p = loaded[name]
        k_ff = W.frac_to_k(0.3, cfg.d_ff) if name.startswith("c3") else cfg.k_ff
        n_x = 8
        xs = prox.from_bits(wl.x_vectors(n_x, B).reshape(n_x, B * cfg.d_model), cfg.dtype,
                            dev).view(n_x, B, cfg.d_model)
        ws = prox.new_workspace(cfg.d_model, cfg.d_ff, B, dev)
        y = torch.empty((B, cfg.d_model), dtype=w.dtype, device=dev)
        mask = torch.empty(cfg.d_ff, dtype=torch.uint8, device=dev)

        def sparse(i):
            prox.ffn_sparse(w, p, xs[i % n_x], cfg.k_in, k_ff, y=y, mask=mask, ws=ws)

        def dense(i):
            prox.ffn_dense(w, xs[i % n_x], y=y, ws=ws)

        for i in range(args.warmup):
            sparse(i)
            dense(i)
        su = statistics.median(timed_calls(sparse, n, flush, sink, torch))
        du = statistics.median(timed_calls(dense, n, flush, sink, torch))
        byts = sum(algorithmic_bytes(cfg, B, cfg.k_in, k_ff).values())
        out[f"{name}_b{B}"] = {
            "d_model": cfg.d_model, "d_ff": cfg.d_ff, "batch": B, "k_in": cfg.k_in, "k_ff": k_ff,
            "ffn_sparsity_s2": round(1 - k_ff / cfg.d_ff, 4),
            "us_per_call": round(su, 2), "tokens_per_s": round(B * 1e6 / su, 1),
            "algorithmic_bytes": byts, "gbs": round(byts / (su * 1e-6) / 1e9, 1),
            "hbm_frac": round(byts / (su * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
            "dense_us_per_call": round(du, 2), "speedup_vs_dense": round(du / su, 3)}
        del ws, xs
    loaded.clear()
    torch.cuda.empty_cache()
    out["c5_stack36_4096x12288_bf16_b1"] = stack_leg(args, np, torch, prox, W, dev)
    return out


def stack_leg(args, np, torch, prox, W, dev):
    """The 36-layer stack per token (prox_ffn_sparse then the residual RMSNorm
    per layer, back to back on one stream), next to the dense stack."""
    L = W.STACK_LAYERS
    layers = []
    for l in range(L):
        cfg = W.stack_layer_config(l)
        wl = W.make_workload(cfg)
        w = prox.Weights(*(prox.from_bits(m, cfg.dtype, dev) for m in (wl.w_gate, wl.w_up, wl.w_down)))
        layers.append((w, prox.pack_proxy(w, prox.INT4, cfg.group)))
        del wl
    cfg = W.stack_layer_config(0)
    x0 = prox.from_bits(W.make_workload(cfg, weights=False).x_vectors(1, 1)[0], cfg.dtype, dev)
    ws = prox.new_workspace(cfg.d_model, cfg.d_ff, 1, dev)
    y, x = torch.empty_like(x0), torch.empty_like(x0)
    mask = torch.empty(cfg.d_ff, dtype=torch.uint8, device=dev)

    def token(dense=False):
        x.copy_(x0)
        for w, p in layers:
            if dense:
                prox.ffn_dense(w, x, y=y, ws=ws)
            else:
                prox.ffn_sparse(w, p, x, cfg.k_in, cfg.k_ff, y=y, mask=mask, ws=ws)
            prox.add_rmsnorm(x, y, 1e-6, out=x)

    def per_token(dense):
        token(dense)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(args.config_steps):
            token(dense)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / args.config_steps

    su, du = per_token(False), per_token(True)
    byts = sum(algorithmic_bytes(cfg, 1, cfg.k_in, cfg.k_ff).values()) * L
    out = {"layers": L, "k_in": cfg.k_in, "k_ff": cfg.k_ff, "us_per_token": round(su, 1),
           "tokens_per_s": round(1e6 / su, 1), "algorithmic_bytes_per_token": byts,
           "gbs": round(byts / (su * 1e-6) / 1e9, 1),
           "hbm_frac": round(byts / (su * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
           "dense_us_per_token": round(du, 1), "speedup_vs_dense": round(du / su, 3),
           "protocol": "back-to-back tokens (12.7 GB of weights per token exceed the caches)"}
    del layers
    torch.cuda.empty_cache()
    return out


def bench_stack(args, np, torch, prox, W, dev):
    """36-layer stack: per token, prox_ffn_sparse then residual RMSNorm per
    layer, back-to-back on one stream."""
    L = W.STACK_LAYERS
    layers = []
    t_gen = time.perf_counter()
    for l in range(L):
        cfg = W.stack_layer_config(l)
        wl = W.make_workload(cfg)
        w = prox.Weights(*(prox.from_bits(m, cfg.dtype, dev) for m in (wl.w_gate, wl.w_up, wl.w_down)))
        layers.append((w, prox.pack_proxy(w, prox.INT4, cfg.group)))
        del wl
    cfg = W.stack_layer_config(0)
    x0 = prox.from_bits(W.make_workload(cfg, weights=False).x_vectors(1, 1)[0], cfg.dtype, dev)
    ws = prox.new_workspace(cfg.d_model, cfg.d_ff, 1, dev)
    y = torch.empty_like(x0)
    x = torch.empty_like(x0)
    mask = torch.empty(cfg.d_ff, dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    gen_s = time.perf_counter() - t_gen

    def token(dense=False):
        x.copy_(x0)
        for w, p in layers:
            if dense:
                prox.ffn_dense(w, x, y=y, ws=ws)
            else:
                prox.ffn_sparse(w, p, x, cfg.k_in, cfg.k_ff, y=y, mask=mask, ws=ws)
            prox.add_rmsnorm(x, y, 1e-6, out=x)

    for _ in range(args.warmup):
        token()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    t0 = time.perf_counter()
    for a, b in evs:
        a.record(); token(); b.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3
    us = [a.elapsed_time(b) * 1e3 for a, b in evs]
    dense_us = None
    if not args.no_dense:
        token(dense=True)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(args.steps):
            token(dense=True)
        b.record()
        torch.cuda.synchronize()
        dense_us = a.elapsed_time(b) * 1e3 / args.steps
    tau = None
    if not args.no_tau:
        tau = stack_threshold_leg(args, cfg, layers, x0, y, mask, ws, L, np, torch, prox, W, dev)
    ab = sum(algorithmic_bytes(cfg, 1, cfg.k_in, cfg.k_ff).values()) * L
    mean = statistics.mean(us)
    gbs = ab / (mean * 1e-6) / 1e9
    out = {"metric": "36-layer sparse FFN stack µs/token (back-to-back on one stream)",
           "value": round(1e6 / mean, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": round(mean / 1e3, 4), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
           "config": {"workload": "c5_stack36_4096x12288_bf16_b1", "layers": L,
                      "k_in": cfg.k_in, "k_ff": cfg.k_ff},
           "us_per_token": round(mean, 1), "achieved_gbs": round(gbs, 1),
           "hbm_frac": round(gbs / PEAK_HBM_GBS, 4), "dense_us_per_token":
               None if dense_us is None else round(dense_us, 1),
           "speedup_vs_dense": None if dense_us is None else round(dense_us / mean, 3),
           "protocol": "back-to-back tokens (12.7 GB of weights per token exceed the caches)",
           "wall_ms_timed_region": round(wall_ms, 1), "setup_s": round(gen_s, 1),
           "threshold_mode": tau}
    print(json.dumps(out), flush=True)


def stack_threshold_leg(args, cfg, layers, x0, y, mask, ws, L, np, torch, prox, W, dev):
    """The stack with per-layer thresholds from Alg. 1 (sequential, each layer
    calibrated on inputs that passed through the finished earlier layers) on
    held-out synthetic tokens, then timed per token like the top-k stack."""
    from paper_2607_27591_amd import calibrate as C
    s1, s2 = 1 - cfg.k_in / cfg.d_model, 1 - cfg.k_ff / cfg.d_ff
    cal = prox.from_bits(W.make_workload(cfg, weights=False).x_vectors(
        1 + args.calib_tokens, 1)[1:, 0, :], cfg.dtype, dev)
    t0 = time.perf_counter()
    taus = C.calibrate_stack(layers, cal, s1, s2, 200000, W.reservoir_draws(cfg.seed))
    cal_s = time.perf_counter() - t0
    counts = torch.zeros((L, 2), dtype=torch.int32, device=dev)
    x = torch.empty_like(x0)

    def token():
        x.copy_(x0)
        for l, ((w, p), (tx, ts)) in enumerate(zip(layers, taus)):
            prox.ffn_sparse_tau(w, p, x, tx, ts, y=y, mask=mask, counts=counts[l], ws=ws)
            prox.add_rmsnorm(x, y, 1e-6, out=x)

    for _ in range(args.warmup):
        token()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    for _ in range(args.steps):
        token()
    b.record()
    torch.cuda.synchronize()
    us = a.elapsed_time(b) * 1e3 / args.steps
    cnt = counts.cpu().numpy()
    return {"us_per_token": round(us, 1), "tokens_per_s": round(1e6 / us, 1),
            "calibration": f"Alg. 1 over {L} layers on {args.calib_tokens} held-out synthetic "
                           f"tokens, reservoir 200000, s1={s1:.4f} s2={s2:.4f}, {cal_s:.1f} s",
            "k_in_mean": round(float(cnt[:, 0].mean()), 1),
            "k_ff_mean": round(float(cnt[:, 1].mean()), 1),
            "k_ff_range": [int(cnt[:, 1].min()), int(cnt[:, 1].max())]}


if __name__ == "__main__":
    main()
