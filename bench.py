"""Encoder-stage forward + backward throughput on one MI355X.

One step = stage_forward + stage_backward of a block of post-LN BERT encoder
layers (every kernel of the hot path) over one batch of synthetic input
already resident in HBM.  Default workload: 4 BERT-large-shaped layers
(h 1024, 16 heads, FFN 4096), batch 32 x seq 512, no padding, bf16 storage
with fp32 accumulation.

Prints one JSON line: tokens/s, ms per step, TFLOP/s and fraction of the bf16
MFMA peak, a roofline entry for the dominant kernel (timed with HIP events on
the stage stream over the timed region), and the fp64 CPU oracle timed on a
bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0

# Kernels the roofline entry can report on: a kernel (one compiled
# instantiation) and the launch sites that use it in one step.
ROOFLINE_KERNELS = {
    # the four weight-gradient GEMMs of a layer, dW = dY^T X over all tokens
    # (split over tokens, fp32 partials), in one group launch: the kernel
    # with the largest share of step time
    "wgrad_gemm": ("gemm_bf16_kernel<256, 256, false, false, 4, true, true>",
                   ["wgrad_group_gemm"]),
    "ffn1_gelu_gemm": ("gemm_bf16_kernel<256, 256, true, true, 1, false, false>",
                       ["ffn1_gelu_gemm_fwd"]),
    "ffn2_dgrad_dgelu_gemm": ("gemm_bf16_kernel<256, 256, true, true, 2, false, false>",
                              ["ffn2_dgrad_dgelu_gemm"]),
}


def site_flops(site: str, cfg, lengths) -> float:
    """Algorithmic FLOPs of one launch of a GEMM site (2 M N K)."""
    T, h, f = cfg.batch * cfg.seq, cfg.hidden, cfg.ffn
    S, H = cfg.seq, cfg.heads
    table = {
        "qkv_gemm_fwd": 2.0 * T * 3 * h * h,
        "out_gemm_fwd": 2.0 * T * h * h,
        "ffn1_gelu_gemm_fwd": 2.0 * T * f * h,
        "ffn2_gemm_fwd": 2.0 * T * h * f,
        "w2_wgrad_gemm": 2.0 * h * f * T,
        "ffn2_dgrad_dgelu_gemm": 2.0 * T * f * h,
        "w1_wgrad_gemm": 2.0 * f * h * T,
        "ffn1_dgrad_resid_gemm": 2.0 * T * h * f,
        "wo_wgrad_gemm": 2.0 * h * h * T,
        "out_dgrad_gemm": 2.0 * T * h * h,
        "wqkv_wgrad_gemm": 2.0 * 3 * h * h * T,
        "qkv_dgrad_resid_gemm": 2.0 * T * h * 3 * h,
        # W_2, W_1, W_o and W_qkv gradients in one launch
        "wgrad_group_gemm": 2.0 * T * (2 * h * f + 4 * h * h),
    }
    for k in ("scores_gemm_fwd", "context_gemm_fwd", "dp_gemm_bwd", "dv_gemm_bwd", "dq_gemm_bwd",
              "dk_gemm_bwd"):
        table[k] = 2.0 * cfg.batch * H * S * S * 64
    return table.get(site, 0.0)


def roofline_traffic(key: str, kernel_name: str):
    """HBM bytes per launch of the roofline kernel from the rocprofv3 --pmc
    record under profiles/ (FETCH_SIZE and WRITE_SIZE, scaled by a plain copy
    of known size), or None when no record exists or the GEMM source changed
    since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "roofline_traffic.json")
    src = os.path.join(ROOT, "paper_2202_11836_amd", "csrc", "gemm.hip")
    try:
        rec = json.load(open(path)).get(key)
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    except (OSError, ValueError):
        return None
    if not rec or rec.get("kernel") != kernel_name or rec.get("source_sha256") != sha:
        return None
    return rec["bytes_per_launch"]


def cpu_baseline(cfg, budget_s: float = 10.0):
    """Time the fp64 oracle on whole sequences of the workload (same layers,
    shapes and distributions), repeating until budget_s has elapsed."""
    import numpy as np

    import oracle
    import synth
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = os.cpu_count() or 1
    one = cfg.with_(batch=1)
    params = synth.make_params(one)
    inp = synth.make_inputs(one)
    t0 = time.perf_counter()
    n = 0
    while True:
        y, saved = oracle.stage_forward(inp["x"], inp["mask"], params, cfg.heads)
        oracle.stage_backward(inp["dy"], saved, params)
        n += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    return {"value": n * cfg.seq / dt, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{n} x one sequence of {cfg.seq} tokens through all {cfg.L} layers, "
                      f"fwd+bwd, fp64 numpy ({dt:.1f} s)"}


def depth_sweep(cfg, depths, steps, warmup):
    """Per-layer forward+backward time of cfg at several depths L, and the
    least-squares line t(L) = a L + b over them: the allocator models a
    device's time for a contiguous block of layers as the sum of per-layer
    costs plus a constant (section IV-C), which holds when the fit is
    tight and b is small."""
    import numpy as np
    import torch

    import synth
    from paper_2202_11836_amd import Stage

    inp = synth.make_inputs(cfg)
    dtype = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    x = torch.from_numpy(inp["x"].astype(np.float32)).to(dtype).cuda()
    dy = torch.from_numpy(inp["dy"].astype(np.float32)).to(dtype).cuda()
    mask = torch.from_numpy(inp["mask"]).cuda()
    rows = []
    for L in depths:
        st = Stage(L, cfg.hidden, cfg.heads, cfg.ffn, seed=cfg.seed, dtype=cfg.dtype)
        y = torch.empty_like(x)
        dx = torch.empty_like(x)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        for _ in range(warmup):
            st.forward(x, mask, out=y)
            st.backward(dy, out=dx)
        torch.cuda.synchronize()
        fs, bs = [], []
        for _ in range(steps):
            ev[0].record()
            st.forward(x, mask, out=y)
            ev[1].record()
            st.backward(dy, out=dx)
            ev[2].record()
            torch.cuda.synchronize()
            fs.append(ev[0].elapsed_time(ev[1]))
            bs.append(ev[1].elapsed_time(ev[2]))
        st.close()
        # medians over the steps (a step's fwd and bwd from the same events)
        fwd, bwd = float(np.median(fs)), float(np.median(bs))
        rows.append({"L": L, "fwd_ms": fwd, "bwd_ms": bwd, "step_ms": fwd + bwd,
                     "per_layer_ms": (fwd + bwd) / L})
        print(f"L={L:3d}  step {fwd + bwd:8.3f} ms  per layer {(fwd + bwd) / L:7.3f} ms",
              file=sys.stderr, flush=True)
    Ls = np.array([r["L"] for r in rows], dtype=np.float64)
    ts = np.array([r["step_ms"] for r in rows])
    a, b = np.polyfit(Ls, ts, 1) if len(rows) > 1 else (ts[0] / Ls[0], 0.0)
    pred = a * Ls + b
    ss = float(((ts - ts.mean()) ** 2).sum())
    r2 = 1.0 - float(((ts - pred) ** 2).sum()) / ss if ss > 0 else 1.0
    return {
        "metric": "per-layer fwd+bwd time vs stage depth on 1 MI355X",
        "unit": "ms",
        "higher_is_better": False,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded N(0,1) inputs, N(0,0.02) weights)",
        "steps": steps,
        "warmup": warmup,
        "timing": "fwd_ms, bwd_ms: medians over the steps of HIP events on the stage stream",
        "config": {"workload": f"{cfg.name}: h{cfg.hidden}, {cfg.heads} heads, ffn {cfg.ffn}, "
                               f"B{cfg.batch} x S{cfg.seq}, valid lengths in "
                               f"[{cfg.len_lo},{cfg.len_hi}]"},
        "sweep": rows,
        "fit": {"ms_per_layer": float(a), "ms_constant": float(b), "r2": r2},
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="bert_large_4")
    ap.add_argument("--layers", type=int, default=None, help="override L (depth sweep)")
    ap.add_argument("--roofline-kernel", default="wgrad_gemm", choices=sorted(ROOFLINE_KERNELS))
    ap.add_argument("--breakdown", action="store_true", help="per-site times to stderr")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=10.0)
    ap.add_argument("--sweep-layers", default=None,
                    help="comma-separated depths: time --config at each depth and report the "
                         "per-layer fwd+bwd time and a linear fit of step time against depth "
                         "(the per-layer cost model of the layer allocator, section IV-C)")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="after timing, copy a fresh buffer of this size once (the known-size "
                         "copy that scales rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(a stage shards by layers across GPUs; see the design notes).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    from paper_2202_11836_amd import Stage, stage_mfma_peak, stage_site_count, stage_site_name

    cfg = synth.CONFIGS[args.config]
    if args.sweep_layers:
        torch.cuda.set_device(0)
        print(json.dumps(depth_sweep(cfg, [int(v) for v in args.sweep_layers.split(",")],
                                     args.steps, args.warmup)), flush=True)
        return
    if args.layers is not None:
        cfg = cfg.with_(L=args.layers)
    torch.cuda.set_device(0)
    inp = synth.make_inputs(cfg)
    dtype = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    x = torch.from_numpy(inp["x"].astype(np.float32)).to(dtype).cuda()
    dy = torch.from_numpy(inp["dy"].astype(np.float32)).to(dtype).cuda()
    mask = torch.from_numpy(inp["mask"]).cuda()
    st = Stage(cfg.L, cfg.hidden, cfg.heads, cfg.ffn, seed=cfg.seed, dtype=cfg.dtype)
    y = torch.empty_like(x)
    dx = torch.empty_like(x)

    def step():
        st.forward(x, mask, out=y)
        st.backward(dy, out=dx)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # Timed region: exactly --steps steps.  Each step is bracketed by HIP
    # events on the stage stream (torch's current stream), with one more
    # between its forward and backward, so the per-step median and spread
    # and the forward / backward split (the paper reports them separately)
    # come from the same timed steps; the dominant kernel's launches are
    # traced with HIP events on that stream as well.
    kernel_name, roof_sites = ROOFLINE_KERNELS[args.roofline_kernel]
    st.trace(roof_sites)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        ev[i][0].record()
        st.forward(x, mask, out=y)
        ev[i][1].record()
        st.backward(dy, out=dx)
        ev[i][2].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    launches, site_ms = st.trace_read()
    st.trace(None)
    fwd_s = np.array([e[0].elapsed_time(e[1]) for e in ev])
    bwd_s = np.array([e[1].elapsed_time(e[2]) for e in ev])
    step_s = np.array([e[0].elapsed_time(e[2]) for e in ev])
    fwd_ms, bwd_ms = float(np.median(fwd_s)), float(np.median(bwd_s))

    ms_per_step = (t1 - t0) * 1000.0 / args.steps
    tokens = cfg.batch * cfg.seq
    flops = synth.flops_per_step(cfg, inp["lengths"] if cfg.len_lo is not None else None)
    tflops = flops / (ms_per_step / 1000.0) / 1e12

    # Algorithmic FLOPs per launch: 2 M N K of each traced launch in a step,
    # averaged over the step's launches of the kernel.
    per_launch_flops = sum(site_flops(s, cfg, inp["lengths"]) for s in roof_sites) / len(roof_sites)
    avg_ms = site_ms / max(launches, 1)
    achieved = per_launch_flops / (avg_ms / 1000.0) / 1e12 if launches else 0.0
    traffic = roofline_traffic(args.roofline_kernel, kernel_name)

    if args.breakdown:
        rows = []
        for i in range(stage_site_count()):
            name = stage_site_name(i)
            st.trace(name)
            step()
            n, ms = st.trace_read()
            rows.append((name, n, ms))
        st.trace(None)
        total = sum(r[2] for r in rows)
        print(f"{'site':32s} {'launches':>8s} {'ms/step':>9s} {'share':>6s} {'TFLOP/s':>8s}",
              file=sys.stderr)
        for name, n, ms in sorted(rows, key=lambda r: -r[2]):
            fl = site_flops(name, cfg, inp["lengths"]) * n
            tf = fl / (ms / 1000.0) / 1e12 if ms > 0 and fl > 0 else 0.0
            print(f"{name:32s} {n:8d} {ms:9.3f} {100 * ms / total:5.1f}% {tf:8.1f}", file=sys.stderr)
        print(f"{'sum of kernels':32s} {'':8s} {total:9.3f}", file=sys.stderr)

    # The device's achievable dense bf16 MFMA rate and the clock it holds
    # under that load (register-only MFMA chains, after the timed region).
    peak_tf, peak_ghz = stage_mfma_peak(20000)

    out = {
        "metric": "encoder-stage fwd+bwd tokens/s and % bf16 MFMA peak on 1 MI355X",
        "value": tokens / (ms_per_step / 1000.0),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "step_ms_median": float(np.median(step_s)),
        "step_ms_spread": {"min": float(step_s.min()), "p10": float(np.percentile(step_s, 10)),
                           "p90": float(np.percentile(step_s, 90)), "max": float(step_s.max())},
        "fwd_ms": fwd_ms,
        "bwd_ms": bwd_ms,
        "timing": "value and ms_per_step: wall clock over the timed steps (mean); "
                  "step_ms_median / spread, fwd_ms, bwd_ms: medians of per-step HIP events "
                  "on the stage stream over the same steps",
        "tflops": tflops,
        "pct_bf16_peak": 100.0 * tflops / PEAK_BF16_TFLOPS,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded N(0,1) inputs, N(0,0.02) weights; stands in for MNLI)",
        "config": {
            "workload": f"{cfg.name}: {cfg.L} post-LN encoder layers, h{cfg.hidden}, "
                        f"{cfg.heads} heads, ffn {cfg.ffn}, B{cfg.batch} x S{cfg.seq}, "
                        + ("no padding" if cfg.len_lo is None else
                           f"valid lengths in [{cfg.len_lo},{cfg.len_hi}]"),
            "L": cfg.L, "hidden": cfg.hidden, "heads": cfg.heads, "ffn": cfg.ffn,
            "global_batch": cfg.batch, "seq_len": cfg.seq, "gflop_per_step": flops / 1e9,
        },
        "roofline": {
            "kernel": kernel_name,
            "sites": roof_sites,
            "bound": "mfma",
            "achieved": achieved,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS,
            "traffic": traffic,
            "launches": launches,
            "avg_launch_ms": avg_ms,
            "flop_per_launch": per_launch_flops,
            "frac_of_measured_peak": achieved / peak_tf if peak_tf > 0 else None,
        },
        "mfma_peak_measured": {
            "tflops": peak_tf,
            "clock_ghz": peak_ghz,
            "frac_of_published": peak_tf / PEAK_BF16_TFLOPS,
            "step_frac": tflops / peak_tf if peak_tf > 0 else None,
            "method": "one work-group of 8 wavefronts per CU, 8 independent chains of "
                      "32x32x16 bf16 MFMAs on registers per wavefront, HIP events; clock from "
                      "the shader-cycle counter over the constant-rate counter",
        },
    }
    st.close()
    if args.calibrate_copy_mib > 0:
        n = args.calibrate_copy_mib * (1 << 20) // 4
        src = torch.arange(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
