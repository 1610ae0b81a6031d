"""Benchmark: ResNet-50 batch-1 fp32 inference through the blocked-layout plan.

One step = one forward pass of ResNet-50 (224x224, batch 1) through
``neo_run_graph``: the entry layout transform, 53 blocked convolutions with
their fused epilogues, max pool, global average pool, the exit transform
(aliased) and the dense layer.  Input and parameters are resident in HBM
before the timed region.

Printed JSON line (rank 0, one line):
  value      conv TFLOP/s over the whole step (8.174 GFLOP of convolution per
             image / step time); ``latency_ms`` is the step time itself
  roofline   the dominant kernel (conv2d_blocked): algorithmic FLOPs per
             launch / average launch duration, measured with HIP events on the
             launch stream over the 23 distinct ResNet-50 layers weighted by
             their use count (53 launches per forward)
  layers     the per-layer sweep (TFLOP/s, algorithmic GB/s, % of the binding
             roofline)
  cpu_baseline  the CPU oracle timed on this host on a bounded sample
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_TFLOPS = 157.3    # MI355X dense fp32 matrix peak
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def conv_costs(C, K, R, S, H, W, st, pd, N=1, residual=False):
    """Algorithmic FLOPs (real C, no padding) and bytes of one convolution."""
    OH = (H + 2 * pd[0] - R) // st[0] + 1
    OW = (W + 2 * pd[1] - S) // st[1] + 1
    flops = 2 * N * K * C * R * S * OH * OW
    if R == 1 and S == 1:
        touched = N * C * OH * OW          # a strided 1x1 reads only the sampled pixels
    else:
        touched = N * C * H * W
    nbytes = 4 * (touched + K * C * R * S + N * K * OH * OW * (2 if residual else 1) + K)
    return flops, nbytes, OH, OW


def build_plan_inputs(neo, torch, flags=0):
    from paper_1809_02697_amd import workloads as wl
    g = wl.resnet50(1)
    plan = neo.Plan(g, flags=flags)
    x = torch.from_numpy(g.x).cuda()
    out = torch.empty((1, 1000), device="cuda")
    flops = 0
    d = plan.describe()
    for s in d["steps"]:
        if s["kind"] == "conv":
            c = s["conv"]
            flops += conv_costs(c["C"], c["K"], c["R"], c["S"], c["H"], c["W"], c["stride"],
                                c["pad"])[0]
    return g, plan, x, out, flops


def layer_sweep(neo, torch, reps):
    """Config 2: the 23 distinct ResNet-50 layers, each timed alone with HIP
    events around every launch (torch events on the launch stream)."""
    from paper_1809_02697_amd import workloads as wl
    rows = []
    stream = torch.cuda.current_stream()
    for c in wl.resnet50_layer_sweep(1):
        w, b = neo.fold_bn(c.w, c.bias, c.bn["gamma"], c.bn["beta"], c.bn["mean"], c.bn["var"],
                           c.bn["eps"])
        bpad = np.zeros(neo.cblocks(c.K) * 16, np.float32)
        bpad[:c.K] = b
        wp = neo.pack_filter(torch.from_numpy(w).cuda())
        bias = torch.from_numpy(bpad).cuda()
        xb = neo.to_blocked(torch.from_numpy(c.x).cuda())
        res = neo.to_blocked(torch.from_numpy(c.residual).cuda()) if c.epilogue == "res" else None
        act = "none" if c.epilogue == "none" else "relu"
        flops, nbytes, OH, OW = conv_costs(c.C, c.K, c.R, c.S, c.H, c.W, c.stride, c.pad,
                                           residual=res is not None)
        y = torch.empty((1, neo.cblocks(c.K), OH, OW, 16), device="cuda")

        def launch():
            neo.conv2d_blocked(xb, c.C, wp, c.K, c.R, c.S, bias=bias, stride=c.stride,
                               pad=c.pad, act=act, residual=res, out=y)

        # `reps` back-to-back launches captured in one graph, so host launch
        # cost never shows between kernels; HIP events on the launch stream
        # bracket each replay.  Warm up on the capture stream first: the
        # library sizes its per-stream split workspace there, outside capture.
        cap = torch.cuda.Stream()
        with torch.cuda.stream(cap):
            for _ in range(3):
                launch()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=cap):
            for _ in range(reps):
                launch()
        graph.replay()
        torch.cuda.synchronize()
        t = []
        for _ in range(3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            graph.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            t.append(e0.elapsed_time(e1) * 1e3 / reps)
        t = np.array(t)
        us = float(np.mean(t))
        del graph
        tf = flops / (us * 1e-6) / 1e12
        gbs = nbytes / (us * 1e-6) / 1e9
        ai = flops / nbytes
        roof = min(PEAK_FP32_TFLOPS, ai * PEAK_HBM_GBS / 1e3)
        rows.append(dict(id=c.id, shape=f"{c.C}->{c.K} {c.R}x{c.S}/s{c.stride[0]} {c.H}->{OH}",
                         uses=c.uses, us=round(us, 2), us_min=round(float(t.min()), 2),
                         gflop=round(flops / 1e9, 4), tflops=round(tf, 2),
                         alg_gbs=round(gbs, 1),
                         bound="mfma" if ai * PEAK_HBM_GBS / 1e3 >= PEAK_FP32_TFLOPS else "hbm",
                         pct_mfma=round(100 * tf / PEAK_FP32_TFLOPS, 1),
                         pct_hbm=round(100 * gbs / PEAK_HBM_GBS, 1),
                         pct_roof=round(100 * tf / roof, 1)))
    return rows


def cpu_baseline(g, budget_s=12.0):
    """The oracle (plain C direct convolution, OpenMP on all host cores) on
    whole ResNet-50 batch-1 forwards until ~budget_s of work."""
    import oracle
    from paper_1809_02697_amd import workloads as wl  # noqa: F401
    flops = 8_174_272_512
    n = 0
    t0 = time.perf_counter()
    while True:
        oracle.run_graph(g)
        n += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    return dict(value=round(flops * n / dt / 1e12, 6), unit="TFLOP/s", cores=oracle.num_threads(),
                kind="oracle", ms_per_forward=round(dt / n * 1e3, 1),
                sample=f"{n} ResNet-50 batch-1 forward pass(es) through the oracle graph "
                       f"executor ({dt:.1f} s)")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--layer-reps", type=int, default=50)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-layers", action="store_true", help="skip the per-layer sweep")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the batch-1 path has no cross-GPU work "
              "(see the sharding note of the design); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_1809_02697_amd import neo
    neo.lib()
    assert torch.cuda.is_available(), "no GPU"
    g, plan, x, out, conv_flops = build_plan_inputs(neo, torch, neo.PLAN_HIPGRAPH)
    print(f"[bench] plan built: {len(plan.describe()['steps'])} steps", file=sys.stderr, flush=True)

    for _ in range(args.warmup):
        plan.run(x, out)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(args.steps):
        plan.run(x, out)
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = ev0.elapsed_time(ev1) / args.steps
    print(f"[bench] e2e {ms:.3f} ms/step (wall {wall * 1e3 / args.steps:.3f})", file=sys.stderr,
          flush=True)
    # the same plan launched step by step from the host, for reference
    eager = neo.Plan(g)
    for _ in range(3):
        eager.run(x, out)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(args.steps):
        eager.run(x, out)
    ev1.record()
    torch.cuda.synchronize()
    ms_eager = ev0.elapsed_time(ev1) / args.steps
    eager.destroy()

    layers, roofline = None, None
    if not args.no_layers:
        layers = layer_sweep(neo, torch, args.layer_reps)
        tot_f = sum(r["gflop"] * 1e9 * r["uses"] for r in layers)
        tot_t = sum(r["us"] * 1e-6 * r["uses"] for r in layers)
        n_launch = sum(r["uses"] for r in layers)
        achieved = (tot_f / n_launch) / (tot_t / n_launch) / 1e12
        roofline = dict(bound="mfma", achieved=round(achieved, 2), peak=PEAK_FP32_TFLOPS,
                        unit="TFLOP/s", frac=round(achieved / PEAK_FP32_TFLOPS, 4), traffic=None,
                        kernel="conv2d_blocked", launches_per_step=n_launch,
                        avg_launch_us=round(tot_t / n_launch * 1e6, 2),
                        flop_per_launch=round(tot_f / n_launch))
        print(f"[bench] conv sweep: {achieved:.2f} TFLOP/s over {n_launch} launches",
              file=sys.stderr, flush=True)

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(g)
        print(f"[bench] cpu oracle: {cpu['value']} TFLOP/s", file=sys.stderr, flush=True)

    value = conv_flops / (ms * 1e-3) / 1e12
    rec = {
        "metric": "conv TFLOP/s + % fp32 MFMA/HBM roofline; ResNet-50 batch-1 latency ms",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "latency_ms": round(ms, 4),
        "latency_ms_eager_launch": round(ms_eager, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp32",
        "data": "synthetic",
        "config": {"workload": "ResNet-50 forward, batch 1, 3x224x224 fp32, NCHW16c plan "
                               "(1 transform in, 1 out), seed 2; hipGraph replay",
                   "global_batch": 1, "conv_gflop_per_step": round(conv_flops / 1e9, 4),
                   "cache": "warm (working set resident in the 256 MB MALL)"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "layers": layers,
    }
    print(json.dumps(rec))
    plan.destroy()


if __name__ == "__main__":
    main()
