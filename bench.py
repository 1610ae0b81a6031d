"""Benchmark: ResNet-50 batch-1 fp32 inference through the blocked-layout plan.

One step = one forward pass of ResNet-50 (224x224, batch 1) through
``neo_run_graph`` on the full method's plan -- local search of every conv's
launch configuration, global layout search over each conv's (ic_bn, oc_bn),
transforms only where the chosen layouts differ -- replayed as a HIP graph:
the entry layout transform, 53 blocked convolutions with their fused
epilogues, max pool, global average pool, the exit transform (aliased) and
the dense layer.  Input, output and parameters are resident in HBM before the
timed region.

Printed JSON line:
  value        conv TFLOP/s over the whole step (8.174 GFLOP of convolution
               per image / step time); ``latency_ms`` is the step time
  roofline     the dominant kernel, conv2d_blocked: algorithmic FLOPs per
               launch / average launch duration, each conv step of the plan
               timed with HIP events around back-to-back graph replays on the
               plan's stream (sum_conv_us: the forward's conv launches summed,
               at most ms_per_step); a kernel trace of the forwards launched
               step by step (stepwise_forward_ms) gives the same per-launch
               durations from the hardware's own timestamps
  latency      per-forward latency over 1000 single runs: mean, standard
               error, median (warm caches: the batch-1 working set stays in
               the 256 MB MALL between runs)
  layers       per distinct conv shape: us, TFLOP/s, algorithmic GB/s, % of
               the binding roofline, and the launch configuration (warm);
               cold_us / cold_hbm_gbs: the same launch after a 512 MB read
               has flushed the caches, so its operands come from HBM;
               cold_copy_gbs: a plain copy under the same protocol
  models       end-to-end latency of ResNet-50 / VGG-16 / Inception-v3 at
               batch 1 and ResNet-50 at batch 32 for the ablation of Table 3:
               "naive" (transforms around every blocked operation), "eliminated"
               (one block for every conv, transforms only at the ends) and
               "searched" (the global layout search); plus "grouped" (the
               eliminated plan with independent convs fused into launches, pools
               riding along, a global pool folded into its neighbours, pairs
               of pointwise convs and 3x3-led chains fused); all
               with tuned launch configurations
  cpu_baseline the CPU oracle timed on this host on a bounded sample
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


def plan_schemes(desc):
    """{conv node: (ic_bn, oc_bn)} of a plan description."""
    out = {}
    for s in desc["steps"]:
        for m in (s["members"] if s["kind"] in ("conv_group", "conv_pair", "conv_chain", "conv_pool")
                  else [s] if s["kind"] == "conv" else []):
            out[m["node"]] = (m["conv"]["ic_bn"], m["conv"]["oc_bn"])
    return out


def headline_plan(neo, g, tune_db=None, torch=None, steps=100, warmup=10):
    """The plan bench.py times, and how it was chosen.  The global search
    (Section 3.3.2) chooses every conv's scheme from per-conv times measured
    in isolation; the resulting plan and the one-block plan (Section 3.2, all
    convs in NCHW16c) -- both with independent convs fused into launches,
    the global pool folded into the last conv and the dense layer, pairs
    of pointwise convs, 3x3-led chains and the stem with its max pool in one
    launch -- are then both timed end to end and the faster is kept,
    so a search decision that the isolated timings mispredict cannot make the
    step slower.  The kept plan is then timed in both launch modes, replayed
    as one captured hipGraph and with its steps launched one by one on the
    stream, under the protocol of the timed region (`warmup` forwards, then
    `steps` timed), and the faster mode is kept too: stream launches cost the
    GPU less per kernel, but the host's first forward after a synchronize
    enqueues more slowly than graph replay, which short timed regions see.  With a results file from an
    earlier run (``--tune-db``) the schemes and the launch mode that run kept
    are reused from ``<file>.schemes.json`` (so a profiling run executes the
    same plan)."""
    path = (tune_db or "") + ".schemes.json"
    base = (neo.PLAN_GROUP | neo.PLAN_FUSE_GAP | neo.PLAN_FUSE_PAIRS |
            neo.PLAN_FUSE_CHAINS | neo.PLAN_FUSE_POOL)
    if tune_db and os.path.exists(path):
        saved = json.load(open(path))
        sch = {int(k): tuple(v) for k, v in saved["schemes"].items()}
        graph = neo.PLAN_HIPGRAPH if saved["launch"] == "graph" else 0
        return (neo.Plan(g, flags=neo.PLAN_TUNE | base | graph, schemes=sch),
                {"from": path, "launch": saved["launch"]})
    searched = neo.Plan(g, flags=neo.PLAN_GLOBAL_SEARCH | neo.PLAN_HIPGRAPH | base)
    fixed = neo.Plan(g, flags=neo.PLAN_TUNE | neo.PLAN_HIPGRAPH | base)
    x = torch.from_numpy(g.x).cuda()
    out = torch.empty(searched.output_shape[:2], device="cuda")
    t_s = min(e2e_ms(torch, searched, x, out, 100, 10) for _ in range(3))
    t_f = min(e2e_ms(torch, fixed, x, out, 100, 10) for _ in range(3))
    d = searched.describe()
    info = {"searched_ms": round(t_s, 4), "fixed16_ms": round(t_f, 4),
            "searched_schemes": scheme_summary(d),
            "search_predicted_us": round(d["search"]["cost_us"], 1),
            "search_predicted_fixed16_us": round(d["search"]["fixed_block_cost_us"], 1)}
    keep, drop = (searched, fixed) if t_s <= t_f else (fixed, searched)
    info["kept"] = "searched" if keep is searched else "fixed16"
    drop.destroy()
    # the same plan (schemes and tuned configurations) without the captured
    # graph: the host enqueues each step in less time than the GPU runs it
    kd = keep.describe()
    stream = neo.Plan(g, flags=neo.PLAN_TUNE | base, schemes=plan_schemes(kd))
    assert same_steps(stream.describe(), kd), "the stream-launched plan differs from the kept plan"
    t_g, t_d = 1e30, 1e30
    for _ in range(5):
        t_g = min(t_g, e2e_ms(torch, keep, x, out, steps, warmup))
        t_d = min(t_d, e2e_ms(torch, stream, x, out, steps, warmup))
    info["graph_ms"], info["stream_ms"] = round(t_g, 4), round(t_d, 4)
    keep, drop = (keep, stream) if t_g <= t_d else (stream, keep)
    info["launch"] = "graph" if keep.describe()["hipgraph"] else "stream"
    drop.destroy()
    return keep, info


def same_steps(a, b):
    """Two plan descriptions run the same steps with the same configurations."""
    return json.dumps(a["steps"], sort_keys=True) == json.dumps(b["steps"], sort_keys=True)


def conv_launches(desc):
    """The plan's conv launches: (step index, [(conv fields, has residual)],
    launch configuration) -- one conv, or the members of a fused group."""
    out = []
    for i, s in enumerate(desc["steps"]):
        if s["kind"] == "conv":
            c = s["conv"]
            cfg = dict(tile=c["tile"], split=c["split"], waves=c["waves"], ic_bn=c["ic_bn"],
                       oc_bn=c["oc_bn"])
            if c.get("algo") == "winograd":
                cfg["algo"] = "winograd"
            out.append((i, [(c, s["res"] >= 0)], cfg))
        elif s["kind"] == "conv_group":
            out.append((i, [(m["conv"], m["res"] >= 0) for m in s["members"]],
                        dict(tile=s["tile"], split=1, waves=s["waves"], ic_bn=16, oc_bn=16,
                             group=len(s["members"]))))
        elif s["kind"] == "conv_pool":
            # the conv's output stays in LDS; only the pooled map is written
            m = s["members"][0]
            c = dict(m["conv"], lds_out=True, pooled=(s["pool"]["OH"], s["pool"]["OW"]))
            cfg = s["config"]
            out.append((i, [(c, False)], dict(tile=cfg["tile"], waves=cfg["waves"],
                                              pooled_tile=cfg["pooled_tile"], split=1, pool=True,
                                              ic_bn=c["ic_bn"], oc_bn=c["oc_bn"])))
        elif s["kind"] in ("conv_pair", "conv_chain"):
            # every conv after the first reads its input from LDS; a chain's
            # 3x3 output stays there and is never stored
            chain = s["kind"] == "conv_chain"
            ms = [(dict(m["conv"], lds_in=j > 0, lds_out=chain and j == 0), m["res"] >= 0)
                  for j, m in enumerate(s["members"])]
            out.append((i, ms, dict(chain=True, split=1, waves=8, ic_bn=16, oc_bn=16) if chain
                        else dict(pair=True, split=1, waves=8, ic_bn=16, oc_bn=16)))
    return out


def launch_costs(members):
    """Algorithmic FLOPs and bytes of one launch (summed over its convs)."""
    f = b = 0
    for c, res in members:
        ff, bb, OH, OW = conv_costs(c["C"], c["K"], c["R"], c["S"], c["H"], c["W"], c["stride"],
                                    c["pad"], N=c["N"], residual=res)
        if c.get("gap_sums"):   # writes per-16-pixel channel sums, not its outputs
            bb += 4 * c["K"] * (-(-OH * OW // 16) - OH * OW)
        if c.get("lds_in"):     # a pointwise input read from LDS (the launch computed it)
            bb -= 4 * c["N"] * c["C"] * OH * OW
        if c.get("lds_out"):    # an output kept in LDS only
            bb -= 4 * c["N"] * c["K"] * OH * OW
        if c.get("pooled"):     # ... and its max pooling written instead
            bb += 4 * c["N"] * c["K"] * c["pooled"][0] * c["pooled"][1]
        f, b = f + ff, b + bb
    return f, b


def conv_label(c):
    OH = (c["H"] + 2 * c["pad"][0] - c["R"]) // c["stride"][0] + 1
    pool = f" + maxpool ->{c['pooled'][0]}" if c.get("pooled") else ""
    return f"{c['C']}->{c['K']} {c['R']}x{c['S']}/s{c['stride'][0]} {c['H']}->{OH}{pool}"


def plan_conv_flops(desc):
    return sum(launch_costs(m)[0] for _, m, _ in conv_launches(desc))


def time_graph(torch, fn, reps, rounds=3):
    """Average time of fn() over `reps` back-to-back launches captured in one
    graph, best of `rounds` replays, HIP events on the replay stream (us)."""
    cap = torch.cuda.Stream()
    with torch.cuda.stream(cap):
        fn()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=cap):
        for _ in range(reps):
            fn()
    graph.replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    best = 1e30
    for _ in range(rounds):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        graph.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1) * 1e3 / reps)
    del graph
    return best


_FLUSH = None


def _flush_read(torch):
    """Read a 512 MB buffer (twice the 256 MB MALL, far above the L2s) with the
    library's global average pool, which writes only 512 KB: the caches then
    hold its clean lines, so a following launch reads its operands from HBM
    and evicts nothing dirty.  (Overwriting the buffer instead leaves 256 MB
    of dirty lines whose write-back competes with the launch's reads: a plain
    231 MB copy measured 4.3 TB/s after such a write and 5.7 TB/s after the
    read.)"""
    global _FLUSH
    from paper_1809_02697_amd import neo
    if _FLUSH is None:
        _FLUSH = (torch.ones((1, 8192, 32, 32, 16), device="cuda"),
                  torch.empty((1, 8192, 1, 1, 16), device="cuda"))
    neo.global_avgpool_blocked(_FLUSH[0], 8192 * 16, out=_FLUSH[1])


def time_cold(torch, fn, reps):
    """Average time of fn() with caches cold (_flush_read before every launch):
    `reps` (flush, launch) pairs captured in one graph, minus the same number
    of flushes alone, HIP events on the replay stream (us)."""
    both = time_graph(torch, lambda: (_flush_read(torch), fn()), reps, rounds=2)
    flush = time_graph(torch, lambda: _flush_read(torch), reps, rounds=2)
    return max(both - flush, 0.0)


def cold_copy_gbs(torch, mb=256, reps=8):
    """HBM rate of a plain device-to-device copy of `mb` MB under the cold
    protocol of time_cold (bytes read + written per second): what a kernel
    with no arithmetic reaches."""
    a = torch.ones(mb * 2 ** 18, device="cuda")
    b = torch.empty_like(a)
    us = time_cold(torch, lambda: b.copy_(a), reps)
    return round(2 * mb * 2 ** 20 / (us * 1e-6) / 1e9, 1)


def e2e_ms(torch, plan, x, out, steps, warmup):
    for _ in range(warmup):
        plan.run(x, out)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        plan.run(x, out)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def stepwise_forwards(torch, plan, x, out, runs=20, head_start_cycles=5_000_000):
    """Forwards launched one step at a time, each step between two HIP events
    on the plan's stream.  Every forward is queued behind its own spin kernel
    of `head_start_cycles` (about 2 ms), so the host has enqueued the whole
    forward before the GPU starts it and the steps run back to back.  The
    events keep every dispatch from starting before its predecessor has
    ended, so in a kernel trace each dispatch's timestamps are its own
    duration inside a forward (queued back to back without them, a dispatch's
    start stamp can precede the end of the one before, and the durations
    overlap).  Returns the mean forward span in ms, event markers included."""
    stream = torch.cuda.current_stream()
    n = len(plan.describe()["steps"])
    spans = []
    for _ in range(runs):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(n)]
        torch.cuda.synchronize()
        torch.cuda._sleep(head_start_cycles)
        for i, (e0, e1) in enumerate(ev):
            e0.record(stream)
            plan.run_step(i, x, out)
            e1.record(stream)
        torch.cuda.synchronize()
        spans.append(ev[0][0].elapsed_time(ev[-1][1]))
    return float(np.mean(spans))


def e2e_stats(torch, plan, x, out, runs):
    """Per-run latency over `runs` back-to-back forwards, each bracketed by
    its own pair of HIP events (the mean +- standard error and the median,
    as the paper reports the mean of 1000 runs with its standard error)."""
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(runs)]
    torch.cuda.synchronize()
    for e0, e1 in ev:
        e0.record(stream)
        plan.run(x, out)
        e1.record(stream)
    torch.cuda.synchronize()
    t = np.array([e0.elapsed_time(e1) for e0, e1 in ev])
    return dict(runs=runs, mean_ms=round(float(t.mean()), 4),
                se_ms=round(float(t.std(ddof=1) / np.sqrt(runs)), 5),
                median_ms=round(float(np.median(t)), 4), min_ms=round(float(t.min()), 4))


def engine_clock(torch=None, plan=None, x=None, out=None, busy_runs=4000):
    """GPU engine clock as rocm-smi reports it (best effort), sampled while
    `busy_runs` forwards (about a second of work) are executing, since the
    clock drops when the GPU idles."""
    import subprocess
    if plan is not None:
        torch.cuda.synchronize()
        for _ in range(busy_runs):
            plan.run(x, out)
        time.sleep(0.2)
    try:
        r = subprocess.run(["rocm-smi", "--showclocks", "--json"], capture_output=True, text=True,
                           timeout=30)
        d = json.loads(r.stdout)
        card = d[sorted(d)[0]]
        return {k: v for k, v in card.items() if "sclk" in k.lower() or "fclk" in k.lower()
                or "mclk" in k.lower()}
    except Exception as e:  # rocm-smi missing or not parseable: report why
        return {"error": type(e).__name__}
    finally:
        if plan is not None:
            torch.cuda.synchronize()


def wino_mfma_flops(c):
    """MFMA work of a conv by Winograd F(2x2, 3x3): 16 products over the input
    channels per 2x2 output tile (2 * 16 * K * C per tile)."""
    tiles = c["N"] * -(-c["OH"] // 2) * -(-c["OW"] // 2)
    return 2 * 16 * c["K"] * c["C"] * tiles


def layer_table(torch, plan, x, out, reps, cold=True, cold_hbm_only=False, select=None):
    """Each conv step of the plan timed alone (its kernel(s) as the plan
    launches them), grouped by distinct shapes, residuals and launch
    configuration.  cold: also time every step with the caches flushed
    (cold_hbm_only: only the steps whose algorithmic intensity is below the
    ridge, the HBM-bound ones).  select(cfg): the launches to time (default
    all).  FLOPs are the direct convolution's (the metric's definition); a
    Winograd launch also reports the rate of its own MFMA work."""
    d = plan.describe()
    plan.run(x, out)      # intermediate buffers hold real activations
    torch.cuda.synchronize()
    rows = {}
    for i, members, cfg in conv_launches(d):
        if select is not None and not select(cfg):
            continue
        key = tuple((c["C"], c["K"], c["R"], c["S"], tuple(c["stride"]), tuple(c["pad"]), c["H"],
                     c["W"], c["N"], c["ic_bn"], c["oc_bn"], res) for c, res in members)
        key += (json.dumps(cfg, sort_keys=True),)
        us = time_graph(torch, lambda: plan.run_step(i, x, out), reps)
        f_, b_ = launch_costs(members)
        hbm = f_ / b_ * PEAK_HBM_GBS / 1e3 < PEAK_FP32_TFLOPS
        cold_us = (time_cold(torch, lambda: plan.run_step(i, x, out), max(4, reps // 2))
                   if cold and (hbm or not cold_hbm_only) else 0.0)
        if key in rows:
            rows[key]["uses"] += 1
            rows[key]["_t"].append(us)
            rows[key]["_c"].append(cold_us)
            continue
        flops, nbytes = launch_costs(members)
        rows[key] = dict(shape=" + ".join(conv_label(c) + (" +res" if res else "") for c, res in members),
                         uses=1, flops=flops,
                         bytes=nbytes, config=cfg, _t=[us], _c=[cold_us],
                         _wflops=sum(wino_mfma_flops(c) for c, _ in members))
    out_rows = []
    for r in rows.values():
        us = float(np.mean(r.pop("_t")))
        cold_us = float(np.mean(r.pop("_c")))
        tf = r["flops"] / (us * 1e-6) / 1e12
        gbs = r["bytes"] / (us * 1e-6) / 1e9
        ai = r["flops"] / r["bytes"]
        roof = min(PEAK_FP32_TFLOPS, ai * PEAK_HBM_GBS / 1e3)
        r.update(us=round(us, 2), gflop=round(r["flops"] / 1e9, 4), tflops=round(tf, 2),
                 alg_gbs=round(gbs, 1),
                 bound="mfma" if ai * PEAK_HBM_GBS / 1e3 >= PEAK_FP32_TFLOPS else "hbm",
                 pct_mfma=round(100 * tf / PEAK_FP32_TFLOPS, 1),
                 pct_hbm=round(100 * gbs / PEAK_HBM_GBS, 1), pct_roof=round(100 * tf / roof, 1))
        if cold and cold_us > 0:
            r.update(cold_us=round(cold_us, 2),
                     cold_hbm_gbs=round(r["bytes"] / (cold_us * 1e-6) / 1e9, 1))
        if r["config"].get("algo") == "winograd":
            wtf = r.pop("_wflops") / (us * 1e-6) / 1e12
            r.update(wino_mfma_tflops=round(wtf, 2), wino_pct_mfma=round(100 * wtf / PEAK_FP32_TFLOPS, 1))
        else:
            r.pop("_wflops", None)
        out_rows.append(r)
    return out_rows


PEAK_INT8_TOPS = 5000.0     # MI355X dense int8 matrix peak (5.0 POP/s)
# ResNet-50 layers whose output a 3x3 conv reads (its padding 1 becomes the
# int8 output's halo); every other output feeds a 1x1
INT8_NEXT_PAD = {"R02": 1, "R05": 1, "R06": 1, "R10": 1, "R12": 1, "R16": 1, "R18": 1, "R22": 1}


def int8_layer(neo, torch, wl, i, N):
    """ResNet-50 conv shape i at batch N set up for the integer path: seeded
    float32 input in NCHW16c, its quantization (with the conv's halo), the
    packed int8 filter and scales, zero bias, a residual where the layer has
    one.  Returns the shape's figures and the conv and quantize launches."""
    lid, C, K, R, st, pd, H, epi, uses = wl.RESNET50_LAYERS[i]
    rng = np.random.default_rng([11, i])
    OH = (H + 2 * pd - R) // st + 1
    KB = -(-K // 16)
    x = torch.from_numpy(rng.uniform(-1, 1, (N, C, H, H)).astype(np.float32)).cuda()
    w = torch.from_numpy(rng.normal(0, np.sqrt(2 / (C * R * R)), (K, C, R, R)).astype(np.float32)).cuda()
    xb = neo.to_blocked(x)
    del x
    xs = float(xb.abs().max().item() / 127)
    xq = neo.quantize_int8(xb, C, xs, pad=pd)
    wq, ws = neo.pack_filter_int8(w)
    bias = torch.zeros(KB * 16, device="cuda")
    res = torch.zeros((N, KB, OH, OH, 16), device="cuda") if epi == "res" else None
    out = torch.empty((N, KB, OH, OH, 16), device="cuda")
    act = "relu" if epi in ("relu", "res") else "none"

    def conv():
        neo.conv2d_int8(xq, C, wq, ws, K, R, R, xs, bias=bias, stride=st, pad=pd, act=act,
                        residual=res, out=out)

    def quant():
        neo.quantize_int8(xb, C, xs, pad=pd, out=xq)
    # int8 output for the next layer: its halo is the padding of the conv that
    # reads it in ResNet-50 (1 before a 3x3, 0 before a 1x1); output scale of
    # the order of the float output's (its value does not change the time)
    qpad = INT8_NEXT_PAD.get(lid, 0)
    yq = torch.zeros((N, KB, OH + 2 * qpad, OH + 2 * qpad, 16), device="cuda", dtype=torch.int8)

    def conv_q():
        neo.conv2d_int8_q(xq, C, wq, ws, K, R, R, xs, 0.05, bias=bias, stride=st, pad=pd, act=act,
                          residual=res, out_pad=qpad, out=yq)
    ops = 2 * N * K * C * R * R * OH * OH
    rbytes = 4 * N * K * OH * OH if res is not None else 0
    nbytes = N * C * H * H + K * C * R * R + 4 * N * K * OH * OH + rbytes + 8 * K
    nbytes_q = N * C * H * H + K * C * R * R + N * K * OH * OH + rbytes + 8 * K
    label = f"{C}->{K} {R}x{R}/s{st} {H}->{OH}" + (" +res" if res is not None else "")
    return dict(id=lid, shape=label, uses=uses, ops=ops, bytes=nbytes, bytes_q=nbytes_q, conv=conv,
                quant=quant, conv_q=conv_q)


def int8_layer_table(neo, torch, wl, N=32, reps=10, fp32_us=None):
    """The 23 distinct ResNet-50 conv shapes at batch N through the integer
    path (quantized activations with their halo, packed int8 filter, int32
    MFMA accumulation, float32 epilogue with the layer's residual and ReLU),
    each timed alone like layer_table (warm, back-to-back graph replays),
    beside the activation quantization pass the layer needs and, from
    fp32_us ({shape label: us} of the tuned fp32 plan), the fp32 conv of the
    same shape; int8_out_*: the same conv writing its output requantized to
    int8 (the next layer's input, no quantization pass between int8 layers).
    Ops are the direct convolution's; bytes are algorithmic: int8 input and
    filter, float32 (or int8) output, float32 residual."""
    rows = []
    for i in range(len(wl.RESNET50_LAYERS)):
        L = int8_layer(neo, torch, wl, i, N)
        us = time_graph(torch, L["conv"], reps)
        q_us = time_graph(torch, L["quant"], reps)
        us_q = time_graph(torch, L["conv_q"], reps)
        ops, nbytes = L["ops"], L["bytes"]
        ai = ops / nbytes
        roof = min(PEAK_INT8_TOPS, ai * PEAK_HBM_GBS / 1e3)
        tops = ops / (us * 1e-6) / 1e12
        f32 = (fp32_us or {}).get(L["shape"])
        rows.append(dict(id=L["id"], shape=L["shape"], uses=L["uses"],
                         us=round(us, 2), quant_us=round(q_us, 2), tops=round(tops, 1),
                         pct_int8_mfma=round(100 * tops / PEAK_INT8_TOPS, 1),
                         alg_gbs=round(nbytes / (us * 1e-6) / 1e9, 1),
                         bound="mfma" if ai * PEAK_HBM_GBS / 1e3 >= PEAK_INT8_TOPS else "hbm",
                         pct_roof=round(100 * tops / roof, 1),
                         fp32_us=f32, speedup_vs_fp32=round(f32 / us, 2) if f32 else None,
                         int8_out_us=round(us_q, 2),
                         int8_out_tops=round(ops / (us_q * 1e-6) / 1e12, 1),
                         int8_out_alg_gbs=round(L["bytes_q"] / (us_q * 1e-6) / 1e9, 1),
                         _ops=ops))
        del L
    t = sum(r["us"] * r["uses"] for r in rows)
    tq = sum((r["us"] + r["quant_us"]) * r["uses"] for r in rows)
    ops = sum(r.pop("_ops") * r["uses"] for r in rows)
    tqo = sum(r["int8_out_us"] * r["uses"] for r in rows)
    summary = dict(batch=N, convs=sum(r["uses"] for r in rows), sum_us=round(t, 1),
                   sum_with_quant_us=round(tq, 1), tops=round(ops / (t * 1e-6) / 1e12, 1),
                   pct_int8_mfma=round(100 * ops / (t * 1e-6) / 1e12 / PEAK_INT8_TOPS, 2),
                   int8_out_sum_us=round(tqo, 1),
                   int8_out_tops=round(ops / (tqo * 1e-6) / 1e12, 1))
    m = [r for r in rows if r["fp32_us"]]
    if m:
        # over the shapes the fp32 plan launches alone (the stem runs fused
        # with its max pool there)
        t32 = sum(r["fp32_us"] * r["uses"] for r in m)
        t8 = sum(r["us"] * r["uses"] for r in m)
        t8q = sum((r["us"] + r["quant_us"]) * r["uses"] for r in m)
        t8o = sum(r["int8_out_us"] * r["uses"] for r in m)
        summary.update(fp32_matched_convs=sum(r["uses"] for r in m), fp32_sum_us=round(t32, 1),
                       int8_matched_sum_us=round(t8, 1), speedup_vs_fp32=round(t32 / t8, 2),
                       speedup_with_quant=round(t32 / t8q, 2),
                       int8_out_speedup_vs_fp32=round(t32 / t8o, 2))
    return rows, summary


def scheme_summary(d):
    """Histogram of the convs' (ic_bn, oc_bn) in a plan description."""
    h = {}
    for ic, oc in plan_schemes(d).values():
        h[f"{ic}/{oc}"] = h.get(f"{ic}/{oc}", 0) + 1
    return dict(sorted(h.items()))


def model_latencies(neo, torch, wl, steps):
    """End-to-end latency of each model (tuned, graph replay) for the three
    plans of the Table 3 ablation; ResNet-50 also at fixed blocks 32 and 64;
    and with the 3x3 stride-1 convs free to run by Winograd F(2x2, 3x3) (the
    paper's future work; the local search keeps it per conv where faster),
    with and without the fusions; and integer inference (NEO_PLAN_INT8, its
    speedup over the fastest float32 plan of the entry)."""
    res = {}
    for name, builder, batch in [("resnet50", wl.resnet50, 1), ("vgg16", wl.vgg16, 1),
                                 ("inception_v3", wl.inception_v3, 1), ("resnet50", wl.resnet50, 32),
                                 ("vgg16", wl.vgg16, 32)]:
        g = builder(batch)
        x = torch.from_numpy(g.x).cuda()
        entry = {}
        fused = (neo.PLAN_GROUP | neo.PLAN_FUSE_GAP | neo.PLAN_FUSE_PAIRS | neo.PLAN_FUSE_CHAINS |
                 neo.PLAN_FUSE_POOL)
        plans = [("eliminated", 0, 16), ("grouped", fused, 16), ("winograd", neo.PLAN_WINOGRAD, 16),
                 ("winograd_grouped", fused | neo.PLAN_WINOGRAD, 16)]
        if batch == 1:   # (the batch-32 search measures ~190 schemes at ~0.6 s each)
            plans += [("searched", neo.PLAN_GLOBAL_SEARCH, 16), ("naive", neo.PLAN_NAIVE, 16)]
        if name == "resnet50":
            plans += [("eliminated_x32", 0, 32), ("eliminated_x64", 0, 64)]
        if name == "vgg16" and batch == 32:   # (nothing to fuse in a chain of convs)
            plans = [("eliminated", 0, 16), ("winograd", neo.PLAN_WINOGRAD, 16)]
        for label, flags, block in plans:
            t0 = time.perf_counter()
            p = neo.Plan(g, flags=flags | neo.PLAN_TUNE | neo.PLAN_HIPGRAPH, block=block)
            t_plan = time.perf_counter() - t0
            out = p.run(x)
            ms = e2e_ms(torch, p, x, out, steps, 3)
            d = p.describe()
            entry[label] = dict(ms=round(ms, 4), n_transforms=d["n_transforms"],
                                launches=len(d["steps"]), plan_s=round(t_plan, 1))
            if flags & neo.PLAN_WINOGRAD:
                entry[label]["winograd_convs"] = sum(
                    1 for st in d["steps"] if st["kind"] == "conv" and st["conv"]["algo"] == "winograd")
            if label == "searched":
                entry[label]["schemes"] = scheme_summary(d)
                entry[label]["predicted_us"] = round(d["search"]["cost_us"], 1)
                entry[label]["predicted_fixed16_us"] = round(d["search"]["fixed_block_cost_us"], 1)
                entry[label]["schemes_measured"] = d["search"]["schemes_measured"]
            if label == ("searched" if batch == 1 else "eliminated"):
                flops = plan_conv_flops(d)
                entry["conv_tflops"] = round(flops / (ms * 1e-3) / 1e12, 2)
                entry["images_per_s"] = round(batch / (ms * 1e-3), 1)
            p.destroy()
        # integer inference (every conv int8; tuned; calibrated on this input,
        # untimed), graph replay; alone and with independent convs grouped
        # into launches (the int8 entry is the faster)
        int8_runs = {}
        for label, extra in (("int8_plain", 0), ("int8_grouped", neo.PLAN_GROUP)):
            t0 = time.perf_counter()
            p = neo.Plan(g, flags=neo.PLAN_INT8 | neo.PLAN_TUNE | neo.PLAN_HIPGRAPH | extra)
            out = p.calibrate_int8(x)
            t_plan = time.perf_counter() - t0
            ms = e2e_ms(torch, p, x, out, steps, 3)
            d = p.describe()
            q = [c["int8"] for st in d["steps"]
                 for c in ([st["conv"]] if st["kind"] == "conv" else
                           [m["conv"] for m in st.get("members", [])] if st["kind"] == "conv_group" else
                           [st["dense"]] if st["kind"] == "dense" and "int8" in st["dense"] else [])]
            passes = sum(c["quantizes_input"] for c in q)
            int8_runs[label] = dict(ms=round(ms, 4), launches=len(d["steps"]) + passes,
                                    quantization_passes=passes, plan_s=round(t_plan, 1),
                                    groups=sum(st["kind"] == "conv_group" for st in d["steps"]))
            p.destroy()
        best8 = min(int8_runs, key=lambda k: int8_runs[k]["ms"])
        fp32_best = min(v["ms"] for v in entry.values() if isinstance(v, dict))
        entry["int8"] = dict(int8_runs[best8], plan=best8)
        entry.update(int8_runs)
        entry["int8_speedup"] = round(fp32_best / entry["int8"]["ms"], 3)
        if "naive" in entry:
            entry["elimination_speedup"] = round(entry["naive"]["ms"] / entry["eliminated"]["ms"], 3)
        if "searched" in entry:
            entry["search_speedup"] = round(entry["eliminated"]["ms"] / entry["searched"]["ms"], 3)
        if "grouped" in entry:
            entry["group_speedup"] = round(entry["eliminated"]["ms"] / entry["grouped"]["ms"], 3)
        direct = min(entry[k]["ms"] for k in ("eliminated", "grouped") if k in entry)
        wino = min(entry[k]["ms"] for k in ("winograd", "winograd_grouped") if k in entry)
        entry["winograd_speedup"] = round(direct / wino, 3)
        res[f"{name}_b{batch}"] = entry
        del g, x
        print(f"[bench] {name} b{batch}: {entry}", file=sys.stderr, flush=True)
    return res


def measured_traffic():
    """HBM/fabric bytes per conv launch from the committed counter summary,
    or None when the kernel source changed since the counters were taken."""
    from paper_1809_02697_amd.profile_summary import kernel_hash
    path = os.path.join(ROOT, "profiles", "conv2d_blocked_resnet50_b1_traffic.json")
    try:
        t = json.load(open(path))
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256") != kernel_hash():
        return None
    return t["traffic_bytes_per_launch"]


def cpu_model():
    """The host CPU's model string (/proc/cpuinfo) and its logical CPU count."""
    try:
        with open("/proc/cpuinfo") as f:
            names = [l.split(":", 1)[1].strip() for l in f if l.startswith("model name")]
        return (names[0] if names else "unknown"), len(names)
    except OSError:
        return "unknown", 0


def _timed(fn, budget_s, min_runs=1):
    """(seconds per call, calls): fn() repeated until budget_s has passed."""
    n, t0 = 0, time.perf_counter()
    while n < min_runs or time.perf_counter() - t0 < budget_s:
        fn()
        n += 1
    return (time.perf_counter() - t0) / n, n


def cpu_baseline(g, budget_s=8.0):
    """The oracle (plain C direct convolution in double, OpenMP over the host
    cores; batch norm, bias, residual and ReLU unfused in numpy) on the same
    workloads as the GPU, on a bounded sample:
      value      whole ResNet-50 batch-1 forwards until ~budget_s of work;
      e2e_ms     one forward each of the single conv (configuration 1), VGG-16
                 and Inception-v3 at batch 1;
      layers_ms  each of the 23 ResNet-50 layer shapes once (conv + batch norm +
                 residual + ReLU);
      single_core  the single conv on one thread."""
    import oracle
    from paper_1809_02697_amd import workloads as wl
    flops = 8_174_272_512
    model, ncpu = cpu_model()
    cores = oracle.num_threads()
    dt, n = _timed(lambda: oracle.run_graph(g), budget_s)
    out = dict(value=round(flops / dt / 1e12, 6), unit="TFLOP/s", cores=cores,
               kind="oracle", cpu_model=model, host_logical_cpus=ncpu,
               ms_per_forward=round(dt * 1e3, 1),
               sample=f"{n} ResNet-50 batch-1 forward pass(es) through the oracle graph executor "
                      f"({dt * n:.1f} s); plus one forward each of configuration 1, VGG-16 and "
                      f"Inception-v3, the 23 layer shapes once, and configuration 1 on one thread")
    cfg1 = wl.single_conv(0)
    e2e = {}
    for name, gg, gf in [("single_conv", cfg1, 231_211_008), ("vgg16_b1", wl.vgg16(1), 30_693_261_312),
                         ("inception_v3_b1", wl.inception_v3(1), 11_422_336_192)]:
        t, _ = _timed(lambda: oracle.run_graph(gg), 0.0)
        e2e[name] = dict(ms=round(t * 1e3, 1), conv_gflops=round(gf / t / 1e9, 2))
    out["e2e_ms"] = e2e
    layers = {}
    for c in wl.resnet50_layer_sweep(1):
        t, _ = _timed(lambda: oracle.layer_forward(c), 0.0)
        f = 2 * c.N * c.K * c.C * c.R * c.S * ((c.H + 2 * c.pad[0] - c.R) // c.stride[0] + 1) * \
            ((c.W + 2 * c.pad[1] - c.S) // c.stride[1] + 1)
        layers[c.id] = dict(ms=round(t * 1e3, 2), gflops=round(f / t / 1e9, 2))
    out["layers_ms"] = layers
    oracle.set_num_threads(1)
    try:
        t, _ = _timed(lambda: oracle.run_graph(cfg1), 0.0)
    finally:
        oracle.set_num_threads(cores)
    out["single_core"] = dict(workload="configuration 1 (64->64 3x3, 56x56, bias + ReLU)",
                              cores=1, ms=round(t * 1e3, 1), gflops=round(231_211_008 / t / 1e9, 3))
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--layer-reps", type=int, default=20)
    ap.add_argument("--stepwise-runs", type=int, default=20,
                    help="forwards launched step by step between events (for kernel traces)")
    ap.add_argument("--latency-runs", type=int, default=1000,
                    help="single-forward latency samples (mean, standard error, median)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-clock", action="store_true",
                    help="skip the engine-clock sample (4000 forwards under load)")
    ap.add_argument("--no-layers", action="store_true", help="skip the per-layer table")
    ap.add_argument("--no-models", action="store_true", help="skip the other models and ablation")
    ap.add_argument("--tune-db", help="load this local-search results file before planning")
    ap.add_argument("--save-tune-db", help="write the local-search results here at the end")
    ap.add_argument("--int8-only", action="store_true",
                    help="only the batch-32 integer conv table (no fp32 comparison); one JSON line")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the batch-1 path has no cross-GPU work "
              "(see the sharding note of the design); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_1809_02697_amd import neo
    from paper_1809_02697_amd import workloads as wl
    neo.lib()
    assert torch.cuda.is_available(), "no GPU"
    if args.int8_only:
        rows, summary = int8_layer_table(neo, torch, wl, 32, args.layer_reps, None)
        print(json.dumps({"layers_b32_int8": rows, "int8_b32": summary}))
        return

    if args.tune_db:
        neo.tune_db_load(args.tune_db)
    g = wl.resnet50(1)
    t0 = time.perf_counter()
    plan, plan_info = headline_plan(neo, g, args.tune_db, torch, args.steps, args.warmup)
    t_plan = time.perf_counter() - t0
    x = torch.from_numpy(g.x).cuda()
    out = torch.empty((1, 1000), device="cuda")
    desc = plan.describe()
    conv_flops = plan_conv_flops(desc)
    print(f"[bench] plan built and tuned in {t_plan:.1f} s: {len(desc['steps'])} steps",
          file=sys.stderr, flush=True)

    # the single-forward latencies first: the timed steps then start with the
    # GPU at its working clock (after ~20 ms idle, the first ~30 forwards run
    # up to 10 % slower)
    stats = e2e_stats(torch, plan, x, out, args.latency_runs)
    print(f"[bench] latency over {stats['runs']} runs: {stats}", file=sys.stderr, flush=True)
    ms = e2e_ms(torch, plan, x, out, args.steps, args.warmup)
    print(f"[bench] e2e {ms:.3f} ms/step", file=sys.stderr, flush=True)
    clock = None if args.no_clock else engine_clock(torch, plan, x, out)
    print(f"[bench] engine clock under load: {clock}", file=sys.stderr, flush=True)

    stepwise_ms = stepwise_forwards(torch, plan, x, out, args.stepwise_runs)
    print(f"[bench] forward launched step by step between events: {stepwise_ms:.4f} ms",
          file=sys.stderr, flush=True)

    layers, roofline = None, None
    if not args.no_layers:
        layers = layer_table(torch, plan, x, out, args.layer_reps)
        tot_f = sum(r["flops"] * r["uses"] for r in layers)
        tot_t = sum(r["us"] * 1e-6 * r["uses"] for r in layers)
        n_launch = sum(r["uses"] for r in layers)
        achieved = tot_f / tot_t / 1e12
        roofline = dict(bound="mfma", achieved=round(achieved, 2), peak=PEAK_FP32_TFLOPS,
                        unit="TFLOP/s", frac=round(achieved / PEAK_FP32_TFLOPS, 4),
                        traffic=measured_traffic(),
                        kernel="conv2d_blocked (single, fused-group, pointwise-pair and 3x3-chain "
                               "launches, each with its split-reduction pass)",
                        timing=f"HIP events around {args.layer_reps} back-to-back graph replays "
                               f"of each conv step of the plan, on the plan's stream",
                        launches_per_step=n_launch,
                        avg_launch_us=round(tot_t / n_launch * 1e6, 3),
                        sum_conv_us=round(tot_t * 1e6, 1),
                        flop_per_launch=round(tot_f / n_launch))
        for r in layers:
            del r["flops"], r["bytes"]
        print(f"[bench] conv layers: {achieved:.2f} TFLOP/s over {n_launch} launches, "
              f"{tot_t * 1e6:.1f} us per forward", file=sys.stderr, flush=True)

    models = None if args.no_models else model_latencies(neo, torch, wl, 20)

    layers_b32 = layers_b32_winograd = layers_b32_int8 = int8_b32 = None
    if not args.no_layers and not args.no_models:
        # the same kernels with the per-launch floor amortized over 32 images
        g32 = wl.resnet50(32)
        p32 = neo.Plan(g32, flags=neo.PLAN_TUNE | neo.PLAN_HIPGRAPH)
        x32 = torch.from_numpy(g32.x).cuda()
        o32 = p32.run(x32)
        layers_b32 = layer_table(torch, p32, x32, o32, 10, cold_hbm_only=True)
        fp32_b32 = {r["shape"]: r["us"] for r in layers_b32 if "+ maxpool" not in r["shape"]}
        tf32 = sum(r["flops"] * r["uses"] for r in layers_b32) / \
            sum(r["us"] * 1e-6 * r["uses"] for r in layers_b32) / 1e12
        for r in layers_b32:
            del r["flops"], r["bytes"]
        p32.destroy()
        # the 3x3 stride-1 layers again where the local search keeps Winograd
        p32w = neo.Plan(g32, flags=neo.PLAN_TUNE | neo.PLAN_HIPGRAPH | neo.PLAN_WINOGRAD)
        layers_b32_winograd = layer_table(torch, p32w, x32, o32, 10, cold=False,
                                          select=lambda cfg: cfg.get("algo") == "winograd")
        for r in layers_b32_winograd:
            del r["flops"], r["bytes"]
        p32w.destroy()
        del g32, x32, o32
        torch.cuda.empty_cache()
        # the same shapes through the integer path
        layers_b32_int8, int8_b32 = int8_layer_table(neo, torch, wl, 32, 10, fp32_b32)
        print(f"[bench] batch-32 int8 conv layers: {int8_b32}", file=sys.stderr, flush=True)
        print(f"[bench] batch-32 conv layers: {tf32:.2f} TFLOP/s", file=sys.stderr, flush=True)
    copy_gbs = None if args.no_layers else cold_copy_gbs(torch)

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
        "stepwise_forward_ms": round(stepwise_ms, 4),
        "latency": stats,
        "engine_clock": clock,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp32",
        "data": "synthetic",
        "config": {"workload": "ResNet-50 forward, batch 1, 3x224x224 fp32, NCHW[x]c plan (the "
                               "faster of the globally searched and the all-NCHW16c plan), "
                               "tuned, the faster of one hipGraph replay and step-by-step stream "
                               "launches, seed 2",
                   "global_batch": 1, "conv_gflop_per_step": round(conv_flops / 1e9, 4),
                   "cache": "warm (working set resident in the 256 MB MALL)",
                   "plan_build_s": round(t_plan, 2), "schemes": scheme_summary(desc),
                   "n_transforms": desc["n_transforms"], "plan_choice": plan_info},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "layers": layers,
        "layers_b32": layers_b32,
        "layers_b32_winograd": layers_b32_winograd,
        "layers_b32_int8": layers_b32_int8,
        "int8_b32": int8_b32,
        "cold_copy_gbs": copy_gbs,
        "models": models,
    }
    print(json.dumps(rec))
    plan.destroy()
    if args.save_tune_db:
        neo.tune_db_save(args.save_tune_db)
        with open(args.save_tune_db + ".schemes.json", "w") as f:
            json.dump({"schemes": {str(k): list(v) for k, v in plan_schemes(desc).items()},
                       "launch": plan_info["launch"]}, f)
        with open(args.save_tune_db + ".plan.json", "w") as f:
            json.dump(desc, f)


if __name__ == "__main__":
    main()
