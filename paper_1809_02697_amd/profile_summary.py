"""Summarize rocprofv3 output of the ResNet-50 conv kernels into profiles/.

    python -m paper_1809_02697_amd.profile_summary RUN_DIR

RUN_DIR holds (names as written by the commands in COMMANDS below):
  bench.log       the JSON line of a plain ``python bench.py --save-tune-db
                  RUN_DIR/tune_db.txt`` run (and the results file it saved)
  prof_bench/     rocprofv3 --kernel-trace --stats of the same bench command
                  (profiled, with the saved results file, so the plan is the
                  one the plain run timed)
  pmc/            counter passes over profile_layers: FETCH_SIZE and WRITE_SIZE
                  with warm caches and with every step cold (--cold), and the
                  MFMA counters at batch 1 and batch 32

Writes
  profiles/conv2d_blocked_resnet50_b1.md  launch durations, per-layer traffic
      (warm and cold) and MFMA utilisation at batch 1
  profiles/conv2d_blocked_resnet50_b32_mfma.md  MFMA utilisation at batch 32
  profiles/wino_f2x3_resnet50_b32.md  the Winograd kernel's launches in the
      batch-32 plan with NEO_PLAN_WINOGRAD: durations and MFMA utilisation
  profiles/conv_i8_resnet50_b32.md  the integer conv of each ResNet-50 shape at
      batch 32 (INT8_COMMANDS): durations, traffic, MFMA utilisation
  profiles/conv2d_blocked_resnet50_b1_traffic.json  bytes per launch, tied to
      the hash of the kernel source it was measured with (bench.py reports it
      only while the source is unchanged)

Launch durations.  The kernel trace's timestamps of the forwards that bench.py
launches step by step between events (stepwise_forwards: the dispatches after
its spin kernel) are each launch's own duration inside a forward; their mean
is compared with bench.py's HIP-event figure.  Under the profiler, graph
replays are slower and their per-dispatch durations longer, and dispatches
queued back to back overlap in the trace (a start stamp precedes the end of
the dispatch before); both are reported, neither is used.

FETCH_SIZE / WRITE_SIZE are KiB moved between L2 and the fabric per dispatch,
calibrated by the same counters on a plain copy of COPY_MB megabytes (which
reads and writes exactly that many bytes).  Warm, the figures include reads
served by the 256 MB MALL; cold (512 MB written before every step), the reads
come from HBM.  MFMA utilisation is SQ_VALU_MFMA_BUSY_CYCLES summed over the
SIMDs / (GRBM_GUI_ACTIVE x 1024 SIMDs), rocprofv3's MfmaUtil, per dispatch.
"""
import csv
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SRCS = [os.path.join(HERE, "csrc", f)
               for f in ("conv_kernel.h", "conv.hip", "conv_xy.hip", "conv_group.hip", "conv_pair.hip",
                         "conv_pool.hip", "conv_stream.hip")]
PEAK = 157.3
SIMDS = 1024         # 256 CUs x 4
CLOCK_MHZ = 2400.0   # engine clock under load (bench.py's engine_clock)

COMMANDS = [
    "python bench.py --save-tune-db RUN_DIR/tune_db.txt > RUN_DIR/bench.log",
    "rocprofv3 --kernel-trace --stats --output-format csv -d RUN_DIR/prof_bench -o bench -- "
    "python bench.py --no-cpu --no-models --no-clock --tune-db RUN_DIR/tune_db.txt "
    "--latency-runs 100",
    "rocprofv3 --pmc FETCH_SIZE --output-format csv -d RUN_DIR/pmc -o fetch -- "
    "python -m paper_1809_02697_amd.profile_layers RUN_DIR/tune_db.txt",
    "rocprofv3 --pmc WRITE_SIZE --output-format csv -d RUN_DIR/pmc -o write -- "
    "python -m paper_1809_02697_amd.profile_layers RUN_DIR/tune_db.txt",
    "rocprofv3 --pmc FETCH_SIZE --output-format csv -d RUN_DIR/pmc -o fetch_cold -- "
    "python -m paper_1809_02697_amd.profile_layers RUN_DIR/tune_db.txt --cold",
    "rocprofv3 --pmc WRITE_SIZE --output-format csv -d RUN_DIR/pmc -o write_cold -- "
    "python -m paper_1809_02697_amd.profile_layers RUN_DIR/tune_db.txt --cold",
    "rocprofv3 --pmc MfmaUtil SQ_INSTS_VALU_MFMA_MOPS_F32 SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE "
    "--output-format csv -d RUN_DIR/pmc -o mfma -- "
    "python -m paper_1809_02697_amd.profile_layers RUN_DIR/tune_db.txt",
    "rocprofv3 --pmc MfmaUtil SQ_INSTS_VALU_MFMA_MOPS_F32 SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE "
    "--output-format csv -d RUN_DIR/pmc -o mfma32 -- python -m paper_1809_02697_amd.profile_layers RUN_DIR/tune_db.txt --batch 32 "
    "--describe RUN_DIR/plan_b32.json",
    "rocprofv3 --pmc MfmaUtil SQ_INSTS_VALU_MFMA_MOPS_F32 SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE "
    "--output-format csv -d RUN_DIR/pmc -o mfma32w -- python -m paper_1809_02697_amd.profile_layers "
    "RUN_DIR/tune_db.txt --batch 32 --winograd --describe RUN_DIR/plan_b32w.json",
    "rocprofv3 --kernel-trace --stats --output-format csv -d RUN_DIR/prof_wino -o wino -- "
    "python -m paper_1809_02697_amd.profile_layers RUN_DIR/tune_db.txt --batch 32 --winograd --reps 20",
    "python -m paper_1809_02697_amd.profile_summary RUN_DIR",
]
# the integer convs (no plan, no results file), summarized by write_int8
INT8_COMMANDS = [
    "rocprofv3 --kernel-trace --stats --output-format csv -d RUN_DIR/prof_i8 -o i8 -- "
    "python -m paper_1809_02697_amd.profile_layers --int8 --batch 32 --reps 20",
    "rocprofv3 --pmc FETCH_SIZE --output-format csv -d RUN_DIR/pmc -o i8fetch -- "
    "python -m paper_1809_02697_amd.profile_layers --int8 --batch 32",
    "rocprofv3 --pmc WRITE_SIZE --output-format csv -d RUN_DIR/pmc -o i8write -- "
    "python -m paper_1809_02697_amd.profile_layers --int8 --batch 32",
    "rocprofv3 --pmc SQ_INSTS_VALU_MFMA_MOPS_I8 SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE "
    "--output-format csv -d RUN_DIR/pmc -o i8mfma -- "
    "python -m paper_1809_02697_amd.profile_layers --int8 --batch 32",
    "python -m paper_1809_02697_amd.profile_summary RUN_DIR",
]

# whole integer networks at batch 1 (the bench line's int8_grouped plans),
# summarized by write_int8_plans
INT8_PLAN_MODELS = ("resnet50", "inception_v3", "vgg16")
INT8_PLAN_REPS = 20
INT8_PLAN_COMMANDS = [
    f"rocprofv3 --kernel-trace --stats --output-format csv -d RUN_DIR/prof_i8plan -o {m} -- "
    f"python -m paper_1809_02697_amd.profile_layers --int8-plan {m} --batch 1 --reps {INT8_PLAN_REPS}"
    for m in INT8_PLAN_MODELS] + ["python -m paper_1809_02697_amd.profile_summary RUN_DIR"]
# kernel name -> the part of an integer forward it does (first match)
INT8_PLAN_KINDS = [("conv_i8_group", "int8 conv group launches"), ("conv_i8", "int8 convs alone"),
                   ("quantize_kernel", "quantization passes"),
                   ("im2col_q", "quantization passes (im2col rows of the stem)"),
                   ("pool_blk_q", "pools writing an int8 copy"),
                   ("pool_blk", "float32 pools"), ("gap_blk", "global average pool"),
                   ("dense_", "dense layers"), ("_to_", "layout transforms")]


def kernel_hash():
    """sha256[:16] of the conv kernel's sources (templates and instantiations)."""
    h = hashlib.sha256()
    for f in KERNEL_SRCS:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def _rows(path):
    with open(path) as f:
        return list(csv.DictReader(f))


def is_conv_i8(name):
    return "conv_i8" in name


def is_conv(name):
    return ("conv2d_mfma" in name or "conv1x1_pair" in name or "conv3x3_chain" in name or
            "conv_pool_small" in name or "conv1x1_stream" in name or "wino_f2x3" in name)


def is_neo(name):
    return "neo::" in name


def _dispatch_values(path, counter=None):
    """{dispatch id: (kernel name, value)} of a counter file, in dispatch order;
    `counter` picks one counter of a multi-counter pass."""
    out = {}
    for r in _rows(path):
        if counter and r["Counter_Name"] != counter:
            continue
        d = int(r["Dispatch_Id"])
        name, v = out.get(d, (r["Kernel_Name"], 0.0))
        out[d] = (name, v + float(r["Counter_Value"]))
    return [out[d] for d in sorted(out)]


def forward_dispatches(path, counter=None):
    """Counter values of the dispatches after the last copy kernel (one forward
    pass, in launch order, the cold pass's flushes dropped) and of that copy."""
    rows = _dispatch_values(path, counter)
    last_copy = max(i for i, (n, _) in enumerate(rows) if "copyBuffer" in n)
    fwd = [(n, v) for n, v in rows[last_copy + 1:] if is_neo(n)]
    return rows[last_copy][1], fwd


def per_conv(fwd):
    """Group dispatches into conv launches: a conv dispatch (single, fused
    group, pair or chain) and the split_reduce dispatch that may follow it."""
    out = []
    for name, v in fwd:
        if is_conv(name):
            out.append(v)
        elif "split_reduce" in name and out:
            out[-1] += v
    return out


def per_conv_max(fwd):
    """Like per_conv for a ratio counter: the conv dispatch's own value."""
    return [v for name, v in fwd if is_conv(name)]


def stepwise_forward_durations(trace_path, n_steps):
    """Per-launch durations (us) of the conv launches of every forward bench.py
    launched step by step between events, each behind its own spin kernel: a
    list of forwards, each a list of conv launch durations (a split_reduce pass
    added to its conv)."""
    rows = sorted(_rows(trace_path), key=lambda r: int(r["Start_Timestamp"]))
    dur = lambda r: (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    out = []
    spins = [i for i, r in enumerate(rows) if "spin_kernel" in r["Kernel_Name"]]
    for sp in spins:
        cur, steps = [], 0
        for r in rows[sp + 1:]:
            n = r["Kernel_Name"]
            if not is_neo(n):
                break
            if is_conv(n):
                cur.append(dur(r))
            elif "split_reduce" in n and cur:
                cur[-1] += dur(r)
            if "split_reduce" not in n:
                steps += 1
            if steps == n_steps:
                out.append(cur)
                break
    return out


def graph_forward_durations(trace_path, n_steps):
    """Sum of conv durations per back-to-back forward before the spin kernel
    (the profiled e2e and latency runs), and the forward spans.  A forward
    starts at a dispatch of the kernel that starts the step-by-step ones."""
    rows = sorted(_rows(trace_path), key=lambda r: int(r["Start_Timestamp"]))
    spin = min(i for i, r in enumerate(rows) if "spin_kernel" in r["Kernel_Name"])
    first = next(r["Kernel_Name"] for r in rows[spin + 1:] if is_neo(r["Kernel_Name"]))
    starts = [i for i in range(spin) if rows[i]["Kernel_Name"] == first]
    sums, spans = [], []
    for a, b in zip(starts, starts[1:]):
        blk = [r for r in rows[a:b] if is_neo(r["Kernel_Name"])]
        if len([r for r in blk if "split_reduce" not in r["Kernel_Name"]]) != n_steps:
            continue
        d = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in blk]
        sums.append(sum(x for r, x in zip(blk, d) if is_conv(r["Kernel_Name"])
                        or "split_reduce" in r["Kernel_Name"]))
        spans.append((int(blk[-1]["End_Timestamp"]) - int(blk[0]["Start_Timestamp"])) / 1e3)
    return sums, spans


def _median(v):
    v = sorted(v)
    return v[len(v) // 2] if v else float("nan")


def main(run_dir):
    sys.path.insert(0, ROOT)
    from bench import conv_label, conv_launches, launch_costs
    from paper_1809_02697_amd.profile_layers import COPY_MB
    copy_bytes = COPY_MB * 2 ** 20
    pmc = os.path.join(run_dir, "pmc")

    desc = json.load(open(os.path.join(run_dir, "tune_db.txt.plan.json")))
    steps = conv_launches(desc)
    n_steps = len(desc["steps"])
    n = len(steps)
    bench = json.loads([l for l in open(os.path.join(run_dir, "bench.log")) if l.startswith("{")][0])
    ev_avg = bench["roofline"]["avg_launch_us"]
    flops = [launch_costs(m)[0] for _, m, _ in steps]

    # -- launch durations from the kernel trace -------------------------------------------
    trace = os.path.join(run_dir, "prof_bench", "bench_kernel_trace.csv")
    fwds = [f for f in stepwise_forward_durations(trace, n_steps) if len(f) == n]
    per_launch = [sum(f) / n for f in fwds]
    tr_avg = _median(per_launch)
    tr_sum = _median([sum(f) for f in fwds])
    per_step = [_median([f[i] for f in fwds]) for i in range(n)]
    g_sums, g_spans = graph_forward_durations(trace, n_steps)
    launch = bench["config"]["plan_choice"].get("launch", "graph")
    mode = "one hipGraph replay" if launch == "graph" else "steps launched on the stream"
    tr_tf = sum(flops) / (tr_avg * n * 1e-6) / 1e12

    # -- traffic, warm and cold -------------------------------------------------------------
    def traffic(tag):
        f_copy, f_fwd = forward_dispatches(os.path.join(pmc, f"fetch{tag}_counter_collection.csv"))
        w_copy, w_fwd = forward_dispatches(os.path.join(pmc, f"write{tag}_counter_collection.csv"))
        ff, fw = copy_bytes / (f_copy * 1024.0), copy_bytes / (w_copy * 1024.0)
        rd = [v * 1024 * ff for v in per_conv(f_fwd)]
        wr = [v * 1024 * fw for v in per_conv(w_fwd)]
        assert len(rd) == len(wr) == n, (tag, len(rd), len(wr), n)
        return rd, wr, ff, fw
    rd_w, wr_w, ff, fw = traffic("")
    rd_c, wr_c, ffc, fwc = traffic("_cold")
    alg = [launch_costs(m)[1] for _, m, _ in steps]
    tot_w = sum(rd_w) + sum(wr_w)

    # -- MFMA utilisation -------------------------------------------------------------------
    def mfma(tag):
        path = os.path.join(pmc, f"{tag}_counter_collection.csv")
        _, util = forward_dispatches(path, "MfmaUtil")
        _, mops = forward_dispatches(path, "SQ_INSTS_VALU_MFMA_MOPS_F32")
        _, busy = forward_dispatches(path, "SQ_VALU_MFMA_BUSY_CYCLES")
        return per_conv_max(util), per_conv(mops), per_conv(busy)
    util1, mops1, busy1 = mfma("mfma")
    assert len(util1) == n, (len(util1), n)
    # busy MFMA time per SIMD (us), and the cycles one 16x16x4 fp32 MFMA keeps it busy
    busy_us = [b / SIMDS / CLOCK_MHZ for b in busy1]
    cyc_per_mfma = sum(busy1) / (sum(mops1) * 512 / 2048)

    traffic_json = dict(kernel="conv2d_blocked", workload=f"ResNet-50 batch 1, 53 convs in {n} launches",
                        kernel_source_sha256=kernel_hash(),
                        traffic_bytes_per_launch=round(tot_w / n),
                        traffic_bytes_per_launch_cold=round((sum(rd_c) + sum(wr_c)) / n),
                        alg_bytes_per_launch=round(sum(alg) / n),
                        fetch_calibration=round(ff, 4), write_calibration=round(fw, 4))
    os.makedirs(PROFILES, exist_ok=True)
    with open(os.path.join(PROFILES, "conv2d_blocked_resnet50_b1_traffic.json"), "w") as f:
        json.dump(traffic_json, f, indent=1)

    md = [f"# conv2d_blocked, ResNet-50 batch 1 (53 convs in {n} launches per forward)", "",
          "Commands (run from the repository root on one MI355X; RUN_DIR = the directory they write to):", "",
          "```"] + COMMANDS + ["```", "",
          f"Kernel source sha256[:16]: `{kernel_hash()}`", "",
          "## Launch duration", "",
          f"- Kernel-trace timestamps of the {len(fwds)} forwards the profiled bench run launched "
          f"step by step between events: median per conv launch (its split_reduce pass included) "
          f"**{tr_avg:.3f} us**; the {n} conv launches of one forward sum to {tr_sum:.1f} us.",
          f"- bench.py (unprofiled), HIP events around back-to-back graph replays of each conv step: "
          f"**{ev_avg:.3f} us** per launch; trace / events = {tr_avg / ev_avg:.3f}.",
          f"- roofline.frac from the trace: {tr_tf:.2f} TFLOP/s / {PEAK} = "
          f"**{tr_tf / PEAK:.4f}**; bench.py: {bench['roofline']['achieved']} TFLOP/s, frac "
          f"**{bench['roofline']['frac']}**.",
          f"- bench.py e2e ResNet-50 batch 1 ({mode}): {bench['ms_per_step']} ms per forward "
          f"(step by step between events: {bench.get('stepwise_forward_ms', 'n/a')} ms).  The "
          f"traced forward's conv launches ({tr_sum:.1f} us) fit in the e2e forward.",
          f"- Under the profiler, back-to-back forwards run slower: the {len(g_sums)} profiled e2e "
          f"forwards ({mode}) span {_median(g_spans):.1f} us with {_median(g_sums):.1f} us of conv "
          f"dispatches ({_median(g_sums) / n:.2f} us per launch); these are not used.", "",
          "rocprofv3 --stats (the profiled bench run; all dispatches of the run):", "",
          "| kernel | calls | avg us | total % |", "|---|---:|---:|---:|"]
    stats = _rows(os.path.join(run_dir, "prof_bench", "bench_kernel_stats.csv"))
    for r in sorted(stats, key=lambda r: -float(r["Percentage"]))[:12]:
        name = r["Name"].replace("void ", "").replace("neo::(anonymous namespace)::", "")
        name = name.split("(neo")[0].split("(float")[0][:70]
        md.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                  f"{float(r['Percentage']):.1f} |")
    md += ["", "## Per launch: duration in the forward, traffic, MFMA utilisation", "",
           f"Calibration: a {COPY_MB} MB copy gives factors {ff:.3f} (FETCH_SIZE) / {fw:.3f} "
           f"(WRITE_SIZE) warm, {ffc:.3f} / {fwc:.3f} cold.", "",
           f"- warm, mean per launch: **{tot_w / n / 1e6:.3f} MB** measured vs "
           f"{sum(alg) / n / 1e6:.3f} MB algorithmic (ratio {tot_w / sum(alg):.2f})",
           f"- cold (HBM), mean per launch: **{(sum(rd_c) + sum(wr_c)) / n / 1e6:.3f} MB** "
           f"(ratio {(sum(rd_c) + sum(wr_c)) / sum(alg):.2f})",
           f"- MFMA busy time (SQ_VALU_MFMA_BUSY_CYCLES over {SIMDS} SIMDs at {CLOCK_MHZ:.0f} MHz; "
           f"{cyc_per_mfma:.1f} busy cycles per 16x16x4 fp32 MFMA) over the traced duration, all "
           f"launches: **{100 * sum(busy_us) / sum(per_step):.1f} %**.  rocprofv3's MfmaUtil "
           f"divides by the dispatch's active cycles under counter collection, which at batch 1 "
           f"are longer than the unprofiled duration, so it reads lower.", "",
           "| # | layer | us (trace) | TFLOP/s | % peak | alg MB | warm read / write MB | "
           "cold read / write MB | MFMA busy us | busy / us % | MfmaUtil % | MFMA flop / alg flop |",
           "|---:|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    for i, (_, members, _) in enumerate(steps):
        name = " + ".join(conv_label(c) for c, _ in members)
        tf = flops[i] / (per_step[i] * 1e-6) / 1e12
        md.append(f"| {i} | {name} | {per_step[i]:.2f} | {tf:.1f} | {100 * tf / PEAK:.1f} | "
                  f"{alg[i] / 1e6:.3f} | {rd_w[i] / 1e6:.3f} / {wr_w[i] / 1e6:.3f} | "
                  f"{rd_c[i] / 1e6:.3f} / {wr_c[i] / 1e6:.3f} | {busy_us[i]:.2f} | "
                  f"{100 * busy_us[i] / per_step[i]:.1f} | {util1[i]:.1f} | "
                  f"{mops1[i] * 512 / flops[i]:.3f} |")
    with open(os.path.join(PROFILES, "conv2d_blocked_resnet50_b1.md"), "w") as f:
        f.write("\n".join(md) + "\n")

    # -- batch 32 ---------------------------------------------------------------------------
    p32 = os.path.join(pmc, "mfma32_counter_collection.csv")
    if os.path.exists(p32) and os.path.exists(os.path.join(run_dir, "plan_b32.json")):
        d32 = json.load(open(os.path.join(run_dir, "plan_b32.json")))
        s32 = conv_launches(d32)
        _, util = forward_dispatches(p32, "MfmaUtil")
        _, mops = forward_dispatches(p32, "SQ_INSTS_VALU_MFMA_MOPS_F32")
        _, busy = forward_dispatches(p32, "SQ_VALU_MFMA_BUSY_CYCLES")
        util, mops, busy = per_conv_max(util), per_conv(mops), per_conv(busy)
        assert len(util) == len(s32), (len(util), len(s32))
        md = ["# conv2d_blocked, ResNet-50 batch 32: MFMA utilisation per launch", "",
              "Command (from the repository root, RUN_DIR as above; the plan and results file "
              "of the bench run above):", "", "```", COMMANDS[7], COMMANDS[-1], "```", "",
              f"Kernel source sha256[:16]: `{kernel_hash()}`", "",
              "MfmaUtil = busy MFMA cycles summed over the 1024 SIMDs / (GPU active cycles x "
              "1024), per dispatch (the conv kernel; a split_reduce pass is not counted). "
              "The last column is the MFMA work executed (SQ_INSTS_VALU_MFMA_MOPS_F32 x 512) over "
              "the algorithmic FLOPs: above 1 where padded channels or masked pixels are "
              "multiplied.", "",
              "| # | layer | MfmaUtil % | MFMA busy us | MFMA flop / alg flop |",
              "|---:|---|---:|---:|---:|"]
        for i, (_, members, _) in enumerate(s32):
            f32 = launch_costs(members)[0]
            md.append(f"| {i} | {' + '.join(conv_label(c) for c, _ in members)} | {util[i]:.1f} | "
                      f"{busy[i] / SIMDS / CLOCK_MHZ:.2f} | {mops[i] * 512 / f32:.3f} |")
        with open(os.path.join(PROFILES, "conv2d_blocked_resnet50_b32_mfma.md"), "w") as f:
            f.write("\n".join(md) + "\n")
    # -- Winograd, batch 32 ------------------------------------------------------------------
    pw = os.path.join(pmc, "mfma32w_counter_collection.csv")
    tw = os.path.join(run_dir, "prof_wino", "wino_kernel_trace.csv")
    if os.path.exists(pw) and os.path.exists(tw) and os.path.exists(os.path.join(run_dir, "plan_b32w.json")):
        write_winograd(run_dir, pw, tw)
    print(json.dumps(dict(traffic_json, trace_avg_launch_us=round(tr_avg, 3),
                          bench_avg_launch_us=ev_avg, trace_frac=round(tr_tf / PEAK, 4),
                          bench_frac=bench["roofline"]["frac"])))


def write_winograd(run_dir, pmc_path, trace_path):
    """profiles/wino_f2x3_resnet50_b32.md: the Winograd launches of the tuned
    batch-32 plan -- trace durations, MFMA utilisation and executed MFMA work
    over the algorithmic Winograd work and over the direct convolution's."""
    from bench import conv_label, conv_launches, launch_costs, wino_mfma_flops
    d = json.load(open(os.path.join(run_dir, "plan_b32w.json")))
    launches = conv_launches(d)
    wi = [k for k, (_, _, cfg) in enumerate(launches) if cfg.get("algo") == "winograd"]
    _, util = forward_dispatches(pmc_path, "MfmaUtil")
    _, mops = forward_dispatches(pmc_path, "SQ_INSTS_VALU_MFMA_MOPS_F32")
    _, busy = forward_dispatches(pmc_path, "SQ_VALU_MFMA_BUSY_CYCLES")
    util, mops, busy = per_conv_max(util), per_conv(mops), per_conv(busy)
    assert len(util) == len(launches), (len(util), len(launches))
    # trace: the Winograd dispatches (and a split_reduce right after one), in plan order, repeated
    rows = sorted(_rows(trace_path), key=lambda r: int(r["Start_Timestamp"]))
    durs = []
    prev_wino = False
    for r in rows:
        n = r["Kernel_Name"]
        us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        if "wino_f2x3" in n:
            durs.append(us)
            prev_wino = True
        elif "split_reduce" in n and prev_wino:
            durs[-1] += us
        elif is_neo(n):
            prev_wino = False
    nw = len(wi)
    reps = len(durs) // nw
    assert reps >= 2 and len(durs) % nw == 0, (len(durs), nw)
    per = [_median([durs[r * nw + j] for r in range(1, reps)]) for j in range(nw)]
    md = ["# wino_f2x3 (Winograd F(2x2, 3x3)), ResNet-50 batch 32: duration and MFMA utilisation",
          "", "Commands (from the repository root, RUN_DIR as in the batch-1 summary; the results file of the "
          "bench run above, whose `winograd` plan this is):", "", "```", COMMANDS[-3], COMMANDS[-2],
          COMMANDS[-1], "```", "",
          "The tuned one-block plan with NEO_PLAN_WINOGRAD: the local search keeps the Winograd "
          "kernel for the 3x3 stride-1 convs listed.  Duration: median over the profiled repetitions "
          "(the first dropped) of the kernel-trace timestamps.  TFLOP/s counts the direct "
          "convolution's FLOPs (the metric's definition); MFMA work is the executed "
          "SQ_INSTS_VALU_MFMA_MOPS_F32 x 512, against the Winograd algorithm's 2 x 16 x K x C per 2x2 "
          "tile and against the direct FLOPs.", "",
          "| # | layer | config (tile, split, waves) | us | TFLOP/s (direct count) | MfmaUtil % | "
          "MFMA work / Winograd work | MFMA work / direct FLOPs |",
          "|---:|---|---|---:|---:|---:|---:|---:|"]
    for j, k in enumerate(wi):
        _, members, cfg = launches[k]
        c = members[0][0]
        f_direct = launch_costs(members)[0]
        md.append(f"| {k} | {conv_label(c)} | {cfg['tile']}, {cfg['split']}, {cfg['waves']} | "
                  f"{per[j]:.2f} | {f_direct / (per[j] * 1e-6) / 1e12:.1f} | {util[k]:.1f} | "
                  f"{mops[k] * 512 / wino_mfma_flops(c):.3f} | {mops[k] * 512 / f_direct:.3f} |")
    with open(os.path.join(PROFILES, "wino_f2x3_resnet50_b32.md"), "w") as f:
        f.write("\n".join(md) + "\n")


def write_int8(run_dir):
    """profiles/conv_i8_resnet50_b32.md: the integer conv of each ResNet-50
    shape at batch 32 -- kernel-trace durations, HBM traffic against the
    algorithmic bytes, MFMA utilisation."""
    sys.path.insert(0, ROOT)
    from paper_1809_02697_amd import workloads as wl
    from paper_1809_02697_amd.profile_layers import COPY_MB
    copy_bytes = COPY_MB * 2 ** 20
    layers = wl.RESNET50_LAYERS
    n = len(layers)
    # durations: the conv_i8 dispatches after the last copy, n per round
    rows = sorted(_rows(os.path.join(run_dir, "prof_i8", "i8_kernel_trace.csv")),
                  key=lambda r: int(r["Start_Timestamp"]))
    last_copy = max(i for i, r in enumerate(rows) if "copyBuffer" in r["Kernel_Name"])
    durs = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
            for r in rows[last_copy + 1:] if is_conv_i8(r["Kernel_Name"])]
    reps = len(durs) // n
    assert reps >= 2 and len(durs) == reps * n, (len(durs), n)
    per = [_median([durs[r * n + j] for r in range(1, reps)]) for j in range(n)]
    pmc = os.path.join(run_dir, "pmc")

    def after_copy(tag, counter=None):
        copy, fwd = forward_dispatches(os.path.join(pmc, f"{tag}_counter_collection.csv"), counter)
        vals = [v for name, v in fwd if is_conv_i8(name)]
        assert len(vals) == n, (tag, len(vals))
        return copy, vals
    f_copy, fetch = after_copy("i8fetch")
    w_copy, write = after_copy("i8write")
    ff, fw = copy_bytes / (f_copy * 1024.0), copy_bytes / (w_copy * 1024.0)
    _, mops = after_copy("i8mfma", "SQ_INSTS_VALU_MFMA_MOPS_I8")
    _, busy = after_copy("i8mfma", "SQ_VALU_MFMA_BUSY_CYCLES")
    _, gui = after_copy("i8mfma", "GRBM_GUI_ACTIVE")
    N = 32
    md = ["# conv_i8 (INT8 convolution, v_mfma_i32_16x16x64_i8), ResNet-50 shapes at batch 32", "",
          "Commands (from the repository root on one MI355X; RUN_DIR = the directory they write to):",
          "", "```"] + INT8_COMMANDS + ["```", "",
          "Each of the 23 distinct ResNet-50 conv shapes at batch 32 through the integer path "
          "(int8 input with its halo, packed int8 filter, float32 output with the layer's residual "
          "and ReLU), in the launch configuration the library chooses.  Duration: median over the "
          "profiled rounds (the first dropped) of the kernel-trace timestamps; the layers run "
          "round-robin, so each one's operands have left the 256 MB MALL by its turn (the bench "
          "line's layer table replays one layer back to back, warm, and measures less on the "
          "layers with large outputs).  Traffic: FETCH_SIZE "
          "and WRITE_SIZE (KiB per dispatch) scaled by the same counters on a plain copy of "
          f"{COPY_MB} MB (factors {ff:.3f} and {fw:.3f}), warm caches, against the algorithmic "
          "bytes (int8 input and filter once, float32 output and residual).  MFMA utilisation: "
          "SQ_VALU_MFMA_BUSY_CYCLES over (GRBM_GUI_ACTIVE x 1024 SIMDs / 8 XCDs); executed MFMA "
          "work is SQ_INSTS_VALU_MFMA_MOPS_I8 x 512 over the direct convolution's 2 N K C R S OH OW "
          "(above 1 where padded channels are multiplied).", "",
          "| layer | shape | us | TOPS | % of 5.0 POP/s | traffic MB | algorithmic MB | "
          "traffic / alg | MFMA util % | MFMA work / alg ops |",
          "|---|---|---:|---:|---:|---:|---:|---:|---:|---:|"]
    tot_t = tot_ops = 0.0
    for j, (lid, C, K, R, st, pd, H, epi, uses) in enumerate(layers):
        OH = (H + 2 * pd - R) // st + 1
        ops = 2 * N * K * C * R * R * OH * OH
        alg = N * C * H * H + K * C * R * R + 4 * N * K * OH * OH * (2 if epi == "res" else 1) + 8 * K
        traffic = fetch[j] * 1024 * ff + write[j] * 1024 * fw
        util = 100 * busy[j] / (gui[j] / 8 * SIMDS) if gui[j] else 0.0
        tops = ops / (per[j] * 1e-6) / 1e12
        tot_t += per[j] * uses
        tot_ops += ops * uses
        md.append(f"| {lid} | {C}->{K} {R}x{R}/s{st} {H}->{OH}{' +res' if epi == 'res' else ''} | "
                  f"{per[j]:.2f} | {tops:.0f} | {100 * tops / 5000:.1f} | {traffic / 1e6:.2f} | "
                  f"{alg / 1e6:.2f} | {traffic / alg:.2f} | {util:.1f} | {mops[j] * 512 / ops:.3f} |")
    md += ["", f"Whole network (each shape times its uses, 53 convs): {tot_t:.1f} us of conv_i8, "
               f"{tot_ops / (tot_t * 1e-6) / 1e12:.0f} TOPS."]
    with open(os.path.join(PROFILES, "conv_i8_resnet50_b32.md"), "w") as f:
        f.write("\n".join(md) + "\n")


def write_int8_plans(run_dir):
    """profiles/int8_plans_b1.md: where the time of one integer forward at
    batch 1 goes (the tuned, grouped plans the bench line's int8 entries
    time), from the kernel-trace timestamps of graph-replayed forwards."""
    md = ["# Integer networks at batch 1 (NEO_PLAN_INT8 | GROUP | TUNE)", "",
          "Commands (from the repository root on one MI355X; RUN_DIR = the directory they write to):",
          "", "```"] + INT8_PLAN_COMMANDS + ["```", "",
          f"Each workload calibrates the plan on the network's input, runs one forward, a plain copy "
          f"(the marker), then {INT8_PLAN_REPS} forwards step by step, each step alone on the GPU "
          "(under the profiler, back-to-back launches run slower than unprofiled; launched alone "
          "their durations match HIP-event timings).  Per forward: the dispatches after the copy "
          "in equal runs, each kernel's kernel-trace duration summed by what it does (median over "
          "the forwards, the first dropped).  Launched alone, each of these small kernels pays "
          "its whole start-up (wave launch, instruction and argument fetch), which the "
          "unprofiled graph replays of the bench line (models.*.int8_grouped) overlap with the "
          "previous kernel's tail: the sums below exceed that end-to-end latency, so read the "
          "shares, not the absolute times.", ""]
    e2e = {}
    try:
        line = open(os.path.join(run_dir, "bench.log")).read().strip().splitlines()[-1]
        for k, v in (json.loads(line).get("models") or {}).items():
            if isinstance(v.get("int8_grouped"), dict):
                e2e[k] = v["int8_grouped"]["ms"]
    except (OSError, ValueError, IndexError):
        pass
    for m in INT8_PLAN_MODELS:
        path = os.path.join(run_dir, "prof_i8plan", f"{m}_kernel_trace.csv")
        if not os.path.exists(path):
            continue
        rows = sorted(_rows(path), key=lambda r: int(r["Start_Timestamp"]))
        last_copy = max(i for i, r in enumerate(rows) if "copyBuffer" in r["Kernel_Name"])
        fwd = rows[last_copy + 1:]
        n = len(fwd) // INT8_PLAN_REPS
        assert n > 0 and len(fwd) == n * INT8_PLAN_REPS, (m, len(fwd))
        kinds = {}
        spans, totals = [], []
        for r in range(1, INT8_PLAN_REPS):
            part = fwd[r * n:(r + 1) * n]
            spans.append((int(part[-1]["End_Timestamp"]) - int(part[0]["Start_Timestamp"])) / 1e3)
            per = {}
            for row in part:
                name = row["Kernel_Name"]
                kind = next((k for pat, k in INT8_PLAN_KINDS if pat in name), "other")
                t = (int(row["End_Timestamp"]) - int(row["Start_Timestamp"])) / 1e3
                c, u = per.get(kind, (0, 0.0))
                per[kind] = (c + 1, u + t)
            for kind, (c, u) in per.items():
                kinds.setdefault(kind, []).append((c, u))
            totals.append(sum(u for _, u in per.values()))
        ref = (f"; the bench run of this directory replays the forward in {e2e[m + '_b1'] * 1e3:.1f} us"
               if m + "_b1" in e2e else "")
        md += [f"## {m}", "",
               f"{n} dispatches per forward; kernel time, each launched alone, {_median(totals):.1f} us{ref}.",
               "",
               "| part | dispatches | us per forward | share of kernel time |", "|---|---:|---:|---:|"]
        tot = _median(totals)
        for kind, vals in sorted(kinds.items(), key=lambda kv: -_median([u for _, u in kv[1]])):
            u = _median([u for _, u in vals])
            md.append(f"| {kind} | {vals[0][0]} | {u:.1f} | {100 * u / tot:.0f} % |")
        md.append("")
    with open(os.path.join(PROFILES, "int8_plans_b1.md"), "w") as f:
        f.write("\n".join(md) + "\n")


if __name__ == "__main__":
    if len(sys.argv) != 2:
        sys.exit("usage: python -m paper_1809_02697_amd.profile_summary RUN_DIR")
    if os.path.isdir(os.path.join(sys.argv[1], "prof_i8plan")):
        write_int8_plans(sys.argv[1])
    if os.path.exists(os.path.join(sys.argv[1], "prof_i8", "i8_kernel_trace.csv")):
        write_int8(sys.argv[1])
    if os.path.exists(os.path.join(sys.argv[1], "bench.log")):
        main(sys.argv[1])
