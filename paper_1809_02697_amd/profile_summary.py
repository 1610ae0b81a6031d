"""Summarize rocprofv3 output of the ResNet-50 batch-1 conv kernels into profiles/.

    python -m paper_1809_02697_amd.profile_summary RUN_DIR

RUN_DIR holds (names as written by the commands below):
  prof_bench/bench_kernel_stats.csv, prof_bench/bench_kernel_trace.csv
      rocprofv3 --kernel-trace --stats --output-format csv -d RUN_DIR/prof_bench -o bench --
          python bench.py --no-cpu --no-models --tune-db RUN_DIR/tune_db.txt --latency-runs 100
  pmc/fetch_counter_collection.csv, pmc/write_counter_collection.csv
      rocprofv3 --pmc FETCH_SIZE --output-format csv -d RUN_DIR/pmc -o fetch --
          python -m paper_1809_02697_amd.profile_layers        (and WRITE_SIZE / -o write)
  bench.log   the JSON line of a plain `python bench.py --no-cpu --save-tune-db
              RUN_DIR/tune_db.txt` run on the same box

Writes profiles/conv2d_blocked_resnet50_b1.md (durations, traffic per layer)
and profiles/conv2d_blocked_resnet50_b1_traffic.json (bytes per launch, tied to
the hash of the kernel source it was measured with; bench.py reports it only
while the source is unchanged).

FETCH_SIZE / WRITE_SIZE are KiB moved between L2 and the fabric per dispatch.
They are calibrated by the same counters on a plain copy of COPY_MB megabytes
(which reads and writes exactly that many bytes); the figures include reads
served by the 256 MB MALL, which these counters cannot tell from HBM.
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
               for f in ("conv_kernel.h", "conv.hip", "conv_xy.hip", "conv_group.hip", "conv_pair.hip")]


def kernel_hash():
    """sha256[:16] of the conv kernel's sources (templates and instantiations)."""
    h = hashlib.sha256()
    for f in KERNEL_SRCS:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def _rows(path):
    with open(path) as f:
        return list(csv.DictReader(f))


def forward_dispatches(path):
    """Counter values of the dispatches after the last copy kernel (one
    forward pass, in launch order) and of that copy."""
    rows = _rows(path)
    last_copy = max(i for i, r in enumerate(rows) if "copyBuffer" in r["Kernel_Name"])
    copy = float(rows[last_copy]["Counter_Value"])
    fwd = [(r["Kernel_Name"], float(r["Counter_Value"])) for r in rows[last_copy + 1:]]
    return copy, fwd


def conv_launches(run_dir):
    """The conv launches of the plan the bench run timed (its description is
    saved next to the results file): one conv or a fused group each."""
    from bench import conv_launches as launches
    return launches(json.load(open(os.path.join(run_dir, "tune_db.txt.plan.json"))))


def is_conv(name):
    return "conv2d_mfma" in name or "conv1x1_pair" in name or "conv3x3_chain" in name


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


def main(run_dir):
    sys.path.insert(0, ROOT)
    from bench import conv_label, launch_costs
    from paper_1809_02697_amd.profile_layers import COPY_MB
    copy_bytes = COPY_MB * 2 ** 20

    f_copy, f_fwd = forward_dispatches(os.path.join(run_dir, "pmc", "fetch_counter_collection.csv"))
    w_copy, w_fwd = forward_dispatches(os.path.join(run_dir, "pmc", "write_counter_collection.csv"))
    ff = copy_bytes / (f_copy * 1024.0)
    fw = copy_bytes / (w_copy * 1024.0)
    fetch = per_conv(f_fwd)
    write = per_conv(w_fwd)
    steps = conv_launches(run_dir)
    n_convs = sum(len(m) for _, m, _ in steps)
    assert n_convs == 53 and len(fetch) == len(write) == len(steps), (len(fetch), len(write), len(steps))

    layer_rows = []
    tot_alg = tot_traffic = 0.0
    for (_, members, _), fv, wv in zip(steps, fetch, write):
        alg = launch_costs(members)[1]
        rd, wr = fv * 1024 * ff, wv * 1024 * fw
        tot_alg += alg
        tot_traffic += rd + wr
        layer_rows.append((" + ".join(conv_label(c) for c, _ in members), alg, rd, wr))

    trace = _rows(os.path.join(run_dir, "prof_bench", "bench_kernel_trace.csv"))
    dur = lambda r: (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    conv_d = [dur(r) for r in trace if is_conv(r["Kernel_Name"])]
    red_d = [dur(r) for r in trace if "split_reduce" in r["Kernel_Name"]]
    trace_avg = (sum(conv_d) + sum(red_d)) / len(conv_d)
    stats = _rows(os.path.join(run_dir, "prof_bench", "bench_kernel_stats.csv"))
    bench = json.loads([l for l in open(os.path.join(run_dir, "bench.log")) if l.startswith("{")][0])
    ev_avg = bench["roofline"]["avg_launch_us"]

    n = len(steps)
    traffic = dict(kernel="conv2d_blocked", workload=f"ResNet-50 batch 1, 53 convs in {n} launches",
                   kernel_source_sha256=kernel_hash(),
                   traffic_bytes_per_launch=round(tot_traffic / n),
                   alg_bytes_per_launch=round(tot_alg / n),
                   fetch_calibration=round(ff, 4), write_calibration=round(fw, 4))
    os.makedirs(PROFILES, exist_ok=True)
    with open(os.path.join(PROFILES, "conv2d_blocked_resnet50_b1_traffic.json"), "w") as f:
        json.dump(traffic, f, indent=1)

    md = [f"# conv2d_blocked, ResNet-50 batch 1 (53 convs in {n} launches per forward)", "",
          "Commands (run from the repository root on one MI355X; RUN_DIR = gpurun_out):", "",
          "```",
          "python bench.py --save-tune-db RUN_DIR/tune_db.txt > RUN_DIR/bench.log",
          "rocprofv3 --kernel-trace --stats --output-format csv -d RUN_DIR/prof_bench -o bench -- "
          "python bench.py --no-cpu --no-models --tune-db RUN_DIR/tune_db.txt --latency-runs 100",
          "rocprofv3 --pmc FETCH_SIZE --output-format csv -d RUN_DIR/pmc -o fetch -- "
          "python -m paper_1809_02697_amd.profile_layers RUN_DIR/tune_db.txt",
          "rocprofv3 --pmc WRITE_SIZE --output-format csv -d RUN_DIR/pmc -o write -- "
          "python -m paper_1809_02697_amd.profile_layers RUN_DIR/tune_db.txt",
          "python -m paper_1809_02697_amd.profile_summary RUN_DIR",
          "```", "",
          f"Kernel source sha256[:16]: `{kernel_hash()}`", "",
          "## Launch duration", "",
          f"- rocprofv3 kernel trace, mean per conv launch (conv2d_mfma, conv2d_mfma_group, conv1x1_pair or conv3x3_chain + its "
          f"split_reduce pass, "
          f"{len(conv_d)} conv dispatches): **{trace_avg:.2f} us**",
          f"- bench.py HIP events (graph replays of each conv step, weighted by use): "
          f"**{ev_avg:.2f} us** (ratio {trace_avg / ev_avg:.3f})",
          f"- bench.py e2e ResNet-50 batch 1: {bench['latency_ms']} ms; conv layers "
          f"{bench['roofline']['achieved']} TFLOP/s = {100 * bench['roofline']['frac']:.1f} % of "
          f"157.3 TFLOP/s", "",
          "rocprofv3 --stats (profiled bench run; all dispatches of the run):", "",
          "| kernel | calls | avg us | total % |", "|---|---:|---:|---:|"]
    for r in sorted(stats, key=lambda r: -float(r["Percentage"]))[:12]:
        name = r["Name"].replace("void ", "").replace("neo::(anonymous namespace)::", "")
        name = name.split("(neo")[0].split("(float")[0][:70]
        md.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                  f"{float(r['Percentage']):.1f} |")
    md += ["", "## HBM / fabric traffic per conv launch", "",
           f"Calibration: a {COPY_MB} MB copy reads {f_copy / 1024:.1f} MiB (FETCH_SIZE) and writes "
           f"{w_copy / 1024:.1f} MiB (WRITE_SIZE): factors {ff:.3f} / {fw:.3f}.", "",
           f"- mean per launch: **{tot_traffic / n / 1e6:.3f} MB** measured vs "
           f"{tot_alg / n / 1e6:.3f} MB algorithmic (ratio {tot_traffic / tot_alg:.2f})", "",
           "| # | layer | algorithmic MB | read MB | write MB | (read+write)/alg |",
           "|---:|---|---:|---:|---:|---:|"]
    for i, (name, alg, rd, wr) in enumerate(layer_rows):
        md.append(f"| {i} | {name} | {alg / 1e6:.3f} | {rd / 1e6:.3f} | {wr / 1e6:.3f} | "
                  f"{(rd + wr) / alg:.2f} |")
    with open(os.path.join(PROFILES, "conv2d_blocked_resnet50_b1.md"), "w") as f:
        f.write("\n".join(md) + "\n")
    print(json.dumps(traffic))


if __name__ == "__main__":
    main(sys.argv[1] if len(sys.argv) > 1 else "gpurun_out")
