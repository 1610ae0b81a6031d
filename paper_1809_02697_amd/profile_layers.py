"""Workload for hardware-counter passes over the ResNet-50 plan bench.py times.

    rocprofv3 --pmc FETCH_SIZE --output-format csv -d OUT -o fetch -- \\
        python -m paper_1809_02697_amd.profile_layers TUNE_DB [--cold] [--batch 32]
    rocprofv3 --pmc WRITE_SIZE ...                       (the same workload)
    rocprofv3 --pmc MfmaUtil SQ_INSTS_VALU_MFMA_MOPS_F32 ... (the same workload)
    ... profile_layers TUNE_DB --batch 32 --winograd [--reps 20]   (Winograd plan)
    ... profile_layers --int8 --batch 32 [--reps 20]    (the integer convs, no plan)
    ... profile_layers --int8-plan MODEL --batch 1 --reps 20   (a whole int8 network)

Builds the plan bench.py times (batch 1: the headline plan; batch 32: the
tuned one-block plan of the batch-32 layer table).  TUNE_DB is a local-search
results file written by ``bench.py --save-tune-db``: the launch configurations
and the global search's schemes come from that run, so no tuning launches are
profiled.  It runs one forward, then a plain device-to-device copy of COPY_MB
megabytes (the calibration kernel: it reads and writes exactly that many
bytes) and then every step of the plan once, in order: the dispatches after
the copy are one forward pass.  With --cold a 512 MB buffer (twice the 256 MB
MALL) is overwritten before every step, so each step's operands come from HBM
and FETCH_SIZE counts HBM reads.  ``paper_1809_02697_amd.profile_summary``
turns the counter files into per-launch figures.
"""
import argparse
import json
import sys

COPY_MB = 64
FLUSH_MB = 512


def build_plan(neo, torch, wl, db, batch, winograd=False):
    """(plan, graph) of the run whose results file is `db`; with `winograd`
    the tuned one-block plan whose 3x3 stride-1 convs may run by Winograd
    F(2x2, 3x3) (bench.py's ``winograd`` plan)."""
    from bench import headline_plan
    if db:
        neo.tune_db_load(db)
    g = wl.resnet50(batch)
    if winograd:
        plan = neo.Plan(g, flags=neo.PLAN_TUNE | neo.PLAN_HIPGRAPH | neo.PLAN_WINOGRAD)
    elif batch == 1:
        plan, _ = headline_plan(neo, g, db, torch)
    else:
        plan = neo.Plan(g, flags=neo.PLAN_TUNE | neo.PLAN_HIPGRAPH)
    return plan, g


def int8_main(neo, torch, wl, batch, reps):
    """The integer conv of every ResNet-50 shape (set up by bench.int8_layer:
    quantized input with its halo, packed filter), then the calibration copy,
    then the 23 convs in layer order, `reps` times: the conv_i8 dispatches
    after the copy are those rounds."""
    from bench import int8_layer
    layers = [int8_layer(neo, torch, wl, i, batch) for i in range(len(wl.RESNET50_LAYERS))]
    for L in layers:
        L["conv"]()
    torch.cuda.synchronize()
    a = torch.ones(COPY_MB * 2 ** 18, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    for _ in range(reps):
        for L in layers:
            L["conv"]()
    torch.cuda.synchronize()
    print(f"profiled {len(layers)} int8 convs x {reps} after a {COPY_MB} MB copy (batch {batch})",
          file=sys.stderr)


def int8_plan_main(neo, torch, wl, model, batch, reps):
    """The integer network bench.py times as its int8_grouped entry
    (NEO_PLAN_INT8 | GROUP | TUNE | HIPGRAPH, calibrated on the network's
    input): one forward, the calibration copy, then `reps` forwards step by
    step, each step alone on the GPU (a synchronize after it: under the
    profiler, back-to-back launches run slower than they do unprofiled) --
    the dispatches after the copy, in equal runs."""
    g = wl.MODELS[model](batch)
    x = torch.from_numpy(g.x).cuda()
    plan = neo.Plan(g, flags=neo.PLAN_INT8 | neo.PLAN_GROUP | neo.PLAN_TUNE | neo.PLAN_HIPGRAPH)
    out = plan.calibrate_int8(x)
    plan.run(x, out)
    torch.cuda.synchronize()
    a = torch.ones(COPY_MB * 2 ** 18, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    d = plan.describe()
    for _ in range(reps):
        for i in range(len(d["steps"])):
            plan.run_step(i, x, out)
            torch.cuda.synchronize()
    print(f"profiled {reps} int8 forwards of {model} batch {batch} ({len(d['steps'])} steps) "
          f"after a {COPY_MB} MB copy", file=sys.stderr)
    plan.destroy()


def main():
    import torch

    from paper_1809_02697_amd import neo
    from paper_1809_02697_amd import workloads as wl

    ap = argparse.ArgumentParser()
    ap.add_argument("db", nargs="?")
    ap.add_argument("--cold", action="store_true")
    ap.add_argument("--batch", type=int, default=1)
    ap.add_argument("--describe", help="write the plan's description (JSON) here")
    ap.add_argument("--winograd", action="store_true",
                    help="the plan with NEO_PLAN_WINOGRAD (3x3 stride-1 convs by Winograd where faster)")
    ap.add_argument("--reps", type=int, default=1,
                    help="run the step list this many times (for kernel-trace durations)")
    ap.add_argument("--int8", action="store_true",
                    help="instead of a plan: the 23 ResNet-50 conv shapes through the integer "
                         "path (bench.py's int8 layer table), after the copy, --reps times")
    ap.add_argument("--int8-plan", metavar="MODEL",
                    help="instead: the tuned, grouped int8 plan of MODEL (resnet50, vgg16, "
                         "inception_v3), --reps graph replays after the copy")
    args = ap.parse_args()
    if args.int8:
        return int8_main(neo, torch, wl, args.batch, args.reps)
    if args.int8_plan:
        return int8_plan_main(neo, torch, wl, args.int8_plan, args.batch, args.reps)
    plan, g = build_plan(neo, torch, wl, args.db, args.batch, args.winograd)
    if args.describe:
        with open(args.describe, "w") as f:
            json.dump(plan.describe(), f)
    x = torch.from_numpy(g.x).cuda()
    out = torch.empty(plan.output_shape[:2], device="cuda")
    plan.run(x, out)
    flush = torch.empty(FLUSH_MB * 2 ** 18, device="cuda") if args.cold else None
    torch.cuda.synchronize()
    a = torch.ones(COPY_MB * 2 ** 18, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    n = len(plan.describe()["steps"])
    for _ in range(args.reps):
        for i in range(n):
            if flush is not None:
                flush.fill_(1.0)
            plan.run_step(i, x, out)
    torch.cuda.synchronize()
    print(f"profiled {n} steps after a {COPY_MB} MB copy (batch {args.batch}"
          f"{', cold' if args.cold else ''})", file=sys.stderr)
    plan.destroy()


if __name__ == "__main__":
    main()
