"""Workload for hardware-counter passes over the ResNet-50 batch-1 plan.

    rocprofv3 --pmc FETCH_SIZE --output-format csv -d OUT -o fetch -- \
        python -m paper_1809_02697_amd.profile_layers [TUNE_DB]
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d OUT -o write -- \
        python -m paper_1809_02697_amd.profile_layers [TUNE_DB]

Builds the plan bench.py times (with TUNE_DB, a local-search results file
written by ``bench.py --save-tune-db``, the launch configurations and the
global search's schemes come from that run, so no tuning launches are
profiled), runs one forward,
then a plain device-to-device copy of COPY_MB megabytes (the calibration
kernel: it reads and writes exactly that many bytes) and then every step of
the plan once, in order.  The dispatches after the copy are one forward pass.
``paper_1809_02697_amd.profile_summary`` turns the counter files into the
per-launch traffic figures.
"""
import sys

COPY_MB = 64


def main():
    import torch

    from bench import headline_plan
    from paper_1809_02697_amd import neo
    from paper_1809_02697_amd import workloads as wl

    db = sys.argv[1] if len(sys.argv) > 1 else None
    if db:
        neo.tune_db_load(db)
    g = wl.resnet50(1)
    plan, _ = headline_plan(neo, g, db, torch)
    x = torch.from_numpy(g.x).cuda()
    out = torch.empty((1, 1000), device="cuda")
    plan.run(x, out)
    torch.cuda.synchronize()
    a = torch.ones(COPY_MB * 2 ** 18, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    n = len(plan.describe()["steps"])
    for i in range(n):
        plan.run_step(i, x, out)
    torch.cuda.synchronize()
    print(f"profiled {n} steps after a {COPY_MB} MB copy", file=sys.stderr)
    plan.destroy()


if __name__ == "__main__":
    main()
