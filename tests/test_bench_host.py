"""Host checks of bench.py's bookkeeping: the algorithmic FLOPs and bytes of a
conv (closed forms), which convs each launch of a fused plan runs, the bytes a
pair or chain keeps in LDS instead of memory, and the one-GPU contract."""
import os
import subprocess
import sys

import pytest

from paper_1809_02697_amd import neo

import nets

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_conv_costs_closed_forms():
    # 3x3 s1 p1, 64 -> 64 at 56 x 56: 2 K C R S OH OW flops; input, filter,
    # output and bias once
    f, b, OH, OW = bench.conv_costs(64, 64, 3, 3, 56, 56, (1, 1), (1, 1))
    assert (OH, OW) == (56, 56)
    assert f == 2 * 64 * 64 * 9 * 56 * 56
    assert b == 4 * (64 * 56 * 56 + 64 * 64 * 9 + 64 * 56 * 56 + 64)
    # a strided 1x1 reads only the sampled input pixels; a residual is read once more
    f, b, OH, OW = bench.conv_costs(256, 512, 1, 1, 56, 56, (2, 2), (0, 0), N=2, residual=True)
    assert (OH, OW) == (28, 28)
    assert f == 2 * 2 * 512 * 256 * 28 * 28
    assert b == 4 * (2 * 256 * 28 * 28 + 512 * 256 + 2 * 2 * 512 * 28 * 28 + 512)


def _resnet_plan(flags):
    p = neo.Plan(nets.resnet50(), flags=neo.PLAN_HOST_ONLY | flags)
    d = p.describe()
    p.destroy()
    return d


FUSED = neo.PLAN_GROUP | neo.PLAN_FUSE_GAP | neo.PLAN_FUSE_PAIRS | neo.PLAN_FUSE_CHAINS


@pytest.mark.parametrize("flags", [0, neo.PLAN_GROUP, FUSED])
def test_every_conv_in_exactly_one_launch(flags):
    g = nets.resnet50()
    d = _resnet_plan(flags)
    launches = bench.conv_launches(d)
    ran = sorted((c["N"], c["C"], c["H"], c["K"], c["R"], c["stride"][0]) for _, ms, _ in launches
                 for c, _ in ms)
    assert len(ran) == sum(1 for n in g.nodes if n.op == "conv") == 53
    # the FLOPs of the step do not depend on how the convs are launched
    base = bench.plan_conv_flops(_resnet_plan(0))
    assert bench.plan_conv_flops(d) == base
    assert abs(base / 1e9 - 8.1743) < 1e-3          # ResNet-50's conv GFLOP per image


def test_pair_and_chain_bytes_exclude_what_stays_in_lds():
    d = _resnet_plan(FUSED)
    chains = [(ms, cfg) for _, ms, cfg in bench.conv_launches(d) if cfg.get("chain")]
    assert len(chains) == 3
    for ms, cfg in chains:
        (c, _), (a, ares), (b, _) = ms
        parts = sum(bench.conv_costs(m["C"], m["K"], m["R"], m["S"], m["H"], m["W"], m["stride"],
                                     m["pad"], N=m["N"], residual=r)[1] for m, r in ms)
        hw = c["H"] * c["W"]
        kept = 4 * hw * (c["K"]            # the 3x3's output, never stored ...
                         + a["C"]          # ... nor read back by the expansion
                         + b["C"])         # the expansion's output, read by the reduction from LDS
        assert ares
        assert bench.launch_costs(ms)[1] == parts - kept
        assert bench.launch_costs(ms)[0] == sum(
            bench.conv_costs(m["C"], m["K"], m["R"], m["S"], m["H"], m["W"], m["stride"], m["pad"],
                             N=m["N"])[0] for m, _ in ms)
    pd = _resnet_plan(neo.PLAN_FUSE_PAIRS)
    pairs = [ms for _, ms, cfg in bench.conv_launches(pd) if cfg.get("pair")]
    assert len(pairs) == 3
    for ms in pairs:
        (a, _), (b, _) = ms
        parts = sum(bench.conv_costs(m["C"], m["K"], m["R"], m["S"], m["H"], m["W"], m["stride"],
                                     m["pad"], N=m["N"], residual=r)[1] for m, r in ms)
        assert bench.launch_costs(ms)[1] == parts - 4 * b["C"] * b["H"] * b["W"]


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr or "1 GPU" in r.stderr or "--gpus 1" in r.stderr
    assert r.stdout == ""
