"""A network stem's conv and the max pooling that reads it in one launch
(NEO_PLAN_FUSE_POOL): the planner's choice on the host, and on the GPU the
fused launch against the oracle and, bit for bit, against the conv (one wave
per tile, no split) followed by the pooling kernel."""
import numpy as np
import pytest

import oracle as orc
from paper_1809_02697_amd import neo
from paper_1809_02697_amd import workloads as wl

import bench


def _host_plan(g, flags=0, schemes=None):
    p = neo.Plan(g, flags=flags | neo.PLAN_HOST_ONLY, schemes=schemes)
    d = p.describe()
    p.destroy()
    return d


def test_planner_fuses_the_resnet50_stem_and_its_pool():
    g = wl.resnet50(1)
    plain = _host_plan(g)
    fused = _host_plan(g, neo.PLAN_FUSE_POOL)
    assert len(fused["steps"]) == len(plain["steps"]) - 1
    cp = [s for s in fused["steps"] if s["kind"] == "conv_pool"]
    assert len(cp) == 1
    s = cp[0]
    assert g.nodes[s["members"][0]["node"]].name == "conv1"
    assert g.nodes[s["pool"]["node"]].op == "maxpool"
    assert s["pool"]["OH"] == s["pool"]["OW"] == 56
    # the fused step reads the conv's input and writes the pool's output
    pool_step = [t for t in plain["steps"] if t["kind"] == "maxpool"][0]
    assert s["out"] == pool_step["out"]
    assert not any(t["kind"] == "maxpool" for t in fused["steps"])
    # bench accounting: the conv's output is never stored, the pooled map is
    (_, members, cfg), = [l for l in bench.conv_launches(fused) if l[2].get("pool")]
    f, b = bench.launch_costs(members)
    f0, b0 = bench.launch_costs([(dict(members[0][0], lds_out=False, pooled=None), False)])
    assert f == f0 == 2 * 64 * 3 * 49 * 112 * 112
    assert b0 - b == 4 * 64 * (112 * 112 - 56 * 56)


def test_planner_leaves_other_convs_alone():
    # more than 4 input channels: not a stem
    assert not any(s["kind"] == "conv_pool" for s in _host_plan(wl.tiny_graph(), neo.PLAN_FUSE_POOL)["steps"])
    # VGG-16's stem is read by a conv, not a pool
    assert not any(s["kind"] == "conv_pool" for s in _host_plan(wl.vgg16(1), neo.PLAN_FUSE_POOL)["steps"])
    # the fused plan with the stem reading NCHW itself (block 1) and NCHW4c
    g = wl.stem_graph(N=2, H=37, W=41, K=40)
    for sch in ({1: (1, 16)}, {1: (4, 16)}):
        d = _host_plan(g, neo.PLAN_FUSE_POOL, sch)
        assert [s["kind"] for s in d["steps"]].count("conv_pool") == 1


# ---- GPU -------------------------------------------------------------------------------------
CASES = [
    # N, C, H, W, K, R, stride, pad, pool (window, stride, pad)
    (1, 3, 224, 224, 64, 7, 2, 3, (3, 2, 1)),   # ResNet-50's stem
    (2, 3, 37, 41, 40, 7, 2, 3, (3, 2, 1)),     # ragged image and channels, two images
    (1, 4, 20, 18, 16, 3, 1, 1, (2, 2, 0)),
    (1, 1, 29, 17, 33, 5, 2, 2, (3, 2, 0)),
]
IDS = ["resnet50_stem", "ragged_n2", "c4_3x3", "c1_5x5"]


@pytest.fixture(scope="module")
def gpu():
    from gpu_util import torch_cuda
    torch_cuda()
    neo.lib()
    return neo


def _unfused_bits(gpu, p, g, n, monkeypatch):
    """The plan's conv (its folded, packed parameters) through the standalone
    conv with one wave per tile and no split, then the pooling kernel."""
    from gpu_util import dev, host
    c = g.nodes[n]
    C = g.input_shape[1]
    wp, b = p.conv_params(n, c.K, C, c.R, c.S)
    monkeypatch.setenv("NEO_CONV_CONFIG", "1,1,1,1")
    yb = gpu.conv2d_blocked(gpu.to_blocked(dev(g.x)), C, dev(wp), c.K, c.R, c.S, bias=dev(b),
                            stride=c.stride, pad=c.pad, act="relu")
    monkeypatch.delenv("NEO_CONV_CONFIG")
    pn = g.nodes[n + 1]
    pooled = gpu.maxpool2d_blocked(yb, c.K, pn.R, pn.S, pn.stride, pn.pad)
    return host(gpu.from_blocked(pooled, c.K))


@pytest.mark.gpu
@pytest.mark.parametrize("case", CASES, ids=IDS)
@pytest.mark.parametrize("scheme", [None, (1, 16), (4, 16)], ids=["nchw16c", "nchw", "nchw4c"])
def test_fused_stem_pool(gpu, case, scheme, monkeypatch):
    from gpu_util import assert_close, dev, host
    N, C, H, W, K, R, st, pd, pool = case
    g = wl.stem_graph(N=N, C=C, H=H, W=W, K=K, R=R, stride=st, pad=pd, pool=pool)
    p = gpu.Plan(g, flags=gpu.PLAN_FUSE_POOL, schemes={1: scheme} if scheme else None)
    kinds = [s["kind"] for s in p.describe()["steps"]]
    assert "conv_pool" in kinds and "maxpool" not in kinds, kinds
    print(f"\n[conv_pool] {case} scheme {scheme}", flush=True)
    y = host(p.run(dev(g.x)))
    assert_close(y, orc.run_graph(g), f"stem+pool {case}")
    np.testing.assert_array_equal(y, _unfused_bits(gpu, p, g, 1, monkeypatch))
    p.destroy()


CONFIGS = ["1,1,8,2,8", "1,1,10,4,8", "1,1,16,4,12", "1,2,4,2,8", "1,2,5,4,8", "1,2,8,6,8",
           "2,1,8,2,8", "2,1,10,4,8", "2,2,5,4,8", "1,2,5,1,2"]


@pytest.mark.gpu
@pytest.mark.parametrize("cfg", CONFIGS)
def test_every_fused_configuration_is_bit_identical(gpu, cfg, monkeypatch):
    """Every launch configuration of the fused kernel (forced), on the ResNet-50
    stem and on a ragged one, gives the same bits."""
    from gpu_util import dev, host
    for case in (CASES[0], CASES[1]):
        N, C, H, W, K, R, st, pd, pool = case
        g = wl.stem_graph(N=N, C=C, H=H, W=W, K=K, R=R, stride=st, pad=pd, pool=pool)
        monkeypatch.setenv("NEO_CONVPOOL_CONFIG", cfg)
        p = gpu.Plan(g, flags=gpu.PLAN_FUSE_POOL)
        monkeypatch.delenv("NEO_CONVPOOL_CONFIG")
        s = [s for s in p.describe()["steps"] if s["kind"] == "conv_pool"][0]
        want = [int(v) for v in cfg.split(",")]
        got = s["config"]["tile"] + [s["config"]["waves"]] + s["config"]["pooled_tile"]
        if K % (16 * want[0]) and want[0] > 1:      # fk must divide the channel blocks
            assert got != want
            p.destroy()
            continue
        assert got == want, (got, want)
        print(f"\n[conv_pool] forced {cfg} on {case}", flush=True)
        y = host(p.run(dev(g.x)))
        np.testing.assert_array_equal(y, _unfused_bits(gpu, p, g, 1, monkeypatch))
        p.destroy()


@pytest.mark.gpu
def test_tuned_resnet50_with_fused_stem(gpu, tmp_path):
    """ResNet-50 batch 1 with the fused stem, tuned and replayed as a graph:
    the oracle's logits, replays bit-identical, and the keep-or-split choice
    follows the results file, which a later plan reloads."""
    import torch
    from gpu_util import assert_close_network, dev, host, oracle_output
    g = wl.resnet50(1)
    gpu.tune_db_clear()
    fl = gpu.PLAN_FUSE_POOL | gpu.PLAN_TUNE | gpu.PLAN_HIPGRAPH
    p = gpu.Plan(g, flags=fl)
    d = p.describe()
    x = dev(g.x)
    out = torch.empty((1, 1000), device="cuda")
    p.run(x, out)
    y = host(out)
    for _ in range(2):
        out.fill_(0.0)
        p.run(x, out)
        np.testing.assert_array_equal(host(out), y)
    p.destroy()
    assert_close_network(y, oracle_output(g), "resnet50 with the fused stem", graph=g)
    path = tmp_path / "db.txt"
    gpu.tune_db_save(path)
    lines = [l.split() for l in open(path) if l.startswith("convpool ")]
    assert len(lines) == 1
    fused_us = float(lines[0][-1])
    kept = any(s["kind"] == "conv_pool" for s in d["steps"])
    print(f"\nfused stem: {fused_us:.2f} us, kept {kept}")
    gpu.tune_db_clear()
    gpu.tune_db_load(path)
    p2 = gpu.Plan(g, flags=gpu.PLAN_FUSE_POOL | gpu.PLAN_TUNE)
    assert [s["kind"] for s in p2.describe()["steps"]] == [s["kind"] for s in d["steps"]]
    p2.destroy()
