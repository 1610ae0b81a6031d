"""GPU parity of horizontally fused launches (NEO_PLAN_GROUP): the NCHW16c
convs of one round of the list schedule (siblings of one value, and the
parallel branches of a module) run as one launch with a shared launch
configuration.  Checked against the oracle for every configuration the group
kernel instantiates, on the three networks, tuned, and under graph replay."""
import numpy as np
import pytest

import oracle as orc
from paper_1809_02697_amd import workloads as wl

from gpu_util import assert_close, assert_close_network, dev, host, rel_l2, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def neo():
    torch_cuda()
    from paper_1809_02697_amd import neo as n
    n.lib()
    return n


def sibling_graph(seed=11, N=2):
    """One value read by four convs of different shapes (1x1, 3x3/s1, 5x5,
    1x7; ragged K), one of them with a residual; their outputs concatenated
    and reduced by a final conv; a second group further down."""
    b = wl._Builder("siblings", (N, 48, 13, 11), np.random.Generator(np.random.PCG64(seed)))
    x = b.conv(0, 64, 3, pad=1, name="stem")
    r = b.conv(x, 40, 1, act="none", name="res_src")
    a1 = b.conv(x, 40, 1, residual=r, name="a1")
    a2 = b.conv(x, 24, 3, pad=1, name="a2")
    a3 = b.conv(x, 56, 5, pad=2, name="a3")
    a4 = b.conv(x, 20, 1, 7, pad=(0, 3), name="a4")
    y = b.concat([a1, a2, a3], name="cat")
    z = b.conv(a4, 32, 3, pad=1, name="z")
    p = b.conv(y, 33, 1, name="p1")
    q = b.conv(y, 16, 3, stride=2, pad=1, name="p2")
    w = b.conv(z, 16, 3, stride=2, pad=1, name="p3")
    s = b.concat([q, w], name="cat2")
    s = b.gap(s)
    s = b.flatten(s, 32)
    b.output(b.dense(s, 10, name="fc"))
    del p
    return b.finish(lambda rng: rng.normal(0, 1, (N, 48, 13, 11)).astype(np.float32))


def _run(neo, g, flags=0):
    p = neo.Plan(g, flags=flags)
    d = p.describe()
    y = host(p.run(dev(g.x)))
    p.destroy()
    return y, d


GROUP_CFGS = [(fk, fp, wv) for fk in (1, 2, 4) for fp in (1, 2, 4) for wv in (1, 2, 4, 8, 16)
              if wv <= 4 or (wv == 8 and fk * fp <= 4) or (wv == 16 and fk * fp <= 2)]


@pytest.mark.parametrize("cfg", GROUP_CFGS, ids=[f"fk{c[0]}fp{c[1]}w{c[2]}" for c in GROUP_CFGS])
def test_group_every_launch_config(neo, cfg, monkeypatch):
    monkeypatch.setenv("NEO_GROUP_CONFIG", "%d,%d,%d" % cfg)
    g = sibling_graph()
    ref = orc.run_graph(g)
    y, d = _run(neo, g, neo.PLAN_GROUP)
    grp = [s for s in d["steps"] if s["kind"] == "conv_group"]
    assert len(grp) >= 2
    assert_close(y.reshape(ref.shape), ref, f"group {cfg}")


@pytest.mark.parametrize("builder", [wl.tiny_graph, lambda: wl.resnet50(1),
                                     lambda: wl.inception_v3(1)])
def test_grouped_network_matches_oracle(neo, builder):
    g = builder()
    ref = orc.run_graph(g)
    y, d = _run(neo, g, neo.PLAN_GROUP)
    assert any(s["kind"] == "conv_group" for s in d["steps"])
    assert_close_network(y.reshape(ref.shape), ref, g.name)
    y0, _ = _run(neo, g)
    assert rel_l2(y, y0) <= 1e-5


def test_tuned_grouped_resnet50_graph_replay(neo):
    """Tuned groups (each group's configuration searched as one launch) under
    graph replay: every replay equals the eager result and the oracle."""
    torch = torch_cuda()
    g = wl.resnet50(1)
    ref = orc.run_graph(g)
    p = neo.Plan(g, flags=neo.PLAN_GROUP | neo.PLAN_TUNE)
    x = dev(g.x)
    eager = host(p.run(x))
    p.destroy()
    assert_close_network(eager.reshape(ref.shape), ref, "tuned grouped resnet50")
    p = neo.Plan(g, flags=neo.PLAN_GROUP | neo.PLAN_TUNE | neo.PLAN_HIPGRAPH)
    d = p.describe()
    assert all(s["tuned"] for s in d["steps"] if s["kind"] == "conv_group")
    out = torch.empty((1, 1000), device="cuda")
    for _ in range(3):
        out.fill_(-1.0)
        p.run(x, out)
        torch.ones(1000, device="cuda").sum()
        np.testing.assert_array_equal(host(out), eager)
    p.destroy()


def _db_times(path):
    """{conv shape: us} and {tuple of member shapes: us} from a saved results
    file (shape = N C H W K R S sh sw ph pw)."""
    convs, groups = {}, {}
    for line in open(path).read().splitlines():
        f = line.split()
        if not f or f[0].startswith("#"):
            continue
        if f[0] == "group":
            n = int(f[2])
            ints = tuple(int(v) for v in f[3:3 + 11 * n])
            groups[tuple(ints[11 * i:11 * i + 11] for i in range(n))] = float(f[-1])
        elif f[13:15] == ["16", "16"] and f[12] == "1":
            convs[tuple(int(v) for v in f[1:12])] = float(f[-1])
    return convs, groups


def _shape(c):
    return (c["N"], c["C"], c["H"], c["W"], c["K"], c["R"], c["S"], c["stride"][0], c["stride"][1],
            c["pad"][0], c["pad"][1])


def test_tuned_inception_keeps_only_faster_groups(neo, tmp_path):
    """With NEO_PLAN_TUNE a fused launch stays only where its measured time
    is below the sum of its members' own best times; the tuned plan matches
    the oracle, and a plan rebuilt from the saved results file in a clean
    database is the same launch list."""
    neo.tune_db_clear()
    g = wl.inception_v3(1)
    ref = orc.run_graph(g)
    y, d = _run(neo, g, neo.PLAN_GROUP | neo.PLAN_TUNE)
    assert_close_network(y.reshape(ref.shape), ref, "tuned grouped inception")
    path = tmp_path / "db.txt"
    neo.tune_db_save(path)
    convs, groups = _db_times(path)
    kept = set()
    for s in d["steps"]:
        if s["kind"] != "conv_group":
            continue
        key = tuple(_shape(m["conv"]) for m in s["members"])
        kept.add(key)
        assert groups[key] < sum(convs[k] for k in key)
    for key, us in groups.items():
        if key not in kept:
            assert us >= sum(convs[k] for k in key)
    print(f"\n{len(kept)} of {len(groups)} tuned groups kept")
    neo.tune_db_clear()
    neo.tune_db_load(path)
    _, d2 = _run(neo, g, neo.PLAN_GROUP | neo.PLAN_TUNE)
    strip = lambda d: [(s["kind"], s["node"], s.get("tile"), s.get("waves"),
                        s.get("conv", {}).get("tile")) for s in d["steps"]]
    assert strip(d2) == strip(d)


def test_concat_residual_group_matches_oracle(neo):
    from test_group_host import concat_residual_graph
    g = concat_residual_graph()
    ref = orc.run_graph(g)
    y, d = _run(neo, g, neo.PLAN_GROUP)
    assert any(s["kind"] == "conv_group" for s in d["steps"])
    assert_close(y.reshape(ref.shape), ref, "concat residual")
