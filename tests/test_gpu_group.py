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
    assert_close_network(y.reshape(ref.shape), ref, g.name, graph=g)
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
    assert_close_network(eager.reshape(ref.shape), ref, "tuned grouped resnet50", graph=g)
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
    """From a saved results file: {conv shape: us} (NCHW16c convs), {(member
    shapes, pool shape or None): us} and {pool shape: us}; conv shape = N C H
    W K R S sh sw ph pw, pool shape = max N C H W R S sh sw ph pw xb."""
    convs, groups, pools = {}, {}, {}
    for line in open(path).read().splitlines():
        f = line.split()
        if not f or f[0].startswith("#"):
            continue
        if f[0] == "group":
            n, m = int(f[2]), int(f[3])
            ints = [int(v) for v in f[4:4 + 11 * n + 12 * m]]
            mem = tuple(tuple(ints[11 * i:11 * i + 11]) for i in range(n))
            groups[(mem, tuple(ints[11 * n:]) if m else None)] = float(f[-1])
        elif f[0] == "pool":
            pools[tuple(int(v) for v in f[2:14])] = float(f[-1])
        elif f[13:15] == ["16", "16"] and f[12] == "1":
            convs[tuple(int(v) for v in f[1:12])] = float(f[-1])
    return convs, groups, pools


def _shape(c):
    return (c["N"], c["C"], c["H"], c["W"], c["K"], c["R"], c["S"], c["stride"][0], c["stride"][1],
            c["pad"][0], c["pad"][1])


def _pool_shape(g, d, p):
    n = g.nodes[p["node"]]
    v = d["values"][p["in"]]
    N, C, H, W = v["shape"]
    return (1 if p["kind"] == "maxpool" else 0, N, C, H, W, n.R, n.S, n.stride[0], n.stride[1],
            n.pad[0], n.pad[1], int(v["layout"][4:-1]))


def _expected_launches(g, d0, convs, groups, pools):
    """The launch list the keep-or-split rule makes of the untuned plan d0:
    a fused launch (convs and pool) stays when it beats the members' and the
    pool's own launches and, with more than one conv, the convs fused with
    the pool alone; otherwise the cheaper of the two."""
    out = []
    for s in d0["steps"]:
        if s["kind"] != "conv_group":
            out.append((s["kind"], s["node"]))
            continue
        mem = tuple(_shape(m["conv"]) for m in s["members"])
        pool = _pool_shape(g, d0, s["pool"]) if "pool" in s else None
        pool_us = pools[pool] if pool else 0.0
        alone = sum(convs[k] for k in mem) + pool_us
        fused = groups[(mem, pool)]
        split = groups[(mem, None)] + pool_us if pool and len(mem) > 1 else None
        nodes = tuple(m["node"] for m in s["members"])
        if fused < alone and (split is None or fused <= split):
            out.append(("conv_group", nodes, s["pool"]["node"] if pool else None))
        elif split is not None and split < alone:
            out += [(s["pool"]["kind"], s["pool"]["node"]), ("conv_group", nodes, None)]
        else:
            out += ([(s["pool"]["kind"], s["pool"]["node"])] if pool else []) + \
                   [("conv", m["node"]) for m in s["members"]]
    return out


def _launches(d):
    return [("conv_group", tuple(m["node"] for m in s["members"]),
             s["pool"]["node"] if "pool" in s else None) if s["kind"] == "conv_group"
            else (s["kind"], s["node"]) for s in d["steps"]]


def test_tuned_inception_keeps_only_faster_launches(neo, tmp_path):
    """With NEO_PLAN_TUNE every fused launch (convs, and a pooling step
    riding along) is kept, split from its pool, or split into single
    launches by the measured times in the results database; the tuned plan
    matches the oracle, and a plan rebuilt from the saved file in a clean
    database is the same launch list."""
    neo.tune_db_clear()
    g = wl.inception_v3(1)
    ref = orc.run_graph(g)
    p0 = neo.Plan(g, flags=neo.PLAN_GROUP)
    d0 = p0.describe()
    p0.destroy()
    y, d = _run(neo, g, neo.PLAN_GROUP | neo.PLAN_TUNE)
    assert_close_network(y.reshape(ref.shape), ref, "tuned grouped inception", graph=g)
    path = tmp_path / "db.txt"
    neo.tune_db_save(path)
    convs, groups, pools = _db_times(path)
    assert _launches(d) == _expected_launches(g, d0, convs, groups, pools)
    kept = sum(1 for s in d["steps"] if s["kind"] == "conv_group")
    print(f"\n{kept} fused launches kept, {sum(1 for s in d['steps'] if 'pool' in s)} with a pool")
    neo.tune_db_clear()
    neo.tune_db_load(path)
    _, d2 = _run(neo, g, neo.PLAN_GROUP | neo.PLAN_TUNE)
    strip = lambda d: [(s["kind"], s["node"], s.get("tile"), s.get("waves"), s.get("pool", {}).get("node"),
                        s.get("conv", {}).get("tile")) for s in d["steps"]]
    assert strip(d2) == strip(d)


def pool_graph(seed=13, N=2):
    """Pooling steps that share a round with convs: a 3x3/s1/p1 average pool
    next to two branch heads (3x3 convs over 256 channels, so every wave
    count up to 16 is a valid configuration for them), a 2x2/s2 max pool (the generic window path)
    next to two convs of different inputs, and a 3x3/s2 average pool over a
    ragged channel count (40) next to two more; a second pool in the first
    round (a 3x3/s2 max pool writing into a concatenation) runs alone."""
    b = wl._Builder("pools", (N, 24, 15, 13), np.random.Generator(np.random.PCG64(seed)))
    x = b.conv(0, 256, 3, pad=1, name="stem")
    a1 = b.conv(x, 32, 3, stride=2, name="a1")
    a2 = b.conv(x, 16, 3, pad=1, name="a2")
    ap = b.pool("avgpool", x, 3, 1, pad=1, name="ap")
    mp = b.pool("maxpool", x, 3, 2, name="mp")
    a3 = b.conv(a2, 32, 3, stride=2, name="a3")
    ap2 = b.conv(ap, 32, 1, name="ap2")
    m2 = b.pool("maxpool", ap2, 2, 2, name="m2")
    c1 = b.conv(ap2, 40, 3, pad=1, name="c1")
    cat = b.concat([a1, mp, a3], name="cat")
    z = b.conv(cat, 16, 1, name="z")
    q = b.pool("avgpool", c1, 3, 2, name="q")
    c2 = b.conv(c1, 16, 1, name="c2")
    c3 = b.conv(c1, 16, 3, stride=2, name="c3")
    s = b.concat([b.gap(z), b.gap(m2), b.gap(q), b.gap(c2), b.gap(c3)], name="cat2")
    s = b.flatten(s, 16 + 32 + 40 + 16 + 16)
    b.output(b.dense(s, 10, name="fc"))
    return b.finish(lambda rng: rng.normal(0, 1, (N, 24, 15, 13)).astype(np.float32))


@pytest.mark.parametrize("cfg", [(1, 1, 1), (1, 1, 2), (1, 2, 4), (1, 1, 16), (2, 1, 2)],
                         ids=lambda c: "fk%dfp%dw%d" % c)
def test_pools_ride_bit_identical(neo, cfg, monkeypatch):
    """A pooling step run by a fused conv launch gives the same bits as in a
    launch of its own, for workgroups of 64 to 1024 threads."""
    monkeypatch.setenv("NEO_GROUP_CONFIG", "%d,%d,%d" % cfg)
    g = pool_graph()
    ref = orc.run_graph(g)
    y, d = _run(neo, g, neo.PLAN_GROUP)
    assert sum(1 for s in d["steps"] if "pool" in s) == 3
    assert_close(y.reshape(ref.shape), ref, f"pools ride {cfg}")
    monkeypatch.setenv("NEO_GROUP_POOLS", "0")
    y0, d0 = _run(neo, g, neo.PLAN_GROUP)
    assert not any("pool" in s for s in d0["steps"])
    np.testing.assert_array_equal(y, y0)


def test_pool_rides_with_a_lone_conv(neo):
    """A round of one conv and one pooling step becomes a one-conv fused
    launch carrying the pool."""
    b = wl._Builder("lone", (1, 32, 11, 9), np.random.Generator(np.random.PCG64(17)))
    x = b.conv(0, 48, 3, pad=1, name="stem")
    a = b.conv(x, 24, 3, stride=2, name="a")
    m = b.pool("maxpool", x, 3, 2, name="m")
    s = b.concat([b.gap(a), b.gap(m)], name="cat")
    s = b.flatten(s, 24 + 48)
    b.output(b.dense(s, 10, name="fc"))
    g = b.finish(lambda rng: rng.normal(0, 1, (1, 32, 11, 9)).astype(np.float32))
    ref = orc.run_graph(g)
    y, d = _run(neo, g, neo.PLAN_GROUP)
    grp = [s for s in d["steps"] if s["kind"] == "conv_group"]
    assert len(grp) == 1 and len(grp[0]["members"]) == 1 and "pool" in grp[0]
    assert_close(y.reshape(ref.shape), ref, "lone conv with pool")


@pytest.mark.parametrize("builder", [wl.tiny_graph, lambda: wl.inception_v3(1)])
def test_pools_ride_network_bit_identical(neo, builder, monkeypatch):
    g = builder()
    y, d = _run(neo, g, neo.PLAN_GROUP)
    assert any("pool" in s for s in d["steps"])
    monkeypatch.setenv("NEO_GROUP_POOLS", "0")
    y0, _ = _run(neo, g, neo.PLAN_GROUP)
    np.testing.assert_array_equal(y, y0)


def test_concat_residual_group_matches_oracle(neo):
    from test_group_host import concat_residual_graph
    g = concat_residual_graph()
    ref = orc.run_graph(g)
    y, d = _run(neo, g, neo.PLAN_GROUP)
    assert any(s["kind"] == "conv_group" for s in d["steps"])
    assert_close(y.reshape(ref.shape), ref, "concat residual")



def tiny_members_graph(seed=12):
    """Siblings on a 2x3 map of one image: members of one to three workgroups
    (fewer than one per XCD) beside a member of up to 19, so most of each
    small member's padded range exits at once."""
    b = wl._Builder("tiny_members", (1, 40, 2, 3), np.random.Generator(np.random.PCG64(seed)))
    x = b.conv(0, 256, 1, name="stem")
    a1 = b.conv(x, 32, 1, name="a1")                 # 1 pixel tile x 2 channel tiles
    a2 = b.conv(x, 48, 3, pad=1, name="a2")          # 3 channel tiles
    a3 = b.conv(x, 304, 1, name="a3")                # 19 channel tiles
    y = b.concat([a1, a2, a3], name="cat")
    y = b.gap(y)
    y = b.flatten(y, 384)
    b.output(b.dense(y, 10, name="fc"))
    return b.finish(lambda rng: rng.normal(0, 1, (1, 40, 2, 3)).astype(np.float32))


TINY_CFGS = [(1, 1, 1), (1, 1, 4), (2, 1, 1), (2, 1, 4), (2, 1, 8)]


@pytest.mark.parametrize("cfg", TINY_CFGS, ids=[f"fk{c[0]}fp{c[1]}w{c[2]}" for c in TINY_CFGS])
def test_group_members_smaller_than_xcd_count(neo, cfg, monkeypatch):
    """Each member of a fused launch takes whole rounds over the XCDs; members
    with fewer workgroups than XCDs leave the rest of their range idle.  The
    fused launch runs in the forced configuration and matches the oracle."""
    monkeypatch.setenv("NEO_GROUP_CONFIG", "%d,%d,%d" % cfg)
    g = tiny_members_graph()
    ref = orc.run_graph(g)
    y, d = _run(neo, g, neo.PLAN_GROUP)
    grp = [s for s in d["steps"] if s["kind"] == "conv_group"]
    assert len(grp) == 1 and len(grp[0]["members"]) == 3
    assert grp[0]["tile"] == [cfg[0], cfg[1]] and grp[0]["waves"] == cfg[2]
    assert_close(y.reshape(ref.shape), ref, f"tiny members {cfg}")
