"""NEO_PLAN_FUSE_PAIRS: a pointwise conv and a later pointwise conv reading
its output in one launch (the first output kept in LDS per 16 pixels and
still stored).  Host checks of which convs pair and of the launch order; GPU
parity against the oracle and the unpaired plan, tuned and replayed."""
import numpy as np
import pytest

import oracle as orc
from paper_1809_02697_amd import neo
from paper_1809_02697_amd import workloads as wl

import nets
from test_group_host import _launch_items


def _plan(g, flags=0):
    p = neo.Plan(g, flags=neo.PLAN_HOST_ONLY | neo.PLAN_FUSE_PAIRS | flags)
    d = p.describe()
    p.destroy()
    return d


def _pairs(g, d):
    return [[g.nodes[m["node"]].name for m in s["members"]] for s in d["steps"] if s["kind"] == "conv_pair"]


def _valid_order(d):
    vals = d["values"]
    root = {}
    for v in vals:
        r = v["id"]
        while vals[r]["alias_of"] >= 0:
            r = vals[r]["alias_of"]
        root[v["id"]] = r
    written = {}
    for i, _, out, _ in _launch_items(d):
        if out >= 0:
            written.setdefault(root[out], i)
    for i, reads, _, item in _launch_items(d):
        for r in reads:
            if vals[root[r]]["buf"] != -2:
                assert written.get(root[r], 1 << 30) < i, (i, item.get("node"), r)


@pytest.mark.parametrize("flags", [0, neo.PLAN_GROUP | neo.PLAN_FUSE_GAP])
def test_resnet50_pairs_at_the_64_channel_width(flags):
    g = nets.resnet50()
    d = _plan(g, flags)
    assert _pairs(g, d) == [["layer1.0.conv3", "layer1.1.conv1"], ["layer1.1.conv3", "layer1.2.conv1"],
                            ["layer1.2.conv3", "layer2.0.conv1"]]
    launched = sorted(m["node"] for s in d["steps"]
                      for m in (s["members"] if s["kind"] in ("conv_group", "conv_pair")
                                else [s] if s["kind"] == "conv" else []))
    assert launched == sorted(i for i, n in enumerate(g.nodes) if n.op == "conv")
    _valid_order(d)
    for s in d["steps"]:
        if s["kind"] == "conv_pair":
            a, b = s["members"]
            assert b["in"] == a["out"] and s["out"] == a["out"] and s["out2"] == b["out"]


@pytest.mark.parametrize("build", [lambda: nets.inception_v3(), lambda: nets.vgg16(), wl.tiny_graph])
def test_no_pairs_without_a_kernel_for_them(build):
    assert _pairs(build(), _plan(build())) == []


def pair_graph(Ca=64, Ka=256, Kb=64, N=1, hw=9, seed=31):
    """x -> a (1x1, Ca -> Ka, residual from a side conv) -> b (1x1, Ka -> Kb),
    a's output also read later as a residual."""
    b = wl._Builder("pair", (N, 16, hw, hw), np.random.Generator(np.random.PCG64(seed)))
    x = b.conv(0, Ca, 3, pad=1, name="stem")
    r = b.conv(x, Ka, 1, act="none", name="side")
    a = b.conv(x, Ka, 1, residual=r, name="a")
    c = b.conv(a, Kb, 1, name="b")
    d = b.conv(c, Ka, 1, residual=a, name="d")
    b.output(b.dense(b.flatten(b.gap(d), Ka), 10, name="fc"))
    return b.finish(lambda rng: rng.normal(0, 1, (N, 16, hw, hw)).astype(np.float32))


def test_pair_graph_pairs():
    g = pair_graph()
    assert _pairs(g, _plan(g)) == [["a", "b"]]
    assert _pairs(pair_graph(Ca=80), _plan(pair_graph(Ca=80))) == []   # no kernel for 80 -> 256
    assert _pairs(pair_graph(Kb=96), _plan(pair_graph(Kb=96))) == []   # nor for 256 -> 96


# ---- GPU ---------------------------------------------------------------------------------
@pytest.fixture(scope="module")
def gneo():
    from gpu_util import torch_cuda
    torch_cuda()
    neo.lib()
    return neo


def _run(g, flags):
    from gpu_util import dev, host
    p = neo.Plan(g, flags=flags)
    d = p.describe()
    y = host(p.run(dev(g.x)))
    p.destroy()
    return y, d


@pytest.mark.gpu
@pytest.mark.parametrize("Ca,Ka,Kb,N,hw", [(64, 256, 64, 1, 9), (50, 250, 60, 2, 9),
                                           (64, 256, 64, 2, 56), (49, 241, 49, 1, 5),
                                           (64, 256, 128, 1, 56), (50, 250, 120, 2, 9)])
def test_pair_matches_oracle_and_unpaired(gneo, Ca, Ka, Kb, N, hw):
    """Ragged channel counts inside the kernel's blocks, two images whose
    pixels share a 16-pixel tile (81 = 5 * 16 + 1), the 56 x 56 map."""
    from gpu_util import assert_close, rel_l2
    g = pair_graph(Ca, Ka, Kb, N, hw)
    ref = orc.run_graph(g)
    y, d = _run(g, neo.PLAN_FUSE_PAIRS)
    assert any(s["kind"] == "conv_pair" for s in d["steps"])
    assert_close(y.reshape(ref.shape), ref, f"pair {Ca}->{Ka}->{Kb} N={N} {hw}x{hw}")
    y0, _ = _run(g, 0)
    assert rel_l2(y, y0) <= 1e-6


def _db(path):
    convs, pairs = {}, {}
    for line in open(path).read().splitlines():
        f = line.split()
        if not f or f[0].startswith("#"):
            continue
        if f[0] == "pair":
            ints = tuple(int(v) for v in f[2:25])
            pairs[(ints[:11], ints[11:22], ints[22])] = float(f[-1])
        elif f[0] not in ("group", "pool") and f[13:15] == ["16", "16"] and f[12] == "1":
            convs[tuple(int(v) for v in f[1:12])] = float(f[-1])
    return convs, pairs


def _shape(c):
    return (c["N"], c["C"], c["H"], c["W"], c["K"], c["R"], c["S"], c["stride"][0], c["stride"][1],
            c["pad"][0], c["pad"][1])


@pytest.mark.gpu
def test_resnet50_pairs_tuned_replayed(gneo, tmp_path):
    """All of the headline plan's fusions, tuned and replayed: every replay
    equals the first and matches the oracle; a pair is kept exactly where the
    results file says it beats its two convs alone."""
    from gpu_util import assert_close_network, dev, host, torch_cuda
    torch = torch_cuda()
    neo.tune_db_clear()
    g = wl.resnet50(1)
    ref = orc.run_graph(g)
    flags = neo.PLAN_TUNE | neo.PLAN_GROUP | neo.PLAN_FUSE_GAP | neo.PLAN_FUSE_PAIRS
    p = neo.Plan(g, flags=flags | neo.PLAN_HIPGRAPH)
    d = p.describe()
    x = dev(g.x)
    out = torch.empty((1, 1000), device="cuda")
    first = None
    for _ in range(3):
        out.fill_(-1.0)
        p.run(x, out)
        torch.ones(1000, device="cuda").sum()
        y = host(out)
        first = y if first is None else first
        np.testing.assert_array_equal(y, first)
    p.destroy()
    assert_close_network(first, ref, "resnet50 with pairs", graph=g)
    path = tmp_path / "db.txt"
    neo.tune_db_save(path)
    convs, pairs = _db(path)
    d0 = _plan(g, neo.PLAN_GROUP | neo.PLAN_FUSE_GAP)
    kept = {tuple(m["node"] for m in s["members"]) for s in d["steps"] if s["kind"] == "conv_pair"}
    for s in d0["steps"]:
        if s["kind"] != "conv_pair":
            continue
        a, b = s["members"]
        t = pairs[(_shape(a["conv"]), _shape(b["conv"]), int(a["res"] >= 0))]
        faster = t < convs[_shape(a["conv"])] + convs[_shape(b["conv"])]
        assert ((a["node"], b["node"]) in kept) == faster
    print(f"\n{len(kept)} of 3 pairs kept")
