"""NEO_PLAN_FUSE_CHAINS: a 3x3 conv whose output only a pointwise conv reads,
with that conv (and the second conv of its pair) in one launch, the 3x3's
output kept in LDS and never stored.  Host checks of which convs chain and of
the launch order; GPU parity against the oracle and the unchained plan, tuned
and replayed, with the keep-or-split rule checked against the results file."""
import numpy as np
import pytest

import oracle as orc
from paper_1809_02697_amd import neo
from paper_1809_02697_amd import workloads as wl

import nets
from test_fuse_pairs import _db as _pair_db, _pairs, _shape, _valid_order

CHAINS = neo.PLAN_FUSE_PAIRS | neo.PLAN_FUSE_CHAINS


def _plan(g, flags=CHAINS):
    p = neo.Plan(g, flags=neo.PLAN_HOST_ONLY | flags)
    d = p.describe()
    p.destroy()
    return d


def _chains(g, d):
    return [[g.nodes[m["node"]].name for m in s["members"]] for s in d["steps"] if s["kind"] == "conv_chain"]


def _launched(d):
    return sorted(m["node"] for s in d["steps"]
                  for m in (s["members"] if s["kind"] in ("conv_group", "conv_pair", "conv_chain")
                            else [s] if s["kind"] == "conv" else []))


@pytest.mark.parametrize("flags", [CHAINS, CHAINS | neo.PLAN_GROUP | neo.PLAN_FUSE_GAP])
def test_resnet50_chains_at_the_64_channel_width(flags):
    g = nets.resnet50()
    d = _plan(g, flags)
    assert _chains(g, d) == [["layer1.0.conv2", "layer1.0.conv3", "layer1.1.conv1"],
                             ["layer1.1.conv2", "layer1.1.conv3", "layer1.2.conv1"],
                             ["layer1.2.conv2", "layer1.2.conv3", "layer2.0.conv1"]]
    assert _pairs(g, d) == []                         # every pair became a chain's tail
    assert _launched(d) == sorted(i for i, n in enumerate(g.nodes) if n.op == "conv")
    _valid_order(d)
    for s in d["steps"]:
        if s["kind"] == "conv_chain":
            c, a, b = s["members"]
            assert a["in"] == c["out"] and b["in"] == a["out"]
            assert s["in"] == c["in"] and s["out"] == a["out"] and s["out2"] == b["out"]
            assert s["res"] == a["res"] >= 0          # the bottleneck's residual


def test_chains_without_pairs_take_the_expansion_only():
    g = nets.resnet50()
    d = _plan(g, neo.PLAN_FUSE_CHAINS)
    assert _chains(g, d) == [[f"layer1.{i}.conv2", f"layer1.{i}.conv3"] for i in range(3)]
    assert all(s["out2"] == -1 for s in d["steps"] if s["kind"] == "conv_chain")
    assert _launched(d) == sorted(i for i, n in enumerate(g.nodes) if n.op == "conv")
    _valid_order(d)


@pytest.mark.parametrize("build", [lambda: nets.inception_v3(), lambda: nets.vgg16(), wl.tiny_graph])
def test_no_chains_without_a_kernel_for_them(build):
    assert _chains(build(), _plan(build())) == []


def chain_graph(C0=64, K0=64, Ka=256, Kb=64, N=1, hw=9, stride=1, reread=False, seed=37):
    """x -> c (3x3, C0 -> K0) -> a (1x1, K0 -> Ka, residual from a side conv)
    -> b (1x1, Ka -> Kb), a's output read again later as a residual; with
    `reread` c's output is also read by another conv."""
    bld = wl._Builder("chain", (N, 16, hw, hw), np.random.Generator(np.random.PCG64(seed)))
    x = bld.conv(0, C0, 3, pad=1, name="stem")
    c = bld.conv(x, K0, 3, stride=stride, pad=1, name="c")
    r = bld.conv(x, Ka, 1, stride=stride, act="none", name="side")
    a = bld.conv(c, Ka, 1, residual=r, name="a")
    b = bld.conv(a, Kb, 1, name="b")
    d = bld.conv(b, Ka, 1, residual=a, name="d")
    if reread:
        e = bld.conv(c, Ka, 1, residual=d, name="e")
        d = e
    bld.output(bld.dense(bld.flatten(bld.gap(d), Ka), 10, name="fc"))
    return bld.finish(lambda rng: rng.normal(0, 1, (N, 16, hw, hw)).astype(np.float32))


def test_chain_graph_chains():
    g = chain_graph()
    assert _chains(g, _plan(g)) == [["c", "a", "b"]]
    assert _chains(g, _plan(g, neo.PLAN_FUSE_CHAINS)) == [["c", "a"]]
    assert _chains(g, _plan(g, 0)) == []
    for kw in (dict(C0=80), dict(K0=80), dict(Ka=272), dict(stride=2), dict(reread=True)):
        gg = chain_graph(**kw)                       # no kernel, or the 3x3's output read twice
        assert _chains(gg, _plan(gg)) == [], kw
    gg = chain_graph(Kb=96)                          # no pair kernel: the chain takes a alone
    assert _chains(gg, _plan(gg)) == [["c", "a"]]


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
@pytest.mark.parametrize("C0,K0,Ka,Kb,N,hw,flags", [
    (64, 64, 256, 64, 1, 9, CHAINS), (50, 60, 250, 60, 2, 9, CHAINS), (64, 64, 256, 64, 1, 56, CHAINS),
    (64, 64, 256, 128, 1, 56, CHAINS), (49, 63, 241, 120, 2, 5, CHAINS), (64, 64, 256, 64, 2, 56, CHAINS),
    (64, 64, 256, 64, 1, 9, neo.PLAN_FUSE_CHAINS), (60, 64, 256, 96, 2, 7, CHAINS),
    (64, 64, 256, 64, 1, 1, CHAINS)])
def test_chain_matches_oracle_and_unchained(gneo, C0, K0, Ka, Kb, N, hw, flags):
    """Ragged channel counts inside the kernel's blocks, images whose pixels
    share a 16-pixel tile (81 = 5 * 16 + 1, 25, 49), taps outside the image
    on every border, a 1 x 1 map (every tap but the centre outside), the
    56 x 56 map; the two-conv chain (no pairs, or no pair kernel for 96)."""
    from gpu_util import assert_close, rel_l2
    g = chain_graph(C0, K0, Ka, Kb, N, hw)
    ref = orc.run_graph(g)
    y, d = _run(g, flags)
    ch = [s for s in d["steps"] if s["kind"] == "conv_chain"]
    assert len(ch) == 1
    assert len(ch[0]["members"]) == (3 if flags & neo.PLAN_FUSE_PAIRS and Kb in (64, 128, 120, 60) else 2)
    assert_close(y.reshape(ref.shape), ref, f"chain {C0}->{K0}->{Ka}->{Kb} N={N} {hw}x{hw}")
    y0, _ = _run(g, flags & ~neo.PLAN_FUSE_CHAINS)
    assert rel_l2(y, y0) <= 1e-6


def _chain_db(path):
    out = {}
    for line in open(path).read().splitlines():
        f = line.split()
        if f and f[0] == "chain":
            n = int(f[2])
            ints = [int(v) for v in f[3:3 + 11 * n + 1]]
            out[(tuple(tuple(ints[11 * m:11 * m + 11]) for m in range(n)), ints[-1])] = float(f[-1])
    return out


@pytest.mark.gpu
def test_resnet50_chains_tuned_replayed(gneo, tmp_path):
    """The headline plan's fusions with chains, tuned and replayed: every
    replay equals the first and matches the oracle; a chain is kept exactly
    where the results file says it beats its 3x3 alone plus the best of the
    rest (its pair in one launch, or the pair's convs alone)."""
    from gpu_util import assert_close_network, dev, host, torch_cuda
    torch = torch_cuda()
    neo.tune_db_clear()
    g = wl.resnet50(1)
    ref = orc.run_graph(g)
    flags = neo.PLAN_TUNE | neo.PLAN_GROUP | neo.PLAN_FUSE_GAP | CHAINS
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
    assert_close_network(first, ref, "resnet50 with chains", graph=g)
    path = tmp_path / "db.txt"
    neo.tune_db_save(path)
    convs, pairs = _pair_db(path)
    chains = _chain_db(path)
    d0 = _plan(g, neo.PLAN_GROUP | neo.PLAN_FUSE_GAP | CHAINS)
    kept = {tuple(m["node"] for m in s["members"]) for s in d["steps"] if s["kind"] == "conv_chain"}
    for s in d0["steps"]:
        if s["kind"] != "conv_chain":
            continue
        c, a, b = s["members"]
        res = int(a["res"] >= 0)
        t = chains[((_shape(c["conv"]), _shape(a["conv"]), _shape(b["conv"])), res)]
        alone = convs[_shape(a["conv"])] + convs[_shape(b["conv"])]
        rest = min(pairs[(_shape(a["conv"]), _shape(b["conv"]), res)], alone)
        faster = t < convs[_shape(c["conv"])] + rest
        assert ((c["node"], a["node"], b["node"]) in kept) == faster
    print(f"\n{len(kept)} of 3 chains kept")
