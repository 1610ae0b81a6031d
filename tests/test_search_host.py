"""Host-side checks of the global layout search (Section 3.3.2, Algorithm 2)
in libneo against the oracle's: the optimum of neo_layout_search on seeded
cost tables, the validity of its assignment, and the layouts and transforms
of host-only plans built with explicit schemes."""
import math

import numpy as np
import pytest

from oracle import search as S
from paper_1809_02697_amd import neo
from paper_1809_02697_amd import workloads as wl

import nets

from test_search_oracle import chain_graph, concat_graph, random_tables, residual_graph

NB = len(S.BLOCKS)
assert tuple(neo.SEARCH_BLOCKS) == S.BLOCKS


def _arrays(ct, xt):
    a = np.array(ct, np.float64)
    a[~np.isfinite(a)] = -1.0            # the ABI's "not a candidate"
    return a, np.array(xt, np.float64)


GRAPHS = [("chain", lambda: chain_graph(5, 64, 3)), ("residual", residual_graph),
          ("concat", concat_graph), ("tiny", wl.tiny_graph), ("vgg_tiny", wl.vgg_like_tiny)]


@pytest.mark.parametrize("name,make", GRAPHS)
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_search_matches_oracle_integer_costs(name, make, seed):
    """Integer-valued tables make every sum exact: the optimum must be equal,
    and the library's assignment must cost exactly the optimum under the
    oracle's own accounting."""
    g = make()
    ct, xt = random_tables(g, np.random.default_rng(seed), integer=True, p_drop=0.3)
    best, sch = S.global_search(g, ct, xt)
    cost, got = neo.layout_search(g, *_arrays(ct, xt))
    assert cost == best
    assert S.plan_cost(g, got, ct, xt) == best


@pytest.mark.parametrize("build", [nets.resnet50, nets.vgg16, nets.inception_v3])
def test_search_matches_oracle_on_networks(build):
    g = build()
    for seed in (3, 4):
        ct, xt = random_tables(g, np.random.default_rng(seed), integer=True, p_drop=0.2)
        best, _ = S.global_search(g, ct, xt)
        cost, got = neo.layout_search(g, *_arrays(ct, xt))
        assert cost == best
        assert S.plan_cost(g, got, ct, xt) == best
    # real-valued tables: equal up to summation order
    ct, xt = random_tables(g, np.random.default_rng(5), integer=False, p_drop=0.0)
    best, _ = S.global_search(g, ct, xt)
    cost, got = neo.layout_search(g, *_arrays(ct, xt))
    assert math.isclose(cost, best, rel_tol=1e-12)
    assert math.isclose(S.plan_cost(g, got, ct, xt), best, rel_tol=1e-12)


def test_search_respects_given_schemes_and_block():
    g = nets.resnet50()
    ct, xt = random_tables(g, np.random.default_rng(9), integer=True, p_drop=0.0)
    convs = S.conv_nodes(g)
    fixed = {convs[3]: (32, 32), convs[10]: (16, 64)}
    cost, got = neo.layout_search(g, *_arrays(ct, xt), schemes=fixed)
    for v, s in fixed.items():
        assert got[v] == s
    # the oracle with the same restriction
    ct2 = [[row[:] for row in m] for m in ct]
    for v, (a, b) in fixed.items():
        for i in range(NB):
            for j in range(NB):
                if (S.BLOCKS[i], S.BLOCKS[j]) != (a, b):
                    ct2[v][i][j] = S.INF
    assert cost == S.global_search(g, ct2, xt)[0]
    # default block 32: pools after an NCHW input, concats run in 32
    c32, _ = neo.layout_search(g, *_arrays(ct, xt), block=32)
    assert c32 == S.global_search(g, ct, xt, default_block=32)[0]


def test_search_errors():
    g = chain_graph(2, 32, 2)
    ct = np.full((len(g.nodes), NB, NB), -1.0)
    xt = np.ones((len(g.nodes), NB, NB))
    with pytest.raises(neo.NeoError) as e:
        neo.layout_search(g, ct, xt)                     # no candidate scheme anywhere
    assert e.value.code == -2
    ct[1, 3, 3] = ct[2, 3, 3] = 1.0
    xt[0, 0, 3] = -1.0
    with pytest.raises(neo.NeoError) as e:
        neo.layout_search(g, ct, xt)                     # negative transform time
    assert e.value.code == -1
    xt[0, 0, 3] = 1.0
    assert neo.layout_search(g, ct, xt)[1] == {1: (16, 16), 2: (16, 16)}
    with pytest.raises(neo.NeoError):
        neo.layout_search(g, ct, xt, block=8)


# ---- host-only plans with explicit schemes ------------------------------------------------
def _plan_transforms(g, schemes, block=16):
    p = neo.Plan(g, flags=neo.PLAN_HOST_ONLY, schemes=schemes, block=block)
    d = p.describe()
    p.destroy()
    node_of = {v["id"]: v["node"] for v in d["values"]}
    lay = lambda s: 0 if s == "NCHW" else int(s[4:-1])
    got = sorted((node_of[t["from_value"]], lay(t["from"]), lay(t["to"]), t["alias"])
                 for t in d["transforms"])
    return d, got


def _random_schemes(g, rng, blocks=(16, 32, 64)):
    shapes = S.infer_shapes(g)
    out = {}
    for v in S.conv_nodes(g):
        C, K = shapes[g.nodes[v].inputs[0]][1], g.nodes[v].K
        ics = [1, 4, 16] if C <= 4 else [b for b in blocks if C % b == 0 or b == 16]
        ocs = [b for b in blocks if K % b == 0 or b == 16]
        out[v] = (int(rng.choice(ics)), int(rng.choice(ocs)))
    return out


@pytest.mark.parametrize("build,seed", [(wl.tiny_graph, 0), (wl.tiny_graph, 1),
                                        (wl.vgg_like_tiny, 2), (residual_graph, 3),
                                        (concat_graph, 4), (lambda: nets.resnet50(), 5),
                                        (lambda: nets.inception_v3(), 6)])
def test_plan_layouts_follow_the_search_rules(build, seed):
    """The plan inserts exactly the transforms the oracle's accounting pays
    for (and the aliases it counts as free), for random schemes."""
    g = build()
    if g.nodes[1].w is None:                 # structure-only graphs: give convs weights
        for n in g.nodes:
            if n.op == "conv":
                n.w = np.zeros((n.K, 1, n.R, n.S), np.float32)
        shapes = S.infer_shapes(g)
        for n in g.nodes:
            if n.op == "conv":
                n.w = np.zeros((n.K, shapes[n.inputs[0]][1], n.R, n.S), np.float32)
    sch = _random_schemes(g, np.random.default_rng(seed))
    d, got = _plan_transforms(g, sch)
    want = []
    ct = [[[0.0] * NB for _ in range(NB)] for _ in g.nodes]
    # a conv input block of 1 (NCHW1c) is the default layout, block 0
    S.plan_cost(g, {v: (0 if a == 1 else a, b) for v, (a, b) in sch.items()}, ct, ct,
                transforms=want)
    assert got == sorted(want)
    steps = {s["node"]: s for s in d["steps"] if s["kind"] == "conv"}
    for v, (a, b) in sch.items():
        assert (steps[v]["conv"]["ic_bn"], steps[v]["conv"]["oc_bn"]) == (a, b)


def test_fixed_block_plans():
    """block 32 / 64: every conv in that block; ResNet-50 still has one
    transform in and one (aliased) out."""
    g = nets.resnet50()
    for b in (32, 64):
        d, got = _plan_transforms(g, None, block=b)
        assert [t[1:] for t in got] == sorted([(0, b, False), (b, 0, True)])
        assert all((s["conv"]["ic_bn"], s["conv"]["oc_bn"]) == (b, b)
                   for s in d["steps"] if s["kind"] == "conv")


def test_nchw_stem_needs_no_entry_transform():
    """ResNet-50 with the stem's input block 1: the stem reads the network's
    NCHW input itself, so only the exit transform (an alias) remains."""
    g = nets.resnet50()
    stem = S.conv_nodes(g)[0]
    d, got = _plan_transforms(g, {stem: (1, 16)})
    assert [t[1:] for t in got] == [(16, 0, True)]
    st = next(s for s in d["steps"] if s["kind"] == "conv" and s["node"] == stem)
    assert (st["conv"]["ic_bn"], st["conv"]["oc_bn"]) == (1, 16)
    assert d["values"][st["in"]]["buf"] == -2          # the caller's input buffer


def test_plan_scheme_errors():
    g = wl.tiny_graph()
    with pytest.raises(neo.NeoError) as e:
        neo.Plan(g, flags=neo.PLAN_HOST_ONLY, schemes={1: (16, 0)})
    assert e.value.code == -1
    with pytest.raises(neo.NeoError) as e:
        neo.Plan(g, flags=neo.PLAN_HOST_ONLY, schemes={3: (8, 16)})    # main path: no 8
    assert e.value.code == -4
    with pytest.raises(neo.NeoError) as e:
        neo.Plan(g, flags=neo.PLAN_HOST_ONLY, schemes={3: (16, 4)})    # outputs: 16..64
    assert e.value.code == -4
    with pytest.raises(neo.NeoError) as e:
        neo.Plan(g, flags=neo.PLAN_HOST_ONLY, schemes={3: (1, 16)})    # NCHW input: C <= 4 only
    assert e.value.code == -4
    with pytest.raises(neo.NeoError):
        neo.Plan(g, flags=neo.PLAN_HOST_ONLY | neo.PLAN_GLOBAL_SEARCH)
    with pytest.raises(neo.NeoError):
        neo.Plan(g, flags=neo.PLAN_HOST_ONLY, block=8)
