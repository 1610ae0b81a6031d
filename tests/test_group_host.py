"""Host-side checks of horizontal fusion (NEO_PLAN_GROUP): which convs share
a launch (the NCHW16c convs of one round of the list schedule: every step
whose producers ran in earlier rounds), that the launch list stays a valid
order, and that every conv of the network is launched exactly once."""
import numpy as np
import pytest

from paper_1809_02697_amd import neo
from paper_1809_02697_amd import workloads as wl

import nets


def _plan(g, flags=0):
    p = neo.Plan(g, flags=neo.PLAN_HOST_ONLY | neo.PLAN_GROUP | flags)
    d = p.describe()
    p.destroy()
    return d


def _launch_items(d):
    """(step index, reads, writes) per launched conv, pooling or other step."""
    for i, s in enumerate(d["steps"]):
        if s["kind"] == "conv_group":
            for m in s["members"]:
                yield i, [m["in"]] + ([m["res"]] if m["res"] >= 0 else []), m["out"], m
            if "pool" in s:
                yield i, [s["pool"]["in"]], s["pool"]["out"], s["pool"]
        elif s["kind"] == "conv_pair":       # the second conv reads the first's output inside
            a, b = s["members"]
            yield i, [a["in"]] + ([a["res"]] if a["res"] >= 0 else []), a["out"], a
            yield i, [], b["out"], b
        elif s["kind"] == "conv_chain":      # the 3x3's output stays inside, never stored
            c, a = s["members"][:2]
            yield i, [c["in"]], -1, c
            yield i, [a["res"]] if a["res"] >= 0 else [], a["out"], a
            for b in s["members"][2:]:
                yield i, [], b["out"], b
        else:
            yield i, [s["in"]] + ([s["res"]] if s["res"] >= 0 else []), s["out"], s


@pytest.mark.parametrize("build,groups,sizes,pools", [
    (lambda: nets.resnet50(), 4, [2, 2, 2, 2], 0),
    (lambda: nets.inception_v3(), 27, [3, 3, 3, 3, 3, 3, 2, 3, 3, 2, 3, 3, 2, 3, 3, 2, 3, 3, 2, 2, 2,
                                       3, 4, 2, 3, 4, 2], 11),
    (wl.tiny_graph, 2, [2, 2], 1),
    (lambda: nets.vgg16(), 0, [], 0)])
def test_group_structure(build, groups, sizes, pools):
    g = build()
    d = _plan(g)
    grp = [s for s in d["steps"] if s["kind"] == "conv_group"]
    assert len(grp) == groups
    if sizes is not None:
        assert [len(s["members"]) for s in grp] == sizes
    assert sum(1 for s in grp if "pool" in s) == pools
    # every pooling node runs exactly once, alone or in a conv launch
    pooled = sorted([s["pool"]["node"] for s in grp if "pool" in s] +
                    [s["node"] for s in d["steps"] if s["kind"] in ("maxpool", "avgpool")])
    assert pooled == sorted(i for i, n in enumerate(g.nodes) if n.op in ("maxpool", "avgpool"))
    conv_nodes = sorted(i for i, n in enumerate(g.nodes) if n.op == "conv")
    launched = sorted(m["node"] for s in d["steps"] if s["kind"] in ("conv", "conv_group")
                      for m in (s["members"] if s["kind"] == "conv_group" else [s]))
    assert launched == conv_nodes
    for s in grp:
        assert all((m["conv"]["tile"], m["conv"]["waves"]) == (s["tile"], s["waves"])
                   for m in s["members"])
        assert all(m["conv"]["split"] == 1 and m["conv"]["ic_bn"] == 16 and m["conv"]["oc_bn"] == 16
                   for m in s["members"])


@pytest.mark.parametrize("build", [lambda: nets.resnet50(), lambda: nets.inception_v3(),
                                   wl.tiny_graph])
def test_grouped_launch_list_is_a_valid_order(build):
    """Every value a step reads is the network input or was written by an
    earlier step (the members of a group are independent, so never by the
    same step)."""
    g = build()
    d = _plan(g)
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
            written[root[out]] = i
    # a concatenation has no step: it is complete once its inputs (written
    # into slices of its buffer) are; nested concats first (node order)
    for c, n in enumerate(g.nodes):
        if n.op != "concat":
            continue
        cv = [v for v in vals if v["node"] == c][0]
        parts = [written.get(root[u["id"]], 1 << 30) for u in vals
                 if u["node"] in n.inputs and u["view"] and u["buf"] == cv["buf"]]
        written[root[cv["id"]]] = max(parts)
    for i, reads, _, item in _launch_items(d):
        for r in reads:
            rr = root[r]
            if vals[rr]["buf"] == -2:                # the network input
                continue
            assert written.get(rr, 1 << 30) < i, (i, item.get("node"), r)


def _names(g, d):
    """Per launch: the node name of a single step, or the names of a fused
    launch's convs followed by its pooling step's."""
    return [[g.nodes[m["node"]].name for m in s["members"]] +
            ([g.nodes[s["pool"]["node"]].name] if "pool" in s else [])
            if s["kind"] == "conv_group" else g.nodes[s["node"]].name for s in d["steps"]]


def _first(names, name):
    return next(i for i, n in enumerate(names) if n == name or (isinstance(n, list) and name in n))


def test_parallel_branches_share_launches():
    """Inception's first module: the three 1x1 convs that read the module's
    input, and the module's average pool, form round one (the pool runs in
    the convs' launch); the second convs of two branches and the pooling
    branch's 1x1 (three different inputs) form round two; the last conv of
    the double-3x3 branch runs alone."""
    g = nets.inception_v3()
    names = _names(g, _plan(g))
    i = _first(names, "Mixed_5b.branch1x1")
    assert names[i:i + 3] == [
        ["Mixed_5b.branch1x1", "Mixed_5b.branch5x5_1", "Mixed_5b.branch3x3dbl_1", "Mixed_5b.avgpool"],
        ["Mixed_5b.branch5x5_2", "Mixed_5b.branch3x3dbl_2", "Mixed_5b.branch_pool"],
        "Mixed_5b.branch3x3dbl_3"]
    # a 7x7-factorised module: five launches instead of eleven
    i = _first(names, "Mixed_6b.branch1x1")
    assert names[i:i + 5] == [
        ["Mixed_6b.branch1x1", "Mixed_6b.branch7x7_1", "Mixed_6b.branch7x7dbl_1", "Mixed_6b.avgpool"],
        ["Mixed_6b.branch7x7_2", "Mixed_6b.branch7x7dbl_2", "Mixed_6b.branch_pool"],
        ["Mixed_6b.branch7x7_3", "Mixed_6b.branch7x7dbl_3"],
        "Mixed_6b.branch7x7dbl_4", "Mixed_6b.branch7x7dbl_5"]
    # a reduction module: the max pool rides with the two branch heads
    i = _first(names, "Mixed_6a.branch3x3")
    assert names[i] == ["Mixed_6a.branch3x3", "Mixed_6a.branch3x3dbl_1", "Mixed_6a.maxpool"]


def test_pools_alone_when_asked(monkeypatch):
    """NEO_GROUP_POOLS=0 keeps every pooling step in a launch of its own,
    ahead of its round's conv launches."""
    monkeypatch.setenv("NEO_GROUP_POOLS", "0")
    g = nets.inception_v3()
    d = _plan(g)
    assert not any("pool" in s for s in d["steps"] if s["kind"] == "conv_group")
    names = _names(g, d)
    i = names.index("Mixed_5b.avgpool")
    assert names[i + 1] == ["Mixed_5b.branch1x1", "Mixed_5b.branch5x5_1", "Mixed_5b.branch3x3dbl_1"]


def test_ungrouped_plan_keeps_node_order():
    g = nets.inception_v3()
    d = neo.Plan(g, flags=neo.PLAN_HOST_ONLY)
    names = [n for n in _names(g, d.describe()) if not isinstance(n, list)]
    d.destroy()
    assert names.index("Mixed_5b.branch3x3dbl_3") < names.index("Mixed_5b.branch_pool")


def test_group_config_override(monkeypatch):
    g = nets.resnet50()
    monkeypatch.setenv("NEO_GROUP_CONFIG", "2,1,1")
    d = _plan(g)
    assert all((s["tile"], s["waves"]) == ([2, 1], 1) for s in d["steps"] if s["kind"] == "conv_group")
    monkeypatch.setenv("NEO_GROUP_CONFIG", "4,4,16")     # not valid for these groups: ignored
    d = _plan(g)
    assert all(s["waves"] != 16 for s in d["steps"] if s["kind"] == "conv_group")


def concat_residual_graph():
    """x read by three convs; the third adds the concatenation of the first
    two as its residual, so it must not join their launch."""
    b = wl._Builder("catres", (1, 16, 9, 9), np.random.Generator(np.random.PCG64(5)))
    x = b.conv(0, 32, 3, pad=1, name="stem")
    c1 = b.conv(x, 16, 1, name="c1")
    c2 = b.conv(x, 16, 3, pad=1, name="c2")
    cat = b.concat([c1, c2], name="cat")
    a = b.conv(x, 32, 1, residual=cat, name="a")
    b.output(a)
    return b.finish(lambda rng: rng.normal(0, 1, (1, 16, 9, 9)).astype(np.float32))


def test_concat_residual_keeps_its_conv_out_of_the_group():
    g = concat_residual_graph()
    d = _plan(g)
    grp = [s for s in d["steps"] if s["kind"] == "conv_group"]
    assert len(grp) == 1
    assert sorted(m["node"] for m in grp[0]["members"]) == [2, 3]
    names = [g.nodes[s["node"]].name for s in d["steps"] if s["kind"] == "conv"]
    assert "a" in names
