"""Pins of the oracle's global layout search (Section 3.3.2, Algorithm 2):
the paper's printed candidate list, a hand-worked chain, brute force over
every assignment on small graphs, and the chain form of the recurrence."""
import math
import os

import numpy as np
import pytest

from oracle import search as S
from paper_1809_02697_amd import workloads as wl

import nets

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
NB = len(S.BLOCKS)


def _read_golden(name):
    rows = {}
    for line in open(os.path.join(GOLDEN, name)):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        k, v = line.split(":", 1) if ":" in line else line.split(None, 1)
        rows[k.strip()] = v.split()
    return rows


def test_candidate_list_matches_paper_example():
    g = _read_golden("local_search_candidates.txt")
    assert S.candidate_blocks(64) == [int(v) for v in g["channels 64"]]
    # factors only: every candidate divides the count, every divisor but the count is listed
    for c in (3, 16, 80, 96, 192, 2048):
        cand = S.candidate_blocks(c)
        assert all(c % d == 0 for d in cand) and cand == sorted(cand, reverse=True)
        assert len(cand) == sum(1 for d in range(1, c) if c % d == 0)


# ---- graph structures (parameters are irrelevant to the search) --------------------------
def _g(nodes, shape):
    return wl.Graph(name="t", nodes=nodes, input_shape=shape)


def _conv(x, K, R=1, stride=1, pad=0, residual=-1):
    return wl.Node("conv", (x,), K=K, R=R, S=R, stride=(stride, stride), pad=(pad, pad),
                   residual=residual)


def chain_graph(k=2, C=32, HW=2):
    nodes = [wl.Node("input")]
    for i in range(k):
        nodes.append(_conv(len(nodes) - 1, C))
    nodes.append(wl.Node("flatten", (len(nodes) - 1,)))
    nodes.append(wl.Node("output", (len(nodes) - 1,)))
    return _g(nodes, (1, C, HW, HW))


def residual_graph():
    """input -> a; a -> b -> c(+a) ; c -> d(+c) -> gap -> flatten -> output."""
    n = [wl.Node("input"), _conv(0, 32)]
    n.append(_conv(1, 16, 3, pad=1))
    n.append(_conv(2, 32, residual=1))
    n.append(_conv(3, 32, 3, pad=1, residual=3))
    n.append(wl.Node("gap", (4,)))
    n.append(wl.Node("flatten", (5,)))
    n.append(wl.Node("output", (6,)))
    return _g(n, (1, 16, 6, 6))


def concat_graph():
    """Two branches of different widths joined by a concat, a pool on one."""
    n = [wl.Node("input"), _conv(0, 64, 3, stride=2, pad=1)]
    n.append(_conv(1, 32))
    n.append(_conv(1, 64, 3, pad=1))
    n.append(wl.Node("maxpool", (1,), R=3, S=3, stride=(1, 1), pad=(1, 1)))
    n.append(wl.Node("concat", (2, 3, 4)))
    n.append(_conv(5, 64))
    n.append(wl.Node("flatten", (6,)))
    n.append(wl.Node("output", (7,)))
    return _g(n, (1, 3, 8, 8))


def random_tables(graph, rng, blocks=(16, 32, 64), integer=True, p_drop=0.25):
    """conv_time / xform_time tables: every conv gets the (ic, oc) pairs its
    channel counts allow among `blocks` (and 4 on a 3-channel input), some
    dropped at random; all transform pairs get a random time."""
    shapes = S.infer_shapes(graph)
    ct = [[[S.INF] * NB for _ in range(NB)] for _ in graph.nodes]
    xt = [[[0.0] * NB for _ in range(NB)] for _ in graph.nodes]
    draw = (lambda: float(rng.integers(1, 50))) if integer else (lambda: float(rng.uniform(1, 50)))
    for v, n in enumerate(graph.nodes):
        for i in range(NB):
            for j in range(NB):
                xt[v][i][j] = 0.0 if i == j else draw()
        if n.op != "conv":
            continue
        C = shapes[n.inputs[0]][1]
        K = n.K
        ics = [b for b in blocks if C % b == 0] or [16]
        if C <= 4:
            ics = [4, 16]
        ocs = [b for b in blocks if K % b == 0] or [16]
        pairs = [(a, b) for a in ics for b in ocs]
        keep = [p for p in pairs if rng.uniform() > p_drop] or [pairs[0]]
        for a, b in keep:
            ct[v][S.BLOCKS.index(a)][S.BLOCKS.index(b)] = draw()
    return ct, xt


def _tables_from_golden(second=False):
    g = chain_graph(2, 32, 2)
    ct = [[[S.INF] * NB for _ in range(NB)] for _ in g.nodes]
    xt = [[[99.0] * NB for _ in range(NB)] for _ in g.nodes]
    b = S.BLOCKS.index
    ct[1][b(16)][b(16)], ct[1][b(16)][b(32)] = 10, 7
    ct[2][b(16)][b(16)], ct[2][b(32)][b(16)], ct[2][b(32)][b(32)] = 9, 12, 6
    xt[0][b(0)][b(16)] = 2
    xt[1][b(16)][b(32)] = xt[1][b(32)][b(16)] = 3
    xt[2][b(16)][b(0)], xt[2][b(32)][b(0)] = 1, (10 if second else 4)
    return g, ct, xt


def test_hand_worked_chain():
    gold = _read_golden("search_chain_example.txt")
    g, ct, xt = _tables_from_golden()
    best, sch = S.global_search(g, ct, xt)
    assert best == float(gold["optimum"][0])
    want = [tuple(int(t) for t in s.split(",")) for s in gold["optimum"][1:]]
    assert [sch[1], sch[2]] == want
    assert S.plan_cost(g, {1: (16, 16), 2: (32, 16)}, ct, xt) == 28
    g, ct, xt = _tables_from_golden(second=True)
    best, sch = S.global_search(g, ct, xt)
    assert best == float(gold["optimum2"][0])
    assert S.plan_cost(g, sch, ct, xt) == best
    # the greedy (locally fastest) assignment is worse
    assert S.plan_cost(g, {1: (16, 32), 2: (32, 32)}, ct, xt) == 25


def test_plan_cost_semantics():
    """Transform accounting by hand on the residual graph: reuse of a
    transformed value, residual conversion, alias at 1x1."""
    g = residual_graph()
    b = S.BLOCKS.index
    ct = [[[1.0] * NB for _ in range(NB)] for _ in g.nodes]
    xt = [[[0.0] * NB for _ in range(NB)] for _ in g.nodes]
    for v in range(len(g.nodes)):
        for i in range(NB):
            for j in range(NB):
                if i != j:
                    xt[v][i][j] = 100.0 * (v + 1) + 10 * i + j
    all16 = {1: (16, 16), 2: (16, 16), 3: (16, 16), 4: (16, 16)}
    entry = xt[0][b(0)][b(16)]
    # 4 convs + the entry transform; the exit (gap 32x1x1 -> NCHW) is an alias
    assert S.plan_cost(g, all16, ct, xt) == 4 + entry
    # node 3 in 32: its input (node 2, 16) and its residual (node 1, 16) are
    # converted; node 4 reads node 3 at 16 as input and again as residual: paid once
    sch = dict(all16)
    sch[3] = (32, 32)
    conv3 = xt[2][b(16)][b(32)] + xt[1][b(16)][b(32)]
    assert S.plan_cost(g, sch, ct, xt) == 4 + entry + conv3 + xt[3][b(32)][b(16)]
    # node 4 in (32, 32): both reads of node 3 are native; 32 % 32 == 0 keeps the exit an alias
    sch[4] = (32, 32)
    assert S.plan_cost(g, sch, ct, xt) == 4 + entry + conv3
    # node 4 out at 64: the residual is converted to 64, the pool runs in 64 and
    # 32 % 64 != 0 makes the exit a real transform of the pool's value (node 5)
    sch[4] = (32, 64)
    assert S.plan_cost(g, sch, ct, xt) == (4 + entry + conv3 + xt[3][b(32)][b(64)] +
                                          xt[5][b(64)][b(0)])


def test_exit_alias_rule():
    # input 2x2 (the entry is a real transform), a 2x2 valid conv down to 1x1
    g = _g([wl.Node("input"), _conv(0, 32, 2), wl.Node("flatten", (1,)),
            wl.Node("output", (2,))], (1, 32, 2, 2))
    ct = [[[0.0] * NB for _ in range(NB)] for _ in g.nodes]
    xt = [[[7.0] * NB for _ in range(NB)] for _ in g.nodes]
    b = S.BLOCKS.index
    # 32 channels, 1x1: out at 16 or 32 -> NCHW is an alias; only the entry is paid
    assert S.plan_cost(g, {1: (16, 16)}, ct, xt) == 7.0
    assert S.plan_cost(g, {1: (16, 32)}, ct, xt) == 7.0
    # at 64 (32 % 64 != 0) the exit is a real transform
    assert S.plan_cost(g, {1: (16, 64)}, ct, xt) == 14.0
    assert b(64) == NB - 1


@pytest.mark.parametrize("make,seed", [(lambda: chain_graph(4), 0), (residual_graph, 1),
                                       (residual_graph, 2), (concat_graph, 3),
                                       (concat_graph, 4), (lambda: wl.tiny_graph(), 5),
                                       (lambda: wl.vgg_like_tiny(), 6)])
def test_dp_equals_brute_force(make, seed):
    g = make()
    rng = np.random.default_rng(seed)
    ct, xt = random_tables(g, rng, integer=True, p_drop=0.4)
    best, sch = S.global_search(g, ct, xt)
    bf, bsch = S.brute_force(g, ct, xt)
    assert best == bf
    assert S.plan_cost(g, sch, ct, xt) == best
    assert set(sch) == set(S.conv_nodes(g))


def test_chain_reduces_to_the_recurrence():
    """On a list-shaped network the program is the printed recurrence
    GS_i(j) = t_i(j) + min_k [transform(k, j) + GS_{i-1}(k)] over the previous
    CONV's output layout k (its ic_bn choice then fixes the transform)."""
    rng = np.random.default_rng(11)
    for _ in range(5):
        g = chain_graph(6, 64, 3)
        ct, xt = random_tables(g, rng, integer=True, p_drop=0.3)
        convs = S.conv_nodes(g)
        b = S.BLOCKS.index
        # GS over the output layout of each conv
        gs = {}
        for (ic, oc) in S.schemes_of(ct, convs[0]):
            c = ct[convs[0]][b(ic)][b(oc)] + xt[0][b(0)][b(ic)]
            gs[oc] = min(gs.get(oc, S.INF), c)
        for v in convs[1:]:
            nxt = {}
            for (ic, oc) in S.schemes_of(ct, v):
                for k, prev in gs.items():
                    c = ct[v][b(ic)][b(oc)] + (0 if k == ic else xt[v - 1][b(k)][b(ic)]) + prev
                    nxt[oc] = min(nxt.get(oc, S.INF), c)
            gs = nxt
        last = convs[-1]
        want = min(c + xt[last][b(k)][b(0)] for k, c in gs.items())
        assert S.global_search(g, ct, xt)[0] == want


def test_fixed_block_assignment_is_section_3_2_plan():
    """All CONVs in 16 on ResNet-50: the only transform paid is the entry
    (the exit after the global pool is an alias), as in Section 3.2."""
    g = nets.resnet50()
    convs = S.conv_nodes(g)
    ct = [[[1.0] * NB for _ in range(NB)] for _ in g.nodes]
    xt = [[[1000.0] * NB for _ in range(NB)] for _ in g.nodes]
    sch = {v: (16, 16) for v in convs}
    assert S.plan_cost(g, sch, ct, xt) == len(convs) + 1000.0
    # and the search can only do as well, here exactly that
    for v in convs:
        for i in range(NB):
            for j in range(NB):
                ct[v][i][j] = 1.0 if (S.BLOCKS[i], S.BLOCKS[j]) in [(16, 16), (16, 32)] else S.INF
    best, s = S.global_search(g, ct, xt)
    assert best == len(convs) + 1000.0
    assert all(s[v] in [(16, 16), (16, 32)] for v in convs)


def test_search_on_real_networks_beats_or_ties_fixed_layout():
    """On the three evaluated networks with random tables, the optimum is at
    most the cost of every fixed-16 assignment, and equals plan_cost of the
    assignment it returns."""
    rng = np.random.default_rng(5)
    for build in (nets.resnet50, nets.vgg16, nets.inception_v3):
        g = build()
        ct, xt = random_tables(g, rng, integer=False, p_drop=0.0)
        best, sch = S.global_search(g, ct, xt)
        assert math.isclose(S.plan_cost(g, sch, ct, xt), best, rel_tol=1e-12)
        fixed = {v: (16 if S.infer_shapes(g)[g.nodes[v].inputs[0]][1] > 4 else 16, 16)
                 for v in S.conv_nodes(g)}
        assert best <= S.plan_cost(g, fixed, ct, xt) + 1e-9
