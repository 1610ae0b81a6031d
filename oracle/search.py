"""Global layout search (Section 3.3.2, Algorithm 2) -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct statement of what the planner's global
search computes, written from the paper's description:

* Every CONV chooses a scheme, the pair (ic_bn, oc_bn) of the channel split
  factors of its input and output (x in NCHW[x]c).  Each scheme has an
  execution time measured by the local search (Section 3.3.1).
* Operations between CONVs are layout-oblivious or layout-tolerant
  (Section 3.2), so they run in whatever layout their input arrives in;
  operations that need two operands in one layout (Elementwise_Add, here the
  residual fused into a CONV, and Concat) convert the other operands to the
  layout of the first one (the rule the paper gives for its approximate
  solver, Section 3.3.2); Flatten, Dense and the network output need the
  default layout NCHW.
* A LayoutTransform is paid whenever a consumer needs a value in a layout it
  does not have yet; a value transformed once is reused by later consumers.
* The global search minimises the sum of the CONV execution times and the
  transform times over every scheme assignment.

``plan_cost`` is the cost of one assignment, by direct simulation of the
rules above (the definition).  ``global_search`` is Algorithm 2's dynamic
program: nodes in topological order, the memorised optimum for every
combination of layouts of the values that are still to be read (the paper's
"schemes of a CONV may need to be saved for a future use"), which makes the
program exact on any graph.  ``brute_force`` enumerates every assignment (tiny
graphs only) and pins the dynamic program.

Layouts are block sizes: 0 = NCHW, x > 0 = NCHW[x]c.  Costs come in two
tables over the block list ``BLOCKS``:
  conv_time[v][i][j]  execution time of CONV node v with ic_bn = BLOCKS[i],
                      oc_bn = BLOCKS[j]; inf where the pair is no candidate
  xform_time[v][i][j] time of transforming node v's value from BLOCKS[i] to
                      BLOCKS[j]
A transform whose source and destination coincide in memory (a 1x1 map whose
channel count both blocks divide, not written into a concat slice) is an
alias and costs 0.

Only ``tests/`` use this module.  It shares no code with the HIP library.
"""
from __future__ import annotations

import itertools
import math

BLOCKS = (0, 4, 8, 16, 32, 64)
INF = math.inf


def candidate_blocks(channels):
    """Section 3.3.1, step 1: the candidate split factors of a channel count
    are its factors, largest first.  The printed example lists 32, 16, 8, 4,
    2, 1 for 64 channels, i.e. the count itself is left out; this follows the
    example."""
    return [d for d in range(channels - 1, 0, -1) if channels % d == 0]


def _out(n, k, s, p):
    return (n + 2 * p - k) // s + 1


def infer_shapes(graph):
    """(N, C, H, W) of every node's value (flat values have H = W = 1)."""
    shapes = [None] * len(graph.nodes)
    for i, n in enumerate(graph.nodes):
        if n.op == "input":
            shapes[i] = tuple(graph.input_shape)
            continue
        N, C, H, W = shapes[n.inputs[0]]
        if n.op == "conv":
            shapes[i] = (N, n.K, _out(H, n.R, n.stride[0], n.pad[0]),
                         _out(W, n.S, n.stride[1], n.pad[1]))
        elif n.op in ("maxpool", "avgpool"):
            shapes[i] = (N, C, _out(H, n.R, n.stride[0], n.pad[0]),
                         _out(W, n.S, n.stride[1], n.pad[1]))
        elif n.op == "gap":
            shapes[i] = (N, C, 1, 1)
        elif n.op == "concat":
            shapes[i] = (N, sum(shapes[j][1] for j in n.inputs), H, W)
        elif n.op == "flatten":
            shapes[i] = (N, C * H * W, 1, 1)
        elif n.op == "dense":
            shapes[i] = (N, n.K, 1, 1)
        elif n.op == "output":
            shapes[i] = (N, C, H, W)
        else:
            raise ValueError(n.op)
    return shapes


def topo_order(graph):
    """Any topological order (inputs and residuals before their reader); the
    optimum does not depend on which."""
    n = len(graph.nodes)
    deps = [set(nd.inputs) | ({nd.residual} if nd.op == "conv" and nd.residual >= 0 else set())
            for nd in graph.nodes]
    done, order = set(), []
    while len(order) < n:
        for i in range(n):
            if i not in done and deps[i] <= done:
                done.add(i)
                order.append(i)
                break
        else:
            raise ValueError("cycle")
    return order


def _bi(block):
    return BLOCKS.index(block)


def _alias(shape, src, dst, into_concat):
    """Source and destination layouts coincide in memory."""
    _, C, H, W = shape
    if into_concat or H * W != 1:
        return False
    return all(b == 0 or C % b == 0 for b in (src, dst))


def _concat_layout(graph, shapes, v, first_layout, default_block):
    parts = [shapes[j][1] for j in graph.nodes[v].inputs]
    if first_layout > 0 and all(c % first_layout == 0 for c in parts):
        return first_layout
    if all(c % default_block == 0 for c in parts):
        return default_block
    return 0


def plan_cost(graph, schemes, conv_time, xform_time, default_block=16, transforms=None):
    """Cost of one assignment {conv node: (ic_bn, oc_bn)}: walk the nodes,
    give every value the layout its producer leaves it in, and pay a transform
    for each (value, layout) a consumer needs that the value does not have.
    If ``transforms`` is a list, every transform is appended to it as
    (value's node, from block, to block, is_alias)."""
    shapes = infer_shapes(graph)
    native = {}
    have = {}
    total = 0.0

    def need(u, layout, into_concat=False):
        nonlocal total
        if layout in have[u]:
            return
        have[u].add(layout)
        alias = _alias(shapes[u], native[u], layout, into_concat)
        if transforms is not None:
            transforms.append((u, native[u], layout, alias))
        if not alias:
            total += xform_time[u][_bi(native[u])][_bi(layout)]

    for v in topo_order(graph):
        n = graph.nodes[v]
        if n.op == "input":
            lay = 0
        elif n.op == "conv":
            ic, oc = schemes[v]
            total += conv_time[v][_bi(ic)][_bi(oc)]
            need(n.inputs[0], ic)
            if n.residual >= 0:
                need(n.residual, oc)
            lay = oc
        elif n.op in ("maxpool", "avgpool", "gap"):
            u = n.inputs[0]
            lay = native[u] if native[u] > 0 else default_block
            need(u, lay)
        elif n.op == "concat":
            lay = _concat_layout(graph, shapes, v, native[n.inputs[0]], default_block)
            for u in n.inputs:
                need(u, lay, into_concat=True)
        else:  # flatten, dense, output: the default layout
            need(n.inputs[0], 0)
            lay = 0
        native[v] = lay
        have[v] = {lay}
    return total


def conv_nodes(graph):
    return [i for i, n in enumerate(graph.nodes) if n.op == "conv"]


def schemes_of(conv_time, v):
    """The candidate schemes of CONV node v: pairs with a finite time."""
    return [(BLOCKS[i], BLOCKS[j]) for i in range(len(BLOCKS)) for j in range(len(BLOCKS))
            if conv_time[v][i][j] < INF]


def brute_force(graph, conv_time, xform_time, default_block=16):
    """Minimum of plan_cost over every assignment (tiny graphs only)."""
    convs = conv_nodes(graph)
    best, arg = INF, None
    for combo in itertools.product(*[schemes_of(conv_time, v) for v in convs]):
        sch = dict(zip(convs, combo))
        c = plan_cost(graph, sch, conv_time, xform_time, default_block)
        if c < best:
            best, arg = c, sch
    return best, arg


def global_search(graph, conv_time, xform_time, default_block=16):
    """Algorithm 2.  Visit the nodes in topological order; for a CONV, every
    candidate scheme j costs its execution time plus, for each predecessor
    scheme k already memorised, the transform from k to j plus the optimum up
    to k; keep the best per combination.  The memorised combinations are the
    layouts of every value still to be read (a value read by several later
    nodes keeps its layout in the state, with the set of layouts it has been
    transformed to).  Returns (optimal cost, {conv node: (ic_bn, oc_bn)})."""
    shapes = infer_shapes(graph)
    order = topo_order(graph)
    pos = {v: k for k, v in enumerate(order)}
    last = {}
    for v in order:
        n = graph.nodes[v]
        for u in tuple(n.inputs) + ((n.residual,) if n.op == "conv" and n.residual >= 0 else ()):
            last[u] = max(last.get(u, -1), pos[v])

    # state: tuple of (value, native layout, frozenset of layouts it has),
    # sorted by value; entry: (cost, previous state, choice)
    layers = [{(): (0.0, None, None)}]
    for v in order:
        n = graph.nodes[v]
        nxt = {}
        if n.op == "conv":
            choices = schemes_of(conv_time, v)
        else:
            choices = [None]
        for key, (cost, _, _) in layers[-1].items():
            st = {u: (nat, have) for u, nat, have in key}
            for ch in choices:
                s2 = dict(st)
                c = cost

                def fetch(u, layout, into_concat=False):
                    nat, have = s2[u]
                    if layout in have:
                        return 0.0
                    s2[u] = (nat, have | {layout})
                    if _alias(shapes[u], nat, layout, into_concat):
                        return 0.0
                    return xform_time[u][_bi(nat)][_bi(layout)]

                if n.op == "input":
                    lay = 0
                elif n.op == "conv":
                    ic, oc = ch
                    c += conv_time[v][_bi(ic)][_bi(oc)]
                    c += fetch(n.inputs[0], ic)
                    if n.residual >= 0:
                        c += fetch(n.residual, oc)
                    lay = oc
                elif n.op in ("maxpool", "avgpool", "gap"):
                    nat = s2[n.inputs[0]][0]
                    lay = nat if nat > 0 else default_block
                    c += fetch(n.inputs[0], lay)
                elif n.op == "concat":
                    lay = _concat_layout(graph, shapes, v, s2[n.inputs[0]][0], default_block)
                    for u in n.inputs:
                        c += fetch(u, lay, into_concat=True)
                else:
                    c += fetch(n.inputs[0], 0)
                    lay = 0
                if c == INF:
                    continue
                if last.get(v, -1) > pos[v]:
                    s2[v] = (lay, frozenset([lay]))
                k2 = tuple(sorted((u, nat, have) for u, (nat, have) in s2.items()
                                  if last.get(u, -1) > pos[v]))
                if k2 not in nxt or c < nxt[k2][0]:
                    nxt[k2] = (c, key, ch)
        if not nxt:
            return INF, None
        layers.append(nxt)

    # the last layer holds the empty state (nothing is read after the output)
    key = min(layers[-1], key=lambda k: layers[-1][k][0])
    best = layers[-1][key][0]
    schemes = {}
    for k in range(len(order), 0, -1):
        cost, prev, ch = layers[k][key]
        if ch is not None:
            schemes[order[k - 1]] = ch
        key = prev
    return best, schemes
