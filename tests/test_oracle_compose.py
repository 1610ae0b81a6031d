"""Pins of the oracle's composing functions -- the reference graph executor
(``run_graph``), one conv node with its unfused epilogue (``conv_node``,
``layer_forward``), ``bias_add``, ``concat`` and ``flatten`` -- against values
computed by hand, explicit index loops, and the already-pinned primitives
composed by hand.

Every hand example is chosen so that a plausible slip changes the answer:
ReLU before the residual add, batch norm before the bias, a dropped residual,
bias or epsilon, the residual taken from the wrong node, the bias broadcast
along the wrong axis, concat parts in the wrong order or along the wrong axis,
an (h, w, c) flatten, a dense layer without its ReLU.  All values are exact in
float32, so the comparisons are exact."""
import itertools

import numpy as np
import pytest

from paper_1809_02697_amd.workloads import Graph, LayerCase, Node

rng = np.random.default_rng(2024)


def f32(a):
    return np.asarray(a, np.float32)


# ---- one conv node: conv -> + bias -> batch norm -> + residual -> ReLU ---------------------
# Input (1, 2, 1, 3); 1x1 filter, two output channels:
#   k = 0: 2 * x0            k = 1: x0 + x1
# bias (1, -2); batch norm with eps = 1:
#   k = 0: gamma 4, var 3 -> scale 4 / sqrt(3 + 1) = 2, mean 0.5, beta -1: 2 t - 2
#   k = 1: gamma 1, var 0 -> scale 1,                    mean -1,  beta 0.5: t + 1.5
X = f32([[[[-1, 0.25, 3]], [[2, -0.5, 1]]]])
W = f32([[2, 0], [1, 1]]).reshape(2, 2, 1, 1)
BIAS = f32([1, -2])
BN = dict(gamma=f32([4, 1]), beta=f32([-1, 0.5]), mean=f32([0.5, -1]), var=f32([3, 0]), eps=1.0)
RES = f32([[[[0.5, -4, 1]], [[-3, 1, -10]]]])
# conv          k0: [-2, 0.5, 6]        k1: [1, -0.25, 4]
# + bias        k0: [-1, 1.5, 7]        k1: [-1, -2.25, 2]
# batch norm    k0: [-4, 1, 12]         k1: [0.5, -0.75, 3.5]
# + residual    k0: [-3.5, -3, 13]      k1: [-2.5, 0.25, -6.5]
# ReLU          k0: [0, 0, 13]          k1: [0, 0.25, 0]
WANT_RES_RELU = f32([[[[0, 0, 13]], [[0, 0.25, 0]]]])
WANT_BN_RELU = f32([[[[0, 1, 12]], [[0.5, 0, 3.5]]]])
WANT_BN = f32([[[[-4, 1, 12]], [[0.5, -0.75, 3.5]]]])
WANT_BIAS_RELU = f32([[[[0, 1.5, 7]], [[0, 0, 2]]]])
# The slips give, for the residual + ReLU node:
#   ReLU before the add      k1: [-2.5, 1, -6.5]   (negative outputs)
#   batch norm before bias   k0: [0, 0, 12]
#   no residual              k0: [0, 1, 12]
#   bias dropped             k0: [0, 0, 11]
#   eps dropped (sqrt(3))    k0: not an integer at all


def _conv(act="relu", residual=-1, bias=True, bn=True):
    return Node(op="conv", inputs=(0,), K=2, R=1, S=1, act=act, residual=residual, w=W,
                bias=BIAS if bias else None, bn=BN if bn else None)


def test_conv_node_epilogue_order(orc):
    np.testing.assert_array_equal(orc.conv_node(_conv(), X, RES), WANT_RES_RELU)
    np.testing.assert_array_equal(orc.conv_node(_conv(), X), WANT_BN_RELU)
    np.testing.assert_array_equal(orc.conv_node(_conv(act="none"), X), WANT_BN)
    np.testing.assert_array_equal(orc.conv_node(_conv(bn=False), X), WANT_BIAS_RELU)
    # batch norm without a bias: k0 = 2 (2x) - 2 = [-6, -1, 10]; k1 = [2.5, 1.25, 5.5]
    np.testing.assert_array_equal(orc.conv_node(_conv(act="none", bias=False), X),
                                  f32([[[[-6, -1, 10]], [[2.5, 1.25, 5.5]]]]))


@pytest.mark.parametrize("epi,bn,bias,want", [
    ("res", True, True, WANT_RES_RELU),
    ("relu", True, True, WANT_BN_RELU),
    ("none", True, True, WANT_BN),
    ("bias_relu", False, True, WANT_BIAS_RELU),
])
def test_layer_forward_epilogues(orc, epi, bn, bias, want):
    case = LayerCase("hand", 2, 2, 1, 1, (1, 1), (0, 0), 1, 3, 1, epi, 1, X, W,
                     BIAS if bias else None, BN if bn else None,
                     RES.shape if epi == "res" else None, RES if epi == "res" else None)
    np.testing.assert_array_equal(orc.layer_forward(case), want)


def test_conv_node_strided_padded_matches_parts(orc):
    """A 3x3/s2/p1 node with every epilogue term equals the pinned primitives
    applied one after the other in the stated order (bit-exact)."""
    x = f32(rng.uniform(-1, 1, (2, 5, 9, 7)))
    w = f32(rng.normal(0, 0.3, (6, 5, 3, 3)))
    b = f32(rng.normal(0, 0.1, 6))
    bn = dict(gamma=f32(rng.uniform(0.5, 1.5, 6)), beta=f32(rng.normal(0, 0.1, 6)),
              mean=f32(rng.normal(0, 0.1, 6)), var=f32(rng.uniform(0.5, 1.5, 6)), eps=1e-5)
    res = f32(rng.uniform(-1, 1, (2, 6, 5, 4)))
    n = Node(op="conv", inputs=(0,), K=6, R=3, S=3, stride=(2, 2), pad=(1, 1), act="relu",
             residual=1, w=w, bias=b, bn=bn)
    t = orc.conv2d(x, w, 2, 1)
    t = orc.bias_add(t, b)
    t = orc.batchnorm(t, bn["gamma"], bn["beta"], bn["mean"], bn["var"], bn["eps"])
    t = orc.relu(orc.add(t, res))
    np.testing.assert_array_equal(orc.conv_node(n, x, res), t)


# ---- bias_add, concat, flatten: explicit index loops ---------------------------------------
def test_bias_add_channel_axis(orc):
    """The bias runs along channel axis 1."""
    b = f32([10, 200, 3000])
    # (2, 3, 4, 5): a bias along any other axis cannot broadcast; (2, 3, 4, 3):
    # it can along the width, and gives other values
    for shape in ((2, 3, 4, 5), (2, 3, 4, 3)):
        y = f32(rng.integers(-50, 50, shape))
        out = orc.bias_add(y, b)
        assert out.shape == y.shape and out.dtype == np.float32
        for n, c, h, w in itertools.product(*map(range, shape)):
            assert out[n, c, h, w] == y[n, c, h, w] + b[c]
    # dense-shaped input: bias along the feature axis
    y2 = f32(rng.integers(-5, 5, (2, 3)))
    out2 = orc.bias_add(y2, b)
    for n, c in itertools.product(range(2), range(3)):
        assert out2[n, c] == y2[n, c] + b[c]


def test_concat_order_and_axis(orc):
    """Parts of 2, 3 and 1 channels (batch 2): the output's channels are the
    first part's, then the second's, then the third's, per image."""
    parts = [f32(1000 * (i + 1) + np.arange(2 * c * 3 * 2).reshape(2, c, 3, 2))
             for i, c in enumerate((2, 3, 1))]
    out = orc.concat(parts)
    assert out.shape == (2, 6, 3, 2)
    owner = [(0, 0), (0, 1), (1, 0), (1, 1), (1, 2), (2, 0)]  # (part, channel in part)
    for n, c, h, w in itertools.product(range(2), range(6), range(3), range(2)):
        p, cc = owner[c]
        assert out[n, c, h, w] == parts[p][n, cc, h, w]


def test_flatten_chw_order(orc):
    N, C, H, W = 2, 3, 4, 5
    x = f32(rng.uniform(-1, 1, (N, C, H, W)))
    out = orc.flatten(x)
    assert out.shape == (N, C * H * W)
    for n, c, h, w in itertools.product(range(N), range(C), range(H), range(W)):
        assert out[n, (c * H + h) * W + w] == x[n, c, h, w]


# ---- the reference graph executor ------------------------------------------------------------
def _hand_graph():
    """input -> a = relu(2x - 1) -> b = relu(x + a)  (residual from a)
             -> [maxpool 2x2/s2 of b, avgpool 2x2/s2 of a] concatenated in that
             order -> flatten -> dense with ReLU -> output."""
    nodes = [
        Node(op="input"),
        Node(op="conv", inputs=(0,), K=1, act="relu", w=f32([[[[2]]]]), bias=f32([-1])),
        Node(op="conv", inputs=(0,), K=1, act="relu", residual=1, w=f32([[[[1]]]])),
        Node(op="maxpool", inputs=(2,), R=2, S=2, stride=(2, 2)),
        Node(op="avgpool", inputs=(1,), R=2, S=2, stride=(2, 2)),
        Node(op="concat", inputs=(3, 4)),
        Node(op="flatten", inputs=(5,)),
        Node(op="dense", inputs=(6,), K=3, act="relu", w=f32([[1, -1], [-1, 0.5], [2, 0]]),
             bias=f32([0, 1, -20])),
        Node(op="output", inputs=(7,)),
    ]
    x = f32([[[[1, -2], [3, 4]]]])
    return Graph("hand", nodes, (1, 1, 2, 2), x)


def test_run_graph_hand_values(orc):
    # a = relu(2x - 1)                 = [[1, 0], [5, 7]]
    # b = relu(x + a)                  = relu([[2, -2], [8, 11]]) = [[2, 0], [8, 11]]
    # maxpool(b) = 11, avgpool(a) = 13 / 4 = 3.25; concat -> flatten = [11, 3.25]
    # dense: [11 - 3.25 + 0, -11 + 1.625 + 1, 22 - 20] = [7.75, -8.375, 2] -> ReLU
    g = _hand_graph()
    vals = orc.run_graph(g, keep=True)
    np.testing.assert_array_equal(vals[1], f32([[[[1, 0], [5, 7]]]]))
    np.testing.assert_array_equal(vals[2], f32([[[[2, 0], [8, 11]]]]))
    np.testing.assert_array_equal(vals[5], f32([[[[11]], [[3.25]]]]))
    np.testing.assert_array_equal(vals[6], f32([[11, 3.25]]))
    np.testing.assert_array_equal(orc.run_graph(g), f32([[7.75, 0, 2]]))
    # the slips: concat reversed -> [0, 0, 0.5]; residual from x -> maxpool 8,
    # logits [4.75, 0, 0]; dense without ReLU -> -8.375 in the middle


def test_run_graph_composed_by_hand(orc):
    """A random 9-node graph (ragged channels, BN, residual, both pools, concat of
    unequal parts, flatten after a real spatial map, dense + ReLU, dense) equals
    the pinned operations composed by hand, bit for bit, at every node; the input
    feeds two nodes and a value is read again after it served as a residual."""
    r = np.random.default_rng(99)
    N, C, H, W = 2, 3, 8, 6

    def bn(K):
        return dict(gamma=f32(r.uniform(0.5, 1.5, K)), beta=f32(r.normal(0, 0.1, K)),
                    mean=f32(r.normal(0, 0.1, K)), var=f32(r.uniform(0.5, 1.5, K)), eps=1e-5)

    w1, bn1 = f32(r.normal(0, 0.4, (5, C, 3, 3))), bn(5)
    w2, b2 = f32(r.normal(0, 0.4, (5, C, 1, 1))), f32(r.normal(0, 0.1, 5))
    w4, bn4 = f32(r.normal(0, 0.4, (7, 5, 1, 3))), bn(7)
    wd1, bd1 = f32(r.normal(0, 0.2, (6, 12 * 4 * 3))), f32(r.normal(0, 0.1, 6))
    wd2, bd2 = f32(r.normal(0, 0.2, (4, 6))), f32(r.normal(0, 0.1, 4))
    x = f32(r.normal(0, 1, (N, C, H, W)))
    nodes = [
        Node(op="input"),
        Node(op="conv", inputs=(0,), K=5, R=3, S=3, pad=(1, 1), act="relu", w=w1, bn=bn1),
        Node(op="conv", inputs=(0,), K=5, act="relu", residual=1, w=w2, bias=b2),
        Node(op="maxpool", inputs=(2,), R=3, S=3, stride=(2, 2), pad=(1, 1)),
        Node(op="conv", inputs=(1,), K=7, R=1, S=3, stride=(2, 2), pad=(0, 1), act="none",
             w=w4, bn=bn4),
        Node(op="concat", inputs=(3, 4)),
        Node(op="avgpool", inputs=(5,), R=3, S=3, stride=(1, 1), pad=(1, 1)),
        Node(op="flatten", inputs=(6,)),
        Node(op="dense", inputs=(7,), K=6, act="relu", w=wd1, bias=bd1),
        Node(op="dense", inputs=(8,), K=4, w=wd2, bias=bd2),
        Node(op="output", inputs=(9,)),
    ]
    g = Graph("composed", nodes, (N, C, H, W), x)

    def bnorm(t, p):
        return orc.batchnorm(t, p["gamma"], p["beta"], p["mean"], p["var"], p["eps"])

    v1 = orc.relu(bnorm(orc.conv2d(x, w1, 1, 1), bn1))
    v2 = orc.relu(orc.add(orc.bias_add(orc.conv2d(x, w2, 1, 0), b2), v1))
    v3 = orc.maxpool2d(v2, 3, 3, 2, 1)
    v4 = bnorm(orc.conv2d(v1, w4, (2, 2), (0, 1)), bn4)
    v5 = orc.concat([v3, v4])
    v6 = orc.avgpool2d(v5, 3, 3, 1, 1)
    v7 = orc.flatten(v6)
    v8 = orc.relu(orc.dense(v7, wd1, bd1))
    v9 = orc.dense(v8, wd2, bd2)
    want = [x, v1, v2, v3, v4, v5, v6, v7, v8, v9, v9]
    assert v5.shape == (N, 12, 4, 3) and v8.min() == 0 and (v8 > 0).any()
    got = orc.run_graph(g, keep=True)
    for i, (a, b) in enumerate(zip(got, want)):
        np.testing.assert_array_equal(a, b, err_msg=f"node {i}")
    np.testing.assert_array_equal(orc.run_graph(g), v9)
    # a fresh input through the same graph
    x2 = f32(r.normal(0, 1, (N, C, H, W)))
    assert not np.array_equal(orc.run_graph(g, x=x2), v9)
