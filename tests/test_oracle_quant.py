"""Pins of the oracle's integer (INT8) functions against hand values, closed
forms and brute force (no GPU)."""
import itertools

import numpy as np
import pytest

from oracle import quant as oq


def test_quantize_rounds_half_to_even_and_clamps():
    s = np.float32(0.25)          # a power of two: x / s is exact
    x = s * np.array([0.0, 0.5, 1.5, 2.5, -0.5, -2.5, 3.49, 126.5, 127.5, 300.0, -300.0],
                     np.float32)
    np.testing.assert_array_equal(oq.quantize(x, s), [0, 0, 2, 2, 0, -2, 3, 126, 127, 127, -127])
    # symmetric, and exact multiples of the scale map to their integers
    k = np.arange(-127, 128, dtype=np.float32)
    np.testing.assert_array_equal(oq.quantize(k * s, s), k.astype(np.int8))
    r = np.random.default_rng(0).normal(0, 3, 1000).astype(np.float32)
    np.testing.assert_array_equal(oq.quantize(-r, 0.1), -oq.quantize(r, 0.1))


def test_filter_scales_map_each_channels_extreme_to_127():
    w = np.zeros((3, 2, 1, 2), np.float32)
    w[0] = [[[0.5, -1.0]], [[0.25, 0.0]]]     # max |w| 1.0
    w[1] = [[[-6.35, 2.0]], [[1.0, 3.175]]]   # max |w| 6.35
    q, s = oq.quantize_filter(w)               # channel 2 is all zero
    np.testing.assert_array_equal(s, np.float32([1.0 / 127, 6.35 / 127, 1.0]))
    assert q[0, 0, 0, 1] == -127 and q[1, 0, 0, 0] == -127
    np.testing.assert_array_equal(q[0].ravel(), [64, -127, 32, 0])     # 63.5 -> 64 (ties to even)
    np.testing.assert_array_equal(q[1].ravel(), [-127, 40, 20, 64])    # 63.5 -> 64
    assert (q[2] == 0).all()


def _brute(xq, wq, st, pd):
    N, C, H, W = xq.shape
    K, _, R, S = wq.shape
    OH, OW = (H + 2 * pd[0] - R) // st[0] + 1, (W + 2 * pd[1] - S) // st[1] + 1
    y = np.zeros((N, K, OH, OW), np.int64)
    for n, k, oh, ow in itertools.product(range(N), range(K), range(OH), range(OW)):
        acc = 0
        for c, r, s in itertools.product(range(C), range(R), range(S)):
            ih, iw = oh * st[0] - pd[0] + r, ow * st[1] - pd[1] + s
            if 0 <= ih < H and 0 <= iw < W:
                acc += int(xq[n, c, ih, iw]) * int(wq[k, c, r, s])
        y[n, k, oh, ow] = acc
    return y


@pytest.mark.parametrize("N,C,H,W,K,R,S,st,pd", [
    (1, 3, 5, 4, 2, 3, 3, (1, 1), (1, 1)),
    (2, 2, 6, 7, 3, 1, 3, (2, 1), (0, 1)),
    (1, 4, 7, 5, 2, 3, 1, (1, 2), (2, 0)),
    (1, 1, 4, 4, 1, 2, 2, (2, 2), (0, 0)),
])
def test_integer_conv_equals_brute_force(N, C, H, W, K, R, S, st, pd):
    rng = np.random.default_rng([N, C, H, W, K, R, S])
    xq = rng.integers(-127, 128, (N, C, H, W)).astype(np.int8)
    wq = rng.integers(-127, 128, (K, C, R, S)).astype(np.int8)
    np.testing.assert_array_equal(oq.conv2d_int(xq, wq, st, pd), _brute(xq, wq, st, pd))


def test_integer_conv_closed_forms():
    rng = np.random.default_rng(3)
    # 1x1 stride 1 is a matrix product of integers
    xq = rng.integers(-127, 128, (2, 5, 3, 4)).astype(np.int8)
    wq = rng.integers(-127, 128, (6, 5, 1, 1)).astype(np.int8)
    want = np.einsum("kc,nchw->nkhw", wq[:, :, 0, 0].astype(np.int64), xq.astype(np.int64))
    np.testing.assert_array_equal(oq.conv2d_int(xq, wq), want)
    # a delta filter shifts the input (zero padding)
    x = rng.integers(-127, 128, (1, 2, 5, 6)).astype(np.int8)
    d = np.zeros((2, 2, 3, 3), np.int8)
    d[0, 1, 2, 0] = 1
    d[1, 0, 0, 2] = -1
    y = oq.conv2d_int(x, d, 1, 1)
    xp = np.pad(x.astype(np.int64), ((0, 0), (0, 0), (1, 1), (1, 1)))
    np.testing.assert_array_equal(y[0, 0], xp[0, 1, 2:2 + 5, 0:0 + 6])
    np.testing.assert_array_equal(y[0, 1], -xp[0, 0, 0:5, 2:2 + 6])
    # sums beyond float32's exact range stay exact: all-127 inputs and filters,
    # 512 channels x 3 x 3: 127^2 times the in-bounds taps (up to 74,317,824)
    x = np.full((1, 512, 4, 4), 127, np.int8)
    w = np.full((1, 512, 3, 3), 127, np.int8)
    taps = np.array([[4, 6, 6, 4], [6, 9, 9, 6], [6, 9, 9, 6], [4, 6, 6, 4]])
    np.testing.assert_array_equal(oq.conv2d_int(x, w, 1, 1)[0, 0], 127 * 127 * 512 * taps)


def test_dequantize_by_hand():
    acc = np.array([[[[100]], [[-3]]]], np.int64)          # N=1, K=2, 1x1
    mult = oq.multipliers(0.5, np.float32([0.25, 2.0]))
    np.testing.assert_array_equal(mult, np.float32([0.125, 1.0]))
    bias = np.float32([1.0, 0.5])
    res = np.array([[[[-20.0]], [[1.0]]]], np.float32)
    # 100 * 0.125 + 1 - 20 = -6.5 -> ReLU 0; -3 * 1 + 0.5 + 1 = -1.5 -> 0
    np.testing.assert_array_equal(oq.dequantize(acc, mult, bias, res, "relu").ravel(), [0.0, 0.0])
    np.testing.assert_array_equal(oq.dequantize(acc, mult, bias, res).ravel(), [-6.5, -1.5])
    np.testing.assert_array_equal(oq.dequantize(acc, mult).ravel(), [12.5, -3.0])


def test_epilogue_rounds_each_operation_to_float32():
    # 2^24 + 1 converts to 2^24; adding 1 then ties back to 2^24 (even).  In
    # float64 (or with the sum formed before rounding) the result would be
    # 2^24 + 2, which float32 holds exactly.
    acc = np.array([[[[2 ** 24 + 1]]]], np.int64)
    one = np.float32([1.0])
    assert oq.epilogue_f32(acc, one, one).item() == 2.0 ** 24
    assert oq.dequantize(acc, one, one).item() == 2.0 ** 24 + 2
    # hand values: (100 * 0.125 + 1) - 20 = -6.5 -> ReLU +0; (-3 * 1 + 0.5) + 1 = -1.5
    acc = np.array([[[[100]], [[-3]]]], np.int64)
    mult = oq.multipliers(0.5, np.float32([0.25, 2.0]))
    bias = np.float32([1.0, 0.5])
    res = np.array([[[[-20.0]], [[1.0]]]], np.float32)
    np.testing.assert_array_equal(oq.epilogue_f32(acc, mult, bias, res).ravel(), [-6.5, -1.5])
    y = oq.epilogue_f32(acc, mult, bias, res, "relu").ravel()
    assert (y == 0).all() and not np.signbit(y).any()
    # on random sums it stays within 6 u of the ideal value
    rng = np.random.default_rng(5)
    acc = rng.integers(-2 ** 26, 2 ** 26, (2, 3, 4, 5))
    mult = rng.uniform(1e-5, 1e-3, 3).astype(np.float32)
    b = rng.normal(0, 1, 3).astype(np.float32)
    r = rng.normal(0, 1, acc.shape).astype(np.float32)
    y32 = oq.epilogue_f32(acc, mult, b, r).astype(np.float64)
    y64 = oq.dequantize(acc, mult, b, r).astype(np.float64)
    mag = np.abs(acc * mult.astype(np.float64)[None, :, None, None]) + \
        np.abs(b.astype(np.float64))[None, :, None, None] + np.abs(r)
    assert (np.abs(y32 - y64) <= 6 * 2.0 ** -24 * mag).all()


def test_requantize_multiplies_by_the_float32_reciprocal():
    s = np.float32(0.25)                       # reciprocal 4, exact
    y = np.float32([0.125, 0.375, -0.375, 1.0, 40.0, -40.0])
    np.testing.assert_array_equal(oq.requantize(y, s), [0, 2, -2, 4, 127, -127])
    # 45.5 / 7 is an exact tie (6.5 -> 6), but 45.5 * float32(1/7) rounds to
    # just above 6.5 in float32 (-> 7)
    assert oq.quantize(np.float32([45.5]), 7.0)[0] == 6
    assert oq.requantize(np.float32([45.5]), 7.0)[0] == 7



def test_fold_bn_by_hand_and_against_the_unfolded_conv():
    import oracle as fo
    # var + eps = 4: s = gamma / 2; b' = (b - mean) s + beta
    bn = dict(gamma=np.float32([2.0, 1.0]), beta=np.float32([0.5, -1.0]), mean=np.float32([1.0, 0.0]),
              var=np.float32([4.0 - 2.0 ** -10, 4.0 - 2.0 ** -10]), eps=2.0 ** -10)
    w = np.float32([3.0, -6.0]).reshape(2, 1, 1, 1)
    w2, b2 = oq.fold_bn(w, np.float32([5.0, 2.0]), bn)
    np.testing.assert_array_equal(w2.ravel(), [3.0, -3.0])
    np.testing.assert_array_equal(b2, [(5 - 1) * 1 + 0.5, (2 - 0) * 0.5 - 1.0])
    assert oq.fold_bn(w, None, bn)[1][0] == (0 - 1) * 1 + 0.5
    # a folded conv equals the conv followed by batch norm (pinned primitives)
    rng = np.random.default_rng(8)
    x = rng.normal(0, 1, (1, 4, 6, 6)).astype(np.float32)
    w = rng.normal(0, 0.3, (5, 4, 3, 3)).astype(np.float32)
    bn = dict(gamma=rng.uniform(0.5, 1.5, 5).astype(np.float32), beta=rng.normal(0, 0.1, 5).astype(np.float32),
              mean=rng.normal(0, 0.1, 5).astype(np.float32), var=rng.uniform(0.5, 1.5, 5).astype(np.float32),
              eps=1e-5)
    w2, b2 = oq.fold_bn(w, None, bn)
    got = fo.bias_add(fo.conv2d(x, w2, 1, 1), b2)
    want = fo.batchnorm(fo.conv2d(x, w, 1, 1), bn["gamma"], bn["beta"], bn["mean"], bn["var"], bn["eps"])
    np.testing.assert_allclose(got, want, rtol=1e-5, atol=1e-6)


def test_act_scale():
    assert oq.act_scale(np.float32([[-254.0, 3.0]])) == np.float32(2.0)
    assert oq.act_scale(np.zeros(5, np.float32)) == np.float32(1.0)
    assert oq.act_scale(np.float32([0.5])) == np.float32(0.5) / np.float32(127)


def _integer_graph():
    """A network on which every quantization is exact: an integer input of
    max 127, convs whose filters are 127 times a 0/1 pattern (per-channel
    scale 1), so each conv's output is 127 times its input's integers and
    the next scale a power of 127.  Conv 1's output is read by conv 2 alone
    (a chained, requantized input); the rest take their own quantization.
    The dense layer reads the concatenation [P, 128 P] (P the pool's output,
    128 P the residual block's) at scale 128 * 127^2: the 128 P half
    quantizes exactly, and the dense weights (127 times a -1/0/1 pattern,
    row scale 1) are zero on the P half, whose quantization is not exact."""
    from paper_1809_02697_amd.workloads import Graph, Node
    rng = np.random.default_rng(12)
    x = rng.integers(-127, 128, (2, 3, 6, 5)).astype(np.float32)
    x[0, 0, 0, 0] = 127.0
    eye = lambda K, C: (127.0 * np.eye(K, C)).reshape(K, C, 1, 1).astype(np.float32)
    shift = np.zeros((3, 3, 3, 3), np.float32)
    for k in range(3):
        shift[k, k, 1, 1] = 127.0        # a centred delta: the identity with padding
    wd = np.zeros((4, 6 * 3 * 2), np.float32)
    wd[:, 18:] = 127.0 * rng.integers(-1, 2, (4, 18))
    wd[:, 18] = 127.0                    # every row nonzero: row scale 1
    nodes = [
        Node("input"),
        Node("conv", (0,), K=3, R=1, S=1, w=eye(3, 3)),                       # 127 x
        Node("conv", (1,), K=3, R=3, S=3, pad=(1, 1), w=shift),               # 127^2 x
        Node("maxpool", (2,), R=2, S=2, stride=(2, 2)),                      # 3 x 3 x 2
        Node("conv", (3,), K=3, R=1, S=1, w=eye(3, 3), residual=3, act="relu"),
        Node("concat", (3, 4)),
        Node("flatten", (5,)),
        Node("dense", (6,), K=4, w=wd),
        Node("output", (7,)),
    ]
    return Graph("integer", nodes, x.shape, x)


def test_integer_network_equals_the_float_network():
    """Every scale is a power of 127 and every quantization exact (the last
    conv's products round once, on both sides alike), so the integer path
    reproduces the float oracle's network exactly, with the scales fixed by
    hand: 1 for the input, 127 for conv 1's output, 127^2 for the pool's,
    128 * 127^2 for the dense layer's input (the dense sums stay below 2^24
    and round once on both sides)."""
    import oracle as fo
    g = _integer_graph()
    y8, scales = oq.run_graph_int8(g)
    np.testing.assert_array_equal(scales, np.float32([1.0, 127.0, 16129.0, 128.0 * 16129.0]))
    np.testing.assert_array_equal(y8, fo.run_graph(g))


def test_dense_layers_chain_by_requantization():
    """A dense layer's output read by the next dense layer is requantized
    (the reciprocal), the network input of the first quantized by division.
    By hand: the input [7, 0, 127] has scale 1; dense 1 (rows 127 e0 and
    127 e1, row scale 1, bias [0, 45.5]) gives [889, 45.5], scale 7; 45.5 / 7
    is the exact tie 6.5, requantized to 7 (division: 6), 889 to 127; dense 2
    (rows 127 e1 and 127 e0) then gives 127 * 7 * 7 = 6223 and
    127 * 127 * 7 = 112903."""
    from paper_1809_02697_amd.workloads import Graph, Node
    x = np.float32([7.0, 0.0, 127.0]).reshape(1, 3, 1, 1)
    wa = np.float32([[127, 0, 0], [0, 127, 0]])
    wb = np.float32([[0, 127], [127, 0]])
    nodes = [
        Node("input"),
        Node("flatten", (0,)),
        Node("dense", (1,), K=2, w=wa, bias=np.float32([0.0, 45.5])),
        Node("dense", (2,), K=2, w=wb),
        Node("output", (3,)),
    ]
    y, scales = oq.run_graph_int8(Graph("dense chain", nodes, x.shape, x))
    np.testing.assert_array_equal(scales, np.float32([1.0, 7.0]))
    np.testing.assert_array_equal(y, np.float32([[6223.0, 112903.0]]))


def test_integer_dense_sums_exactly():
    """dense_int is the exact integer matrix product: brute force on a small
    case, and the extreme 127^2 * 25088 (VGG-16's first dense layer)."""
    rng = np.random.default_rng(9)
    xq = rng.integers(-127, 128, (3, 37)).astype(np.int8)
    wq = rng.integers(-127, 128, (5, 37)).astype(np.int8)
    want = np.array([[sum(int(xq[n, i]) * int(wq[k, i]) for i in range(37)) for k in range(5)]
                     for n in range(3)])
    np.testing.assert_array_equal(oq.dense_int(xq, wq), want)
    big = oq.dense_int(np.full((1, 25088), 127, np.int8), np.full((2, 25088), -127, np.int8))
    assert big.dtype == np.int64 and (big == -127 * 127 * 25088).all()


def test_conv_output_read_with_two_paddings_is_requantized():
    """A conv's output read by a 1x3 conv (padding (0, 1)) and a 3x1 conv
    (padding (1, 0)) is requantized by the reciprocal for both.  The value
    45.5 at scale 7 is the exact tie 6.5: division rounds it to 6 (half to
    even), 45.5 * float32(1/7) to 7.  By hand: the input's scale is 1 (its
    maximum 127 sits in a channel no filter reads); the first conv gives
    127 * x0 (at most 889 = 7 * 127, so scale 7) and the constant 45.5 from
    its bias; the delta filters (127 at the centre tap of channel 1) then
    give 127 * 7 * 7 = 6223 at every pixel (5334 with the division)."""
    from paper_1809_02697_amd.workloads import Graph, Node
    rng = np.random.default_rng(3)
    x = np.zeros((1, 3, 4, 5), np.float32)
    x[0, 0] = rng.integers(-7, 8, (4, 5))
    x[0, 0, 2, 3] = 7.0
    x[0, 2, 1, 1] = 127.0
    wa = np.zeros((2, 3, 1, 1), np.float32)
    wa[0, 0] = 127.0
    wa[1, 1] = 127.0
    wb = np.zeros((1, 2, 1, 3), np.float32)
    wb[0, 1, 0, 1] = 127.0
    wc = np.zeros((1, 2, 3, 1), np.float32)
    wc[0, 1, 1, 0] = 127.0
    nodes = [
        Node("input"),
        Node("conv", (0,), K=2, R=1, S=1, w=wa, bias=np.float32([0.0, 45.5])),
        Node("conv", (1,), K=1, R=1, S=3, pad=(0, 1), w=wb),
        Node("conv", (1,), K=1, R=3, S=1, pad=(1, 0), w=wc),
        Node("concat", (2, 3)),
        Node("output", (4,)),
    ]
    g = Graph("two paddings", nodes, x.shape, x)
    y, scales = oq.run_graph_int8(g)
    np.testing.assert_array_equal(scales, np.float32([1.0, 7.0, 7.0]))
    np.testing.assert_array_equal(y, np.full((1, 2, 4, 5), 6223.0, np.float32))


def test_concatenation_is_assembled_by_its_parts_producers():
    """A concatenation of a conv's output and a pool's output (each read by
    nothing else), read by a conv: its int8 tensor has the concatenation's
    scale, the conv part requantized by the reciprocal and the pool part
    quantized by division.  Both parts hold 45.5 at scale 7 (the exact tie
    6.5): the conv part gives 7, the pool part 6, so the reading conv (delta
    filters on one channel of each part) gives 127 * 7 * 7 = 6223 and
    127 * 6 * 7 = 5334 at every pixel; quantizing the whole concatenation
    one way would give one of them twice.  Scales by hand: 1 for the
    input (its 127 sits in a channel no filter reads), 1 for it again, 7
    for the concatenation (maximum 127 * 7 = 889 in the conv part)."""
    from paper_1809_02697_amd.workloads import Graph, Node
    rng = np.random.default_rng(5)
    x = np.zeros((1, 3, 4, 5), np.float32)
    x[0, 0] = rng.integers(-7, 8, (4, 5))
    x[0, 0, 3, 4] = 7.0
    x[0, 2, 0, 2] = 127.0
    wa = np.zeros((2, 3, 1, 1), np.float32)
    wa[0, 0] = 127.0
    wa[1, 1] = 127.0
    wb = np.zeros((2, 3, 1, 1), np.float32)
    wb[0, 1] = 127.0     # the conv part's constant channel
    wb[1, 2] = 127.0     # the pool part
    nodes = [
        Node("input"),
        Node("conv", (0,), K=2, R=1, S=1, w=wa, bias=np.float32([0.0, 45.5])),
        Node("conv", (0,), K=1, R=1, S=1, w=np.zeros((1, 3, 1, 1), np.float32), bias=np.float32([45.5])),
        Node("maxpool", (2,), R=1, S=1, stride=(1, 1)),
        Node("concat", (1, 3)),
        Node("conv", (4,), K=2, R=1, S=1, w=wb),
        Node("output", (5,)),
    ]
    g = Graph("assembled concatenation", nodes, x.shape, x)
    y, scales = oq.run_graph_int8(g)
    np.testing.assert_array_equal(scales, np.float32([1.0, 1.0, 7.0]))
    want = np.stack([np.full((4, 5), 6223.0), np.full((4, 5), 5334.0)])[None].astype(np.float32)
    np.testing.assert_array_equal(y, want)


def test_nested_concatenation_is_assembled_by_its_parts_producers():
    """The same assembly through a concatenation nested in another: the
    outer concatenation [conv part, [pool part]] reads like the flat one
    (6223 and 5334 by hand, scales 1, 1, 7)."""
    from paper_1809_02697_amd.workloads import Graph, Node
    rng = np.random.default_rng(5)
    x = np.zeros((1, 3, 4, 5), np.float32)
    x[0, 0] = rng.integers(-7, 8, (4, 5))
    x[0, 0, 3, 4] = 7.0
    x[0, 2, 0, 2] = 127.0
    wa = np.zeros((2, 3, 1, 1), np.float32)
    wa[0, 0] = 127.0
    wa[1, 1] = 127.0
    wb = np.zeros((2, 3, 1, 1), np.float32)
    wb[0, 1] = 127.0
    wb[1, 2] = 127.0
    nodes = [
        Node("input"),
        Node("conv", (0,), K=2, R=1, S=1, w=wa, bias=np.float32([0.0, 45.5])),
        Node("conv", (0,), K=1, R=1, S=1, w=np.zeros((1, 3, 1, 1), np.float32), bias=np.float32([45.5])),
        Node("maxpool", (2,), R=1, S=1, stride=(1, 1)),
        Node("concat", (3,)),
        Node("concat", (1, 4)),
        Node("conv", (5,), K=2, R=1, S=1, w=wb),
        Node("output", (6,)),
    ]
    y, scales = oq.run_graph_int8(Graph("nested concatenation", nodes, x.shape, x))
    np.testing.assert_array_equal(scales, np.float32([1.0, 1.0, 7.0]))
    want = np.stack([np.full((4, 5), 6223.0), np.full((4, 5), 5334.0)])[None].astype(np.float32)
    np.testing.assert_array_equal(y, want)
