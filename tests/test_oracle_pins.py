"""Pins of the CPU oracle against facts that do not come from the oracle itself:
brute force over the definition, textbook identities, hand-computed values and
closed-form index maps.  Each test is chosen so that a plausible slip in the
oracle (a dropped term, a flipped kernel, a wrong padding offset or stride, a
transposed operand, float32 accumulation) fails it."""
import itertools

import numpy as np
import pytest

rng = np.random.default_rng(12345)


def _bruteforce_conv(x, w, stride, pad):
    """Per-output dot product of the zero-padded receptive field with the
    filter, in float64 (the definition written with numpy slicing)."""
    (sh, sw), (ph, pw) = stride, pad
    N, C, H, W = x.shape
    K, _, R, S = w.shape
    xp = np.pad(x.astype(np.float64), ((0, 0), (0, 0), (ph, ph), (pw, pw)))
    OH = (H + 2 * ph - R) // sh + 1
    OW = (W + 2 * pw - S) // sw + 1
    y = np.zeros((N, K, OH, OW))
    for n, k, i, j in itertools.product(range(N), range(K), range(OH), range(OW)):
        field = xp[n, :, i * sh:i * sh + R, j * sw:j * sw + S]
        y[n, k, i, j] = np.dot(field.ravel(), w[k].astype(np.float64).ravel())
    return y


SHAPES = [
    # N, C, K, H, W, R, S, stride, pad
    (1, 1, 1, 5, 5, 3, 3, (1, 1), (0, 0)),
    (2, 3, 4, 7, 6, 3, 3, (1, 1), (1, 1)),
    (1, 5, 2, 9, 9, 3, 3, (2, 2), (1, 1)),
    (2, 2, 3, 8, 7, 1, 3, (1, 2), (0, 1)),
    (1, 4, 4, 7, 9, 3, 1, (2, 1), (2, 0)),
    (1, 3, 2, 6, 6, 2, 2, (2, 2), (0, 0)),
    (2, 5, 3, 9, 8, 1, 1, (2, 2), (0, 0)),
    (1, 2, 4, 5, 7, 3, 3, (1, 1), (2, 2)),
]


@pytest.mark.parametrize("shape", SHAPES)
def test_conv_matches_bruteforce(orc, shape):
    N, C, K, H, W, R, S, st, pd = shape
    x = rng.uniform(-1, 1, (N, C, H, W)).astype(np.float32)
    w = rng.normal(0, 1, (K, C, R, S)).astype(np.float32)
    y = orc.conv2d(x, w, st, pd)
    ref = _bruteforce_conv(x, w, st, pd)
    assert y.shape == ref.shape
    np.testing.assert_allclose(y, ref, rtol=2e-7, atol=1e-7)


def test_conv_hand_example(orc):
    """Cross-correlation (no kernel flip): 3x3 input 1..9, 2x2 kernel [[1,2],[3,4]]."""
    x = np.arange(1, 10, dtype=np.float32).reshape(1, 1, 3, 3)
    w = np.array([[1, 2], [3, 4]], np.float32).reshape(1, 1, 2, 2)
    y = orc.conv2d(x, w, 1, 0)
    np.testing.assert_array_equal(y[0, 0], [[37, 47], [67, 77]])
    # padding 1: corner output sees only x[0,0] under w[1,1]
    y = orc.conv2d(x, w, 1, 1)
    assert y.shape == (1, 1, 4, 4)
    assert y[0, 0, 0, 0] == 4 * 1
    assert y[0, 0, 3, 3] == 1 * 9


def test_conv_accumulates_in_double(orc):
    """1 + 1e8 - 1e8 over three channels: float32 running sums give 0."""
    x = np.array([1e8, 1.0, -1e8], np.float32).reshape(1, 3, 1, 1)
    w = np.ones((1, 3, 1, 1), np.float32)
    assert orc.conv2d(x, w)[0, 0, 0, 0] == 1.0


@pytest.mark.parametrize("stride", [1, 2])
def test_conv_1x1_is_matmul(orc, stride):
    x = rng.uniform(-1, 1, (1, 24, 9, 10)).astype(np.float32)
    w = rng.normal(0, 1, (7, 24, 1, 1)).astype(np.float32)
    y = orc.conv2d(x, w, stride, 0)
    xs = x[0, :, ::stride, ::stride].astype(np.float64)
    ref = (w[:, :, 0, 0].astype(np.float64) @ xs.reshape(24, -1)).reshape(7, *xs.shape[1:])
    np.testing.assert_allclose(y[0], ref, rtol=2e-7, atol=1e-7)


@pytest.mark.parametrize("R,S,st,pd,r0,s0", [(3, 3, (1, 1), (1, 1), 0, 2),
                                             (3, 3, (2, 2), (1, 1), 2, 1),
                                             (1, 7, (1, 1), (0, 3), 0, 5),
                                             (7, 1, (2, 1), (3, 0), 6, 0),
                                             (5, 5, (1, 2), (2, 2), 1, 3)])
def test_conv_delta_kernel_is_shift(orc, R, S, st, pd, r0, s0):
    """w[k,c,r,s] = [k==c][r==r0][s==s0] picks x[c, oh*sh-ph+r0, ow*sw-pw+s0] (bit-exact)."""
    C, H, W = 3, 11, 9
    x = rng.uniform(-1, 1, (2, C, H, W)).astype(np.float32)
    w = np.zeros((C, C, R, S), np.float32)
    for c in range(C):
        w[c, c, r0, s0] = 1
    y = orc.conv2d(x, w, st, pd)
    N, K, OH, OW = y.shape
    for oh, ow in itertools.product(range(OH), range(OW)):
        ih, iw = oh * st[0] - pd[0] + r0, ow * st[1] - pd[1] + s0
        want = x[:, :, ih, iw] if (0 <= ih < H and 0 <= iw < W) else np.zeros((2, C), np.float32)
        np.testing.assert_array_equal(y[:, :, oh, ow], want)


def test_conv_linearity(orc):
    x1 = rng.uniform(-1, 1, (1, 6, 8, 8)).astype(np.float32)
    x2 = rng.uniform(-1, 1, (1, 6, 8, 8)).astype(np.float32)
    w1 = rng.normal(0, 1, (5, 6, 3, 3)).astype(np.float32)
    w2 = rng.normal(0, 1, (5, 6, 3, 3)).astype(np.float32)
    lhs = orc.conv2d(x1 + x2, w1, 1, 1)
    np.testing.assert_allclose(lhs, orc.conv2d(x1, w1, 1, 1).astype(np.float64)
                               + orc.conv2d(x2, w1, 1, 1), rtol=1e-5, atol=2e-6)
    lhs = orc.conv2d(x1, w1 + w2, 1, 1)
    np.testing.assert_allclose(lhs, orc.conv2d(x1, w1, 1, 1).astype(np.float64)
                               + orc.conv2d(x1, w2, 1, 1), rtol=1e-5, atol=2e-6)


def test_conv_zero_pad_equivalence(orc):
    x = rng.uniform(-1, 1, (2, 4, 7, 6)).astype(np.float32)
    w = rng.normal(0, 1, (3, 4, 3, 5)).astype(np.float32)
    a = orc.conv2d(x, w, (2, 1), (1, 2))
    b = orc.conv2d(np.pad(x, ((0, 0), (0, 0), (1, 1), (2, 2))), w, (2, 1), (0, 0))
    np.testing.assert_array_equal(a, b)


def test_maxpool_hand(orc):
    x = np.arange(16, dtype=np.float32).reshape(1, 1, 4, 4)
    np.testing.assert_array_equal(orc.maxpool2d(x, 2, 2, 2)[0, 0], [[5, 7], [13, 15]])
    # 3x3/s2/p1 windows: rows/cols {0,1}, {0,1} x {1,2,3}, ...; padding must not
    # win over the negative values
    y = orc.maxpool2d(-x, 3, 3, 2, 1)
    np.testing.assert_array_equal(y[0, 0], [[0, -1], [-4, -5]])


def test_avgpool_counts_in_bounds_taps(orc):
    x = np.arange(9, dtype=np.float32).reshape(1, 1, 3, 3)
    y = orc.avgpool2d(x, 3, 3, 1, 1)
    assert y[0, 0, 0, 0] == np.float32((0 + 1 + 3 + 4) / 4)
    assert y[0, 0, 1, 1] == np.float32(4.0)
    assert y[0, 0, 0, 1] == np.float32((0 + 1 + 2 + 3 + 4 + 5) / 6)
    ones = np.ones((1, 2, 5, 5), np.float32)
    np.testing.assert_array_equal(orc.avgpool2d(ones, 3, 3, 1, 1), ones)


def test_global_avgpool(orc):
    x = rng.uniform(-1, 1, (2, 3, 7, 5)).astype(np.float32)
    y = orc.global_avgpool(x)
    np.testing.assert_allclose(y[:, :, 0, 0], x.astype(np.float64).mean(axis=(2, 3)),
                               rtol=2e-7, atol=1e-8)


def test_dense_matches_matmul(orc):
    x = rng.uniform(-1, 1, (3, 40)).astype(np.float32)
    w = rng.normal(0, 1, (9, 40)).astype(np.float32)
    b = rng.normal(0, 1, 9).astype(np.float32)
    ref = x.astype(np.float64) @ w.astype(np.float64).T + b
    np.testing.assert_allclose(orc.dense(x, w, b), ref, rtol=2e-7, atol=1e-7)


def test_batchnorm_closed_form(orc):
    y = rng.uniform(-1, 1, (1, 3, 2, 2)).astype(np.float32)
    # mean 0, var 1 - eps, gamma 1, beta 0 -> identity
    out = orc.batchnorm(y, np.ones(3), np.zeros(3), np.zeros(3), np.full(3, 1 - 1e-5), 1e-5)
    np.testing.assert_array_equal(out, y)
    # var + eps = 4, gamma 2 -> (y - mean), then + beta
    out = orc.batchnorm(y, np.full(3, 2.0), np.array([1., 2., 3.]), np.full(3, 0.5),
                        np.full(3, 4.0 - 1e-5), 1e-5)
    ref = (y.astype(np.float64) - 0.5) + np.array([1., 2., 3.]).reshape(1, 3, 1, 1)
    np.testing.assert_allclose(out, ref, rtol=1e-7, atol=1e-7)


def test_relu_add(orc):
    a = np.array([-1.5, 0.0, 2.0], np.float32)
    np.testing.assert_array_equal(orc.relu(a), [0, 0, 2])
    np.testing.assert_array_equal(orc.add(a, a), [-3, 0, 4])


# ---- layout maps (Section 3.1.1): explicit index loops on tiny tensors ----------------------
@pytest.mark.parametrize("C,block", [(1, 16), (3, 16), (5, 4), (16, 16), (17, 16), (33, 16),
                                     (48, 32), (80, 32)])
def test_to_blocked_index_map(orc, C, block):
    N, H, W = 2, 3, 4
    x = rng.uniform(-1, 1, (N, C, H, W)).astype(np.float32)
    xb = orc.to_blocked(x, block)
    CB = -(-C // block)
    assert xb.shape == (N, CB, H, W, block)
    for n, c, h, w in itertools.product(range(N), range(CB * block), range(H), range(W)):
        v = xb[n, c // block, h, w, c % block]
        if c < C:
            assert v == x[n, c, h, w]
        else:
            assert v == 0 and not np.signbit(v)
    np.testing.assert_array_equal(orc.from_blocked(xb, C), x)


def test_pack_filter_index_map(orc):
    K, C, R, S = 20, 5, 3, 2
    w = rng.normal(0, 1, (K, C, R, S)).astype(np.float32)
    wp = orc.pack_filter(w, 4, 16)
    assert wp.shape == (2, 2, R, S, 4, 16)
    for k, c, r, s in itertools.product(range(32), range(8), range(R), range(S)):
        v = wp[k // 16, c // 4, r, s, c % 4, k % 16]
        assert v == (w[k, c, r, s] if (k < K and c < C) else 0)
