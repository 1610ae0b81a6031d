"""Invariants of the synthetic network descriptions against the published
architecture sizes: parameter counts, convolution counts, distinct
convolution shapes and convolution FLOPs."""
import numpy as np
import pytest

from paper_1809_02697_amd import workloads as wl

import nets


def _out(n, k, s, p):
    return (n + 2 * p - k) // s + 1


def walk(g):
    """Shapes (C, H, W) per node and the list of conv shape keys."""
    N, C, H, W = g.input_shape
    shp = []
    convs = []
    for n in g.nodes:
        ins = [shp[i] for i in n.inputs]
        if n.op == "input":
            s = (C, H, W)
        elif n.op == "conv":
            c, h, w = ins[0]
            assert n.w.shape == (n.K, c, n.R, n.S)
            oh, ow = _out(h, n.R, n.stride[0], n.pad[0]), _out(w, n.S, n.stride[1], n.pad[1])
            convs.append((c, n.K, n.R, n.S, n.stride, n.pad, h, w, oh, ow))
            s = (n.K, oh, ow)
            if n.residual >= 0:
                assert shp[n.residual] == s
        elif n.op in ("maxpool", "avgpool"):
            c, h, w = ins[0]
            s = (c, _out(h, n.R, n.stride[0], n.pad[0]), _out(w, n.S, n.stride[1], n.pad[1]))
        elif n.op == "gap":
            s = (ins[0][0], 1, 1)
        elif n.op == "concat":
            assert len({x[1:] for x in ins}) == 1
            s = (sum(x[0] for x in ins),) + ins[0][1:]
        elif n.op == "flatten":
            s = (int(np.prod(ins[0])), 1, 1)
        elif n.op == "dense":
            assert n.w.shape == (n.K, ins[0][0])
            s = (n.K, 1, 1)
        else:
            s = ins[0]
        shp.append(s)
    return shp, convs


def n_params(g, bn_running=False):
    t = 0
    for n in g.nodes:
        if n.w is not None:
            t += n.w.size
        if n.bias is not None:
            t += n.bias.size
        if n.bn is not None:
            t += 2 * n.K + (2 * n.K if bn_running else 0)
    return t


def conv_flops(convs, N=1):
    return sum(2 * N * k * c * r * s * oh * ow for (c, k, r, s, _, _, _, _, oh, ow) in convs)


@pytest.fixture(scope="module")
def r50():
    return nets.resnet50()


def test_resnet50_invariants(r50):
    shp, convs = walk(r50)
    assert len(convs) == 53
    assert len(set(convs)) == 23
    assert conv_flops(convs) == 8_174_272_512
    assert n_params(r50) == 25_557_032
    assert shp[-1] == (1000, 1, 1)
    assert r50.x.shape == (1, 3, 224, 224) and r50.x.dtype == np.float32


def test_resnet50_distinct_shapes_are_the_layer_sweep(r50):
    _, convs = walk(r50)
    sweep = {(C, K, R, R, (s, s), (p, p), H, H) for (_, C, K, R, s, p, H, _, _) in
             wl.RESNET50_LAYERS}
    assert {c[:8] for c in convs} == sweep
    uses = {}
    for c in convs:
        uses[c[:8]] = uses.get(c[:8], 0) + 1
    for (_, C, K, R, s, p, H, _, u) in wl.RESNET50_LAYERS:
        assert uses[(C, K, R, R, (s, s), (p, p), H, H)] == u


def test_vgg16_invariants():
    g = nets.vgg16()
    shp, convs = walk(g)
    assert len(convs) == 13 and len(set(convs)) == 9
    assert conv_flops(convs) == 30_693_261_312
    assert n_params(g) == 138_357_544
    assert shp[-1] == (1000, 1, 1)


def test_inception_v3_invariants():
    g = nets.inception_v3()
    shp, convs = walk(g)
    assert len(convs) == 94
    assert len(set(convs)) == 43
    assert conv_flops(convs) == 11_422_336_192
    widths = [shp[i][0] for i in g.node_ids("concat")]
    assert sorted(set(widths)) == [256, 288, 768, 1280, 2048]
    # every concat part is a whole number of 16-channel blocks
    for i in g.node_ids("concat"):
        for j in g.nodes[i].inputs:
            assert shp[j][0] % 16 == 0
    # torchvision's Inception-v3 has 27,161,264 parameters including the
    # auxiliary head (3,326,696), which this description leaves out
    assert n_params(g) == 27_161_264 - 3_326_696
    assert shp[-1] == (1000, 1, 1)


def test_seeded_draws_are_deterministic():
    a, b = wl.single_conv(0), wl.single_conv(0)
    np.testing.assert_array_equal(a.x, b.x)
    np.testing.assert_array_equal(a.nodes[1].w, b.nodes[1].w)
    c = a.nodes[1]
    assert a.x.shape == (1, 64, 56, 56) and c.w.shape == (64, 64, 3, 3)
    assert -1 <= a.x.min() and a.x.max() <= 1
    assert abs(c.w.std() - np.sqrt(2 / 576)) < 0.002
    sweep = wl.resnet50_layer_sweep()
    assert len(sweep) == 23 and sweep[3].residual.shape == (1, 256, 56, 56)
