"""Seeded synthetic workloads: network descriptions, parameters and inputs.

This module is the only code shared by the HIP path and the CPU oracle.  It
holds no arithmetic of the method: it draws random numbers and records which
operation consumes which tensor.  Convolution, folding, pooling, layout
changes and output shapes are computed by each side on its own.

Networks are the standard architecture definitions of the models the paper
evaluates (Section 4, Table 2): ResNet-50, VGG-16 and Inception-v3.  Trained
weights are not available, so every parameter is drawn at random:

* Draws use ``numpy.random.Generator(PCG64(seed))`` in float64 and are cast
  once to float32.
* Parameters are drawn in node order; for each node: weights, then either the
  batch-norm statistics (gamma, beta, mean, var) or the bias; the input is
  drawn last.
* Convolution and dense weights are Kaiming-normal: std = sqrt(2 / fan_in),
  fan_in = C*R*S (in_features for a dense layer).
* Batch norm: gamma ~ U[0.5, 1.5], beta ~ N(0, 0.1), mean ~ N(0, 0.1),
  var ~ U[0.5, 1.5], eps = 1e-5.  Biases not given by a configuration are
  N(0, 0.1).

Node semantics (what a node computes is defined by the oracle; the fields
here only name the operands):

``conv``      t = conv(x, w) [+ bias] -> [batch norm] -> [+ residual] -> [relu]
``maxpool``   window (R, S), stride, zero-size padding treated as -inf
``avgpool``   window (R, S), stride, pad; divides by the in-bounds tap count
``gap``       global average pool to 1x1
``concat``    channel concatenation of ``inputs`` in order
``flatten``   (N, C, H, W) -> (N, C*H*W), c-major
``dense``     y = W x + b, W stored [out][in] [-> relu]
``output``    marks the network output
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

BN_EPS = 1e-5


@dataclass
class Node:
    op: str
    inputs: tuple = ()
    name: str = ""
    K: int = 0              # conv: output channels; dense: out_features
    R: int = 1              # conv / pool window height
    S: int = 1              # conv / pool window width
    stride: tuple = (1, 1)
    pad: tuple = (0, 0)
    act: str = "none"       # "none" | "relu"
    residual: int = -1      # conv: id of the node added before the activation
    w: Optional[np.ndarray] = None      # conv (K, C, R, S); dense (out, in)
    bias: Optional[np.ndarray] = None   # (K,)
    bn: Optional[dict] = None           # gamma, beta, mean, var (K,), eps


@dataclass
class Graph:
    name: str
    nodes: list = field(default_factory=list)
    input_shape: tuple = (1, 3, 224, 224)
    x: Optional[np.ndarray] = None

    def node_ids(self, op):
        return [i for i, n in enumerate(self.nodes) if n.op == op]


def _f32(a):
    return np.asarray(a, dtype=np.float64).astype(np.float32)


class _Builder:
    """Appends nodes and draws their parameters in node order.

    Tracks only channel counts (needed to size weights)."""

    def __init__(self, name, input_shape, rng):
        self.g = Graph(name=name, input_shape=tuple(input_shape))
        self.rng = rng
        self.ch = []
        self.add("input", (), C=input_shape[1])

    def add(self, op, inputs, C, **kw):
        self.g.nodes.append(Node(op=op, inputs=tuple(inputs), **kw))
        self.ch.append(C)
        return len(self.g.nodes) - 1

    def kaiming(self, shape, fan_in):
        return _f32(self.rng.normal(0.0, np.sqrt(2.0 / fan_in), size=shape))

    def bn_params(self, K):
        r = self.rng
        return dict(gamma=_f32(r.uniform(0.5, 1.5, K)), beta=_f32(r.normal(0.0, 0.1, K)),
                    mean=_f32(r.normal(0.0, 0.1, K)), var=_f32(r.uniform(0.5, 1.5, K)),
                    eps=BN_EPS)

    def conv(self, x, K, R, S=None, stride=1, pad=0, bn=True, bias=False, act="relu",
             residual=-1, name=""):
        S = R if S is None else S
        st = stride if isinstance(stride, tuple) else (stride, stride)
        pd = pad if isinstance(pad, tuple) else (pad, pad)
        C = self.ch[x]
        w = self.kaiming((K, C, R, S), C * R * S)
        b = _f32(self.rng.normal(0.0, 0.1, K)) if bias else None
        bnp = self.bn_params(K) if bn else None
        return self.add("conv", (x,), K, name=name, K=K, R=R, S=S, stride=st, pad=pd,
                        act=act, residual=residual, w=w, bias=b, bn=bnp)

    def pool(self, op, x, R, stride, pad=0, name=""):
        pd = pad if isinstance(pad, tuple) else (pad, pad)
        return self.add(op, (x,), self.ch[x], name=name, R=R, S=R, stride=(stride, stride),
                        pad=pd)

    def gap(self, x):
        return self.add("gap", (x,), self.ch[x], name="gap")

    def concat(self, xs, name=""):
        return self.add("concat", tuple(xs), sum(self.ch[i] for i in xs), name=name)

    def flatten(self, x, features):
        return self.add("flatten", (x,), features, name="flatten")

    def dense(self, x, K, act="none", name=""):
        fan_in = self.ch[x]
        w = self.kaiming((K, fan_in), fan_in)
        b = _f32(self.rng.normal(0.0, 0.1, K))
        return self.add("dense", (x,), K, name=name, K=K, w=w, bias=b, act=act)

    def output(self, x):
        return self.add("output", (x,), self.ch[x], name="output")

    def finish(self, x_draw):
        self.g.x = x_draw(self.rng)
        return self.g


def _normal_input(shape):
    return lambda rng: _f32(rng.normal(0.0, 1.0, size=shape))


# ----------------------------------------------------------------------------------------
# Configuration 1: one 3x3 convolution with bias + ReLU.
# ----------------------------------------------------------------------------------------
def single_conv(seed=0):
    """N=1, C=K=64, 56x56, 3x3/s1/p1, bias + ReLU.

    x ~ U[-1, 1], w ~ N(0, sqrt(2/(64*9))), bias ~ N(0, 0.1)."""
    b = _Builder("single_conv", (1, 64, 56, 56), np.random.Generator(np.random.PCG64(seed)))
    c = b.conv(0, 64, 3, stride=1, pad=1, bn=False, bias=True, act="relu", name="conv")
    b.output(c)
    return b.finish(lambda rng: _f32(rng.uniform(-1.0, 1.0, size=(1, 64, 56, 56))))


# ----------------------------------------------------------------------------------------
# Configuration 2: the distinct ResNet-50 convolution shapes at batch 1.
# ----------------------------------------------------------------------------------------
# (id, C, K, R, stride, pad, H_in, epilogue, uses in the network)
# epilogue: "relu" = BN + ReLU, "res" = BN + residual + ReLU, "none" = BN only.
RESNET50_LAYERS = [
    ("R01", 3, 64, 7, 2, 3, 224, "relu", 1),
    ("R02", 64, 64, 1, 1, 0, 56, "relu", 1),
    ("R03", 64, 64, 3, 1, 1, 56, "relu", 3),
    ("R04", 64, 256, 1, 1, 0, 56, "res", 4),
    ("R05", 256, 64, 1, 1, 0, 56, "relu", 2),
    ("R06", 256, 128, 1, 1, 0, 56, "relu", 1),
    ("R07", 128, 128, 3, 2, 1, 56, "relu", 1),
    ("R08", 128, 512, 1, 1, 0, 28, "res", 4),
    ("R09", 256, 512, 1, 2, 0, 56, "none", 1),
    ("R10", 512, 128, 1, 1, 0, 28, "relu", 3),
    ("R11", 128, 128, 3, 1, 1, 28, "relu", 3),
    ("R12", 512, 256, 1, 1, 0, 28, "relu", 1),
    ("R13", 256, 256, 3, 2, 1, 28, "relu", 1),
    ("R14", 256, 1024, 1, 1, 0, 14, "res", 6),
    ("R15", 512, 1024, 1, 2, 0, 28, "none", 1),
    ("R16", 1024, 256, 1, 1, 0, 14, "relu", 5),
    ("R17", 256, 256, 3, 1, 1, 14, "relu", 5),
    ("R18", 1024, 512, 1, 1, 0, 14, "relu", 1),
    ("R19", 512, 512, 3, 2, 1, 14, "relu", 1),
    ("R20", 512, 2048, 1, 1, 0, 7, "res", 3),
    ("R21", 1024, 2048, 1, 2, 0, 14, "none", 1),
    ("R22", 2048, 512, 1, 1, 0, 7, "relu", 2),
    ("R23", 512, 512, 3, 1, 1, 7, "relu", 2),
]


@dataclass
class LayerCase:
    """One convolution with its operands, drawn on a per-layer stream."""
    id: str
    C: int
    K: int
    R: int
    S: int
    stride: tuple
    pad: tuple
    H: int
    W: int
    N: int
    epilogue: str           # "relu" | "res" | "none" | "bias_relu"
    uses: int
    x: np.ndarray
    w: np.ndarray
    bias: Optional[np.ndarray]
    bn: Optional[dict]
    residual_shape: Optional[tuple]
    residual: Optional[np.ndarray] = None


def _layer_case(lid, C, K, R, S, stride, pad, H, W, epi, uses, rng, N=1, stem=False,
                out_hw=None):
    w = _f32(rng.normal(0.0, np.sqrt(2.0 / (C * R * S)), size=(K, C, R, S)))
    r = rng
    bn = dict(gamma=_f32(r.uniform(0.5, 1.5, K)), beta=_f32(r.normal(0.0, 0.1, K)),
              mean=_f32(r.normal(0.0, 0.1, K)), var=_f32(r.uniform(0.5, 1.5, K)), eps=BN_EPS)
    if stem:
        x = _f32(rng.normal(0.0, 1.0, size=(N, C, H, W)))
    else:
        x = _f32(rng.uniform(-1.0, 1.0, size=(N, C, H, W)))
    case = LayerCase(lid, C, K, R, S, (stride, stride), (pad, pad), H, W, N, epi, uses,
                     x, w, None, bn, None)
    if epi == "res":
        # The residual has the output's shape; for these layers (1x1, stride 1)
        # the output's spatial size is the input's.
        assert out_hw is not None
        case.residual_shape = (N, K) + tuple(out_hw)
        case.residual = _f32(rng.uniform(-1.0, 1.0, size=case.residual_shape))
    return case


def resnet50_layer_sweep(seed=1, N=1):
    """The 23 distinct ResNet-50 convolution shapes (stride on the 3x3 and on
    the projection), batch N.  Layer i draws from its own stream
    ``default_rng([seed, i])``: weights, batch norm, input, residual."""
    cases = []
    for i, (lid, C, K, R, st, pd, H, epi, uses) in enumerate(RESNET50_LAYERS):
        rng = np.random.default_rng([seed, i])
        cases.append(_layer_case(lid, C, K, R, R, st, pd, H, H, epi, uses, rng, N=N,
                                 stem=(lid == "R01"), out_hw=(H, H) if epi == "res" else None))
    return cases


def conv_case(C, K, R, S, stride, pad, H, W, N=1, epilogue="relu", seed=0, with_bn=True,
              out_hw=None):
    """A generic convolution case for tests (ragged shapes, asymmetric kernels).

    ``out_hw`` must be given when ``epilogue == "res"``."""
    rng = np.random.default_rng([seed, C, K, R, S, H, W, N])
    st = stride if isinstance(stride, tuple) else (stride, stride)
    pd = pad if isinstance(pad, tuple) else (pad, pad)
    w = _f32(rng.normal(0.0, np.sqrt(2.0 / (C * R * S)), size=(K, C, R, S)))
    bias = _f32(rng.normal(0.0, 0.1, K))
    bn = None
    if with_bn:
        bn = dict(gamma=_f32(rng.uniform(0.5, 1.5, K)), beta=_f32(rng.normal(0.0, 0.1, K)),
                  mean=_f32(rng.normal(0.0, 0.1, K)), var=_f32(rng.uniform(0.5, 1.5, K)),
                  eps=BN_EPS)
    x = _f32(rng.uniform(-1.0, 1.0, size=(N, C, H, W)))
    case = LayerCase("case", C, K, R, S, st, pd, H, W, N, epilogue, 1, x, w, bias, bn, None)
    if epilogue == "res":
        case.residual_shape = (N, K) + tuple(out_hw)
        case.residual = _f32(rng.uniform(-1.0, 1.0, size=case.residual_shape))
    return case


# ----------------------------------------------------------------------------------------
# Configuration 3: ResNet-50 (stride on the 3x3 of each downsampling bottleneck).
# ----------------------------------------------------------------------------------------
def resnet50(N=1, seed=2, num_classes=1000):
    b = _Builder("resnet50", (N, 3, 224, 224), np.random.Generator(np.random.PCG64(seed)))
    x = b.conv(0, 64, 7, stride=2, pad=3, name="conv1")
    x = b.pool("maxpool", x, 3, 2, 1, name="maxpool")
    inplanes = 64
    for si, (width, blocks, stride) in enumerate([(64, 3, 1), (128, 4, 2), (256, 6, 2),
                                                 (512, 3, 2)]):
        for bi in range(blocks):
            s = stride if bi == 0 else 1
            pre = f"layer{si + 1}.{bi}"
            if bi == 0:
                sc = b.conv(x, width * 4, 1, stride=s, pad=0, act="none", name=pre + ".down")
            else:
                sc = x
            y = b.conv(x, width, 1, name=pre + ".conv1")
            y = b.conv(y, width, 3, stride=s, pad=1, name=pre + ".conv2")
            x = b.conv(y, width * 4, 1, act="relu", residual=sc, name=pre + ".conv3")
            inplanes = width * 4
    x = b.gap(x)
    x = b.flatten(x, inplanes)
    x = b.dense(x, num_classes, name="fc")
    b.output(x)
    return b.finish(_normal_input((N, 3, 224, 224)))


# ----------------------------------------------------------------------------------------
# Configuration 4: VGG-16 (no batch norm, conv bias, dropout = identity at inference).
# ----------------------------------------------------------------------------------------
VGG16_CFG = [64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M",
             512, 512, 512, "M"]


def vgg16(N=1, seed=3, num_classes=1000):
    b = _Builder("vgg16", (N, 3, 224, 224), np.random.Generator(np.random.PCG64(seed)))
    x = 0
    li = 0
    for v in VGG16_CFG:
        if v == "M":
            x = b.pool("maxpool", x, 2, 2, 0, name=f"pool{li}")
        else:
            li += 1
            x = b.conv(x, v, 3, stride=1, pad=1, bn=False, bias=True, name=f"conv{li}")
    x = b.flatten(x, 512 * 7 * 7)
    x = b.dense(x, 4096, act="relu", name="fc6")
    x = b.dense(x, 4096, act="relu", name="fc7")
    x = b.dense(x, num_classes, name="fc8")
    b.output(x)
    return b.finish(_normal_input((N, 3, 224, 224)))


# ----------------------------------------------------------------------------------------
# Configuration 5: Inception-v3 (no auxiliary head), 299x299.
# ----------------------------------------------------------------------------------------
def inception_v3(N=1, seed=4, num_classes=1000):
    b = _Builder("inception_v3", (N, 3, 299, 299), np.random.Generator(np.random.PCG64(seed)))
    c = b.conv
    x = c(0, 32, 3, stride=2, name="Conv2d_1a_3x3")
    x = c(x, 32, 3, name="Conv2d_2a_3x3")
    x = c(x, 64, 3, pad=1, name="Conv2d_2b_3x3")
    x = b.pool("maxpool", x, 3, 2, name="maxpool1")
    x = c(x, 80, 1, name="Conv2d_3b_1x1")
    x = c(x, 192, 3, name="Conv2d_4a_3x3")
    x = b.pool("maxpool", x, 3, 2, name="maxpool2")

    def block_a(x, pool_features, p):
        b1 = c(x, 64, 1, name=p + ".branch1x1")
        b5 = c(x, 48, 1, name=p + ".branch5x5_1")
        b5 = c(b5, 64, 5, pad=2, name=p + ".branch5x5_2")
        b3 = c(x, 64, 1, name=p + ".branch3x3dbl_1")
        b3 = c(b3, 96, 3, pad=1, name=p + ".branch3x3dbl_2")
        b3 = c(b3, 96, 3, pad=1, name=p + ".branch3x3dbl_3")
        bp = b.pool("avgpool", x, 3, 1, 1, name=p + ".avgpool")
        bp = c(bp, pool_features, 1, name=p + ".branch_pool")
        return b.concat([b1, b5, b3, bp], name=p)

    def block_b(x, p):
        b3 = c(x, 384, 3, stride=2, name=p + ".branch3x3")
        bd = c(x, 64, 1, name=p + ".branch3x3dbl_1")
        bd = c(bd, 96, 3, pad=1, name=p + ".branch3x3dbl_2")
        bd = c(bd, 96, 3, stride=2, name=p + ".branch3x3dbl_3")
        bp = b.pool("maxpool", x, 3, 2, name=p + ".maxpool")
        return b.concat([b3, bd, bp], name=p)

    def block_c(x, c7, p):
        b1 = c(x, 192, 1, name=p + ".branch1x1")
        b7 = c(x, c7, 1, name=p + ".branch7x7_1")
        b7 = c(b7, c7, 1, 7, pad=(0, 3), name=p + ".branch7x7_2")
        b7 = c(b7, 192, 7, 1, pad=(3, 0), name=p + ".branch7x7_3")
        bd = c(x, c7, 1, name=p + ".branch7x7dbl_1")
        bd = c(bd, c7, 7, 1, pad=(3, 0), name=p + ".branch7x7dbl_2")
        bd = c(bd, c7, 1, 7, pad=(0, 3), name=p + ".branch7x7dbl_3")
        bd = c(bd, c7, 7, 1, pad=(3, 0), name=p + ".branch7x7dbl_4")
        bd = c(bd, 192, 1, 7, pad=(0, 3), name=p + ".branch7x7dbl_5")
        bp = b.pool("avgpool", x, 3, 1, 1, name=p + ".avgpool")
        bp = c(bp, 192, 1, name=p + ".branch_pool")
        return b.concat([b1, b7, bd, bp], name=p)

    def block_d(x, p):
        b3 = c(x, 192, 1, name=p + ".branch3x3_1")
        b3 = c(b3, 320, 3, stride=2, name=p + ".branch3x3_2")
        b7 = c(x, 192, 1, name=p + ".branch7x7x3_1")
        b7 = c(b7, 192, 1, 7, pad=(0, 3), name=p + ".branch7x7x3_2")
        b7 = c(b7, 192, 7, 1, pad=(3, 0), name=p + ".branch7x7x3_3")
        b7 = c(b7, 192, 3, stride=2, name=p + ".branch7x7x3_4")
        bp = b.pool("maxpool", x, 3, 2, name=p + ".maxpool")
        return b.concat([b3, b7, bp], name=p)

    def block_e(x, p):
        b1 = c(x, 320, 1, name=p + ".branch1x1")
        b3 = c(x, 384, 1, name=p + ".branch3x3_1")
        b3a = c(b3, 384, 1, 3, pad=(0, 1), name=p + ".branch3x3_2a")
        b3b = c(b3, 384, 3, 1, pad=(1, 0), name=p + ".branch3x3_2b")
        b3 = b.concat([b3a, b3b], name=p + ".branch3x3")
        bd = c(x, 448, 1, name=p + ".branch3x3dbl_1")
        bd = c(bd, 384, 3, pad=1, name=p + ".branch3x3dbl_2")
        bda = c(bd, 384, 1, 3, pad=(0, 1), name=p + ".branch3x3dbl_3a")
        bdb = c(bd, 384, 3, 1, pad=(1, 0), name=p + ".branch3x3dbl_3b")
        bd = b.concat([bda, bdb], name=p + ".branch3x3dbl")
        bp = b.pool("avgpool", x, 3, 1, 1, name=p + ".avgpool")
        bp = c(bp, 192, 1, name=p + ".branch_pool")
        return b.concat([b1, b3, bd, bp], name=p)

    x = block_a(x, 32, "Mixed_5b")
    x = block_a(x, 64, "Mixed_5c")
    x = block_a(x, 64, "Mixed_5d")
    x = block_b(x, "Mixed_6a")
    for p, c7 in (("Mixed_6b", 128), ("Mixed_6c", 160), ("Mixed_6d", 160), ("Mixed_6e", 192)):
        x = block_c(x, c7, p)
    x = block_d(x, "Mixed_7a")
    x = block_e(x, "Mixed_7b")
    x = block_e(x, "Mixed_7c")
    x = b.gap(x)
    x = b.flatten(x, 2048)
    x = b.dense(x, num_classes, name="fc")
    b.output(x)
    return b.finish(_normal_input((N, 3, 299, 299)))


def tiny_graph(seed=7, N=2, C=5, H=13, W=11):
    """A small network with every node kind, for fast tests: a ragged-channel
    stem, a residual bottleneck, both pools, a concat of odd-width branches, GAP
    and a dense head."""
    b = _Builder("tiny", (N, C, H, W), np.random.Generator(np.random.PCG64(seed)))
    x = b.conv(0, 32, 3, stride=1, pad=1, name="stem")
    x = b.pool("maxpool", x, 3, 2, 1, name="pool")
    sc = b.conv(x, 48, 1, act="none", name="down")
    y = b.conv(x, 16, 1, name="c1")
    y = b.conv(y, 16, 3, pad=1, name="c2")
    x = b.conv(y, 48, 1, residual=sc, name="c3")
    p1 = b.conv(x, 16, 1, 3, pad=(0, 1), name="b1")
    p2 = b.conv(x, 32, 3, 1, pad=(1, 0), name="b2")
    p3 = b.pool("avgpool", x, 3, 1, 1, name="ap")
    x = b.concat([p1, p2, p3], name="cat")
    x = b.conv(x, 64, 3, stride=2, pad=1, bias=True, bn=False, name="c4")
    x = b.gap(x)
    x = b.flatten(x, 64)
    x = b.dense(x, 10, name="fc")
    b.output(x)
    return b.finish(_normal_input((N, C, H, W)))


def stem_graph(seed=9, N=1, C=3, H=224, W=224, K=64, R=7, S=None, stride=2, pad=3,
               pool=(3, 2, 1), input_dist="normal"):
    """A network stem alone: conv (batch norm, ReLU) and the max pooling that
    reads it, as the network output.  pool = (window, stride, pad)."""
    b = _Builder("stem", (N, C, H, W), np.random.Generator(np.random.PCG64(seed)))
    x = b.conv(0, K, R, S, stride=stride, pad=pad, name="stem")
    x = b.pool("maxpool", x, pool[0], pool[1], pool[2], name="pool")
    b.output(x)
    if input_dist == "uniform":
        return b.finish(lambda rng: _f32(rng.uniform(-1.0, 1.0, size=(N, C, H, W))))
    return b.finish(_normal_input((N, C, H, W)))


def pointwise_graph(seed=10, N=2, C=64, H=56, W=56, K=64, residual=False):
    """One 1x1 conv (batch norm, ReLU) over the input, with, when `residual`,
    another 1x1 conv of the input (batch norm, no activation) added to it
    before the ReLU."""
    b = _Builder("pointwise", (N, C, H, W), np.random.Generator(np.random.PCG64(seed)))
    sc = b.conv(0, K, 1, act="none", name="shortcut") if residual else -1
    x = b.conv(0, K, 1, residual=sc, name="pointwise")
    b.output(x)
    return b.finish(lambda rng: _f32(rng.uniform(-1.0, 1.0, size=(N, C, H, W))))


def vgg_like_tiny(seed=8, N=2):
    """A small plain network whose flatten follows a real spatial map (so the
    exit transform is a real permutation), with two dense layers."""
    b = _Builder("vgg_tiny", (N, 3, 16, 16), np.random.Generator(np.random.PCG64(seed)))
    x = b.conv(0, 16, 3, pad=1, bn=False, bias=True, name="conv1")
    x = b.pool("maxpool", x, 2, 2, name="pool1")
    x = b.conv(x, 32, 3, pad=1, bn=False, bias=True, name="conv2")
    x = b.pool("maxpool", x, 2, 2, name="pool2")
    x = b.flatten(x, 32 * 4 * 4)
    x = b.dense(x, 64, act="relu", name="fc1")
    x = b.dense(x, 10, name="fc2")
    b.output(x)
    return b.finish(_normal_input((N, 3, 16, 16)))


MODELS = {
    "resnet50": resnet50,
    "vgg16": vgg16,
    "inception_v3": inception_v3,
}
