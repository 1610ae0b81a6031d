"""CPU oracle for blocked-layout CNN inference -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct implementation of what the HIP path
computes, written from the paper's statement of the problem, in the default
NCHW layout:

* ``conv2d`` -- the convolution of Section 3.1.1 (sliding window, element-wise
  product, accumulation over input channel, kernel height and kernel width),
  in C with double accumulation (``oracle.c``).
* ``batchnorm`` / ``bias_add`` / ``add`` / ``relu`` -- the memory-bound
  operations the paper fuses into the convolution (Section 2.2 and the
  inherited graph optimizations of Section 3), each applied separately and
  unfolded, in float64 with one rounding to float32.
* pools, ``concat``, ``flatten``, ``dense`` -- the remaining operators of the
  evaluated networks (Section 4).
* ``to_blocked`` / ``from_blocked`` / ``pack_filter`` -- the NCHW[x]c and
  KCRS[x]c[y]k layouts of Section 3.1.1 as closed-form index maps.
* ``run_graph`` -- a reference graph executor: node by node in NCHW, with
  float32 storage between operations, as any float32 framework would run the
  network before the paper's layout optimization.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg use this package.  It shares no code with the HIP library and imports
nothing from it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force=True):
    """Compile ``oracle.c`` into ``liboracle.so`` (gcc, OpenMP, no fast-math)."""
    if not force and os.path.exists(_LIB):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", _SRC,
                           "-o", tmp, "-lm"])
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        I = ctypes.c_int
        lib.orc_conv2d.argtypes = [P, I, I, I, I, P, I, I, I, I, I, I, I, P]
        for f in (lib.orc_maxpool2d, lib.orc_avgpool2d):
            f.argtypes = [P, I, I, I, I, I, I, I, I, I, I, P]
        lib.orc_global_avgpool.argtypes = [P, I, I, I, I, P]
        lib.orc_dense.argtypes = [P, I, I, P, I, P, P]
        lib.orc_num_threads.restype = I
        lib.orc_set_num_threads.argtypes = [I]
        _lib = lib
    return _lib


def num_threads():
    return _load().orc_num_threads()


def set_num_threads(n):
    """Host threads the C operations use from now on (timing only)."""
    _load().orc_set_num_threads(int(n))


def _c(a):
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a, a.ctypes.data_as(ctypes.c_void_p)


def _pair(v):
    return tuple(v) if isinstance(v, (tuple, list)) else (v, v)


def out_size(n, k, s, p):
    """Floor output size of a window of k taps, stride s, symmetric pad p."""
    return (n + 2 * p - k) // s + 1


# --------------------------------------------------------------------------------------
# Operations (NCHW, float32 in / float32 out)
# --------------------------------------------------------------------------------------
def conv2d(x, w, stride=1, pad=0):
    """Cross-correlation with zero padding, double accumulation, one rounding."""
    (sh, sw), (ph, pw) = _pair(stride), _pair(pad)
    x, xp = _c(x)
    w, wp = _c(w)
    N, C, H, W = x.shape
    K, C2, R, S = w.shape
    assert C == C2, (x.shape, w.shape)
    OH, OW = out_size(H, R, sh, ph), out_size(W, S, sw, pw)
    assert OH > 0 and OW > 0
    y = np.empty((N, K, OH, OW), np.float32)
    _load().orc_conv2d(xp, N, C, H, W, wp, K, R, S, sh, sw, ph, pw,
                       y.ctypes.data_as(ctypes.c_void_p))
    return y


def _pool(fn, x, R, S, stride, pad):
    (sh, sw), (ph, pw) = _pair(stride), _pair(pad)
    x, xp = _c(x)
    N, C, H, W = x.shape
    OH, OW = out_size(H, R, sh, ph), out_size(W, S, sw, pw)
    y = np.empty((N, C, OH, OW), np.float32)
    fn(xp, N, C, H, W, R, S, sh, sw, ph, pw, y.ctypes.data_as(ctypes.c_void_p))
    return y


def maxpool2d(x, R, S, stride, pad=0):
    return _pool(_load().orc_maxpool2d, x, R, S, stride, pad)


def avgpool2d(x, R, S, stride, pad=0):
    return _pool(_load().orc_avgpool2d, x, R, S, stride, pad)


def global_avgpool(x):
    x, xp = _c(x)
    N, C, H, W = x.shape
    y = np.empty((N, C, 1, 1), np.float32)
    _load().orc_global_avgpool(xp, N, C, H, W, y.ctypes.data_as(ctypes.c_void_p))
    return y


def dense(x, w, b=None):
    x, xp = _c(x.reshape(x.shape[0], -1))
    w, wp = _c(w)
    N, IN = x.shape
    OUT, IN2 = w.shape
    assert IN == IN2
    bp = None
    if b is not None:
        b, bp = _c(b)
    y = np.empty((N, OUT), np.float32)
    _load().orc_dense(xp, N, IN, wp, OUT, bp, y.ctypes.data_as(ctypes.c_void_p))
    return y


def _chan(v, ndim):
    v = np.asarray(v, np.float64)
    return v.reshape((1, -1) + (1,) * (ndim - 2))


def bias_add(y, b):
    return (y.astype(np.float64) + _chan(b, y.ndim)).astype(np.float32)


def batchnorm(y, gamma, beta, mean, var, eps):
    """Inference batch norm: gamma * (y - mean) / sqrt(var + eps) + beta."""
    nd = y.ndim
    t = (y.astype(np.float64) - _chan(mean, nd)) / np.sqrt(_chan(var, nd) + eps)
    return (_chan(gamma, nd) * t + _chan(beta, nd)).astype(np.float32)


def add(a, b):
    return (a.astype(np.float64) + b.astype(np.float64)).astype(np.float32)


def relu(y):
    return np.where(y > 0, y, np.float32(0)).astype(np.float32)


def concat(xs):
    return np.concatenate(xs, axis=1)


def flatten(x):
    return x.reshape(x.shape[0], -1)


# --------------------------------------------------------------------------------------
# Layout maps of Section 3.1.1 (closed form)
# --------------------------------------------------------------------------------------
def _ceil_to(v, m):
    return -(-v // m) * m


def to_blocked(x, block=16):
    """NCHW -> NCHW[x]c: [N][C/x][H][W][x], channels zero-padded to a multiple of x."""
    N, C, H, W = x.shape
    Cp = _ceil_to(C, block)
    xp = np.zeros((N, Cp, H, W), x.dtype)
    xp[:, :C] = x
    return np.ascontiguousarray(xp.reshape(N, Cp // block, block, H, W).transpose(0, 1, 3, 4, 2))


def from_blocked(xb, C):
    """NCHW[x]c -> NCHW, dropping the padded channels."""
    N, CB, H, W, blk = xb.shape
    return np.ascontiguousarray(xb.transpose(0, 1, 4, 2, 3).reshape(N, CB * blk, H, W)[:, :C])


def pack_filter(w, ic_bn=16, oc_bn=16):
    """KCRS -> KCRS[x]c[y]k: [K/y][C/x][R][S][x][y] (y innermost), zero-padded."""
    K, C, R, S = w.shape
    Kp, Cp = _ceil_to(K, oc_bn), _ceil_to(C, ic_bn)
    wp = np.zeros((Kp, Cp, R, S), w.dtype)
    wp[:K, :C] = w
    return np.ascontiguousarray(
        wp.reshape(Kp // oc_bn, oc_bn, Cp // ic_bn, ic_bn, R, S).transpose(0, 2, 4, 5, 3, 1))


# --------------------------------------------------------------------------------------
# Reference graph executor
# --------------------------------------------------------------------------------------
def conv_node(n, x, residual=None):
    """One conv node of a network description, unfused and unfolded."""
    y = conv2d(x, n.w, n.stride, n.pad)
    if n.bias is not None:
        y = bias_add(y, n.bias)
    if n.bn is not None:
        y = batchnorm(y, n.bn["gamma"], n.bn["beta"], n.bn["mean"], n.bn["var"], n.bn["eps"])
    if residual is not None:
        y = add(y, residual)
    if n.act == "relu":
        y = relu(y)
    return y


def run_graph(graph, x=None, keep=False):
    """Run a network description node by node.  Returns the output, or the
    list of every node's output when ``keep`` is true."""
    x = graph.x if x is None else x
    vals = [None] * len(graph.nodes)
    last_use = list(range(len(graph.nodes)))
    for i, n in enumerate(graph.nodes):
        for j in tuple(n.inputs) + ((n.residual,) if n.residual >= 0 else ()):
            last_use[j] = max(last_use[j], i)
    for i, n in enumerate(graph.nodes):
        ins = [vals[j] for j in n.inputs]
        if n.op == "input":
            v = np.asarray(x, np.float32)
        elif n.op == "conv":
            v = conv_node(n, ins[0], vals[n.residual] if n.residual >= 0 else None)
        elif n.op == "maxpool":
            v = maxpool2d(ins[0], n.R, n.S, n.stride, n.pad)
        elif n.op == "avgpool":
            v = avgpool2d(ins[0], n.R, n.S, n.stride, n.pad)
        elif n.op == "gap":
            v = global_avgpool(ins[0])
        elif n.op == "concat":
            v = concat(ins)
        elif n.op == "flatten":
            v = flatten(ins[0])
        elif n.op == "dense":
            v = dense(ins[0], n.w, n.bias)
            if n.act == "relu":
                v = relu(v)
        elif n.op == "output":
            v = ins[0]
        else:
            raise ValueError("unknown op " + n.op)
        vals[i] = v
        if not keep:
            for j in set(n.inputs) | ({n.residual} if n.residual >= 0 else set()):
                if last_use[j] == i and j != len(graph.nodes) - 1:
                    vals[j] = None
    return vals if keep else vals[-1]


def layer_forward(case):
    """Reference output of one layer case (conv [+bias] [+BN] [+res] [+ReLU])."""
    y = conv2d(case.x, case.w, case.stride, case.pad)
    if case.bias is not None:
        y = bias_add(y, case.bias)
    if case.bn is not None:
        b = case.bn
        y = batchnorm(y, b["gamma"], b["beta"], b["mean"], b["var"], b["eps"])
    if case.epilogue == "res":
        y = add(y, case.residual)
    if case.epilogue in ("relu", "res", "bias_relu"):
        y = relu(y)
    return y
