"""Integer (INT8) convolution, the paper's other future work -- TEST INFRASTRUCTURE ONLY.

The paper names integer (8-bit) inference as future work and gives no
scheme, so this module fixes one, the usual symmetric linear quantization:

* activations: one scale s_x per tensor (given by the caller);
  q = clamp(round_half_even(x / s_x), -127, 127) with the division in float32;
* filters: one scale per output channel, s_w[k] = max |w[k, :, :, :]| / 127
  (float32; 1 for an all-zero channel), q = clamp(round_half_even(w / s_w[k]));
* the convolution of the quantized values accumulates exact integers
  (|sum| <= 127^2 * C * R * S, below 2^31 for every layer here);
* the output is dequantized with the per-channel multiplier m[k] = s_x * s_w[k]
  (a float32 product, the value the library receives):
  y = act(acc * m[k] + bias[k] + residual), in float64, rounded once
  (``dequantize``, the ideal value); ``epilogue_f32`` is the same expression
  evaluated the way the library's interface fixes it, each operation rounded
  to float32 in that order, no fused multiply-add;
* an int8 output (the next layer's input) requantizes that float32 value with
  the next layer's scale s_y: q = clamp(round_half_even(y * r), -127, 127),
  r = 1 / s_y rounded to float32 and the product in float32 (one multiply per
  value; it can differ from x / s_y by one step at an exact tie).

Integer inference of a whole network (``run_graph_int8``): every conv's
input has the scale max |x| / 127 of the float32 tensor it reads
(calibrated on the run itself) and is quantized by division, except an
input that is the output of a conv: that conv writes it requantized (by the
reciprocal, as above), one int8 tensor shared by every conv that reads it,
whatever their paddings (the padding is storage, not arithmetic); and a
concatenation whose parts are conv or pool outputs that nothing else reads
(through nested concatenations): each part's producer writes its slice with
the concatenation's scale (a conv part requantized, a pool part by
division).  The filter is the
batch-norm-folded one (``fold_bn``) quantized per output channel, and the
conv's output is the float32 epilogue above.  Dense layers take the same
path: weights quantized per output row, the flattened input with one scale
(requantized by the producing dense layer, else quantized by division),
exact integer dot products, the same float32 epilogue.  Pools,
concatenation and flatten are the float32 oracle's own.

Only ``tests/`` and ``__graft_entry__.smoke()`` use this module.  It shares no code with
the HIP library.
"""
from __future__ import annotations

import numpy as np

QMAX = 127


def quantize(x, scale):
    """float32 tensor -> int8 with one scale (float32 division, ties to even)."""
    q = np.rint(np.asarray(x, np.float32) / np.float32(scale))
    return np.clip(q, -QMAX, QMAX).astype(np.int8)


def filter_scales(w):
    """Per-output-channel scales max |w[k]| / 127 in float32 (1 for a zero channel)."""
    w = np.asarray(w, np.float32)
    m = np.abs(w).reshape(w.shape[0], -1).max(axis=1)
    s = (m / np.float32(QMAX)).astype(np.float32)
    s[m == 0] = np.float32(1.0)
    return s


def quantize_filter(w):
    """KCRS float32 -> (KCRS int8, per-channel float32 scales)."""
    s = filter_scales(w)
    q = np.rint(np.asarray(w, np.float32) / s[:, None, None, None])
    return np.clip(q, -QMAX, QMAX).astype(np.int8), s


def conv2d_int(xq, wq, stride=1, pad=0):
    """Cross-correlation of integer tensors with zero padding (NCHW x KCRS),
    exact: the windows are unrolled and multiplied with a float64 matrix
    product, whose every partial sum is an integer below 2^53.  int64 out."""
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    x = np.asarray(xq, np.float64)
    w = np.asarray(wq, np.float64)
    N, C, H, W = x.shape
    K, _, R, S = w.shape
    OH, OW = (H + 2 * ph - R) // sh + 1, (W + 2 * pw - S) // sw + 1
    xp = np.zeros((N, C, H + 2 * ph, W + 2 * pw))
    xp[:, :, ph:ph + H, pw:pw + W] = x
    cols = np.empty((N, OH, OW, C, R, S))
    for r in range(R):
        for s in range(S):
            cols[:, :, :, :, r, s] = xp[:, :, r:r + sh * (OH - 1) + 1:sh,
                                        s:s + sw * (OW - 1) + 1:sw].transpose(0, 2, 3, 1)
    y = cols.reshape(N * OH * OW, C * R * S) @ w.reshape(K, C * R * S).T
    return np.rint(y).astype(np.int64).reshape(N, OH, OW, K).transpose(0, 3, 1, 2).copy()


def multipliers(x_scale, w_scales):
    """The per-channel dequantization multipliers s_x * s_w[k] (float32)."""
    return (np.float32(x_scale) * np.asarray(w_scales, np.float32)).astype(np.float32)


def dequantize(acc, mult, bias=None, residual=None, act="none"):
    """act(acc * mult[k] + bias[k] + residual) in float64, rounded once."""
    y = np.asarray(acc, np.float64) * np.asarray(mult, np.float64)[None, :, None, None]
    if bias is not None:
        y = y + np.asarray(bias, np.float64)[None, :, None, None]
    if residual is not None:
        y = y + np.asarray(residual, np.float64)
    if act == "relu":
        y = np.maximum(y, 0.0)
    return y.astype(np.float32)


def epilogue_f32(acc, mult, bias=None, residual=None, act="none"):
    """act(((float32(acc) * m[k]) + bias[k]) + residual), every operation
    rounded to float32 in this order (the int32 -> float32 conversion to
    nearest, ties to even); ReLU maps every value not above 0 to +0."""
    y = np.asarray(acc).astype(np.float32) * np.asarray(mult, np.float32)[None, :, None, None]
    if bias is not None:
        y = y + np.asarray(bias, np.float32)[None, :, None, None]
    if residual is not None:
        y = y + np.asarray(residual, np.float32)
    if act == "relu":
        y = np.where(y > 0, y, np.float32(0)).astype(np.float32)
    return y.astype(np.float32)


def requantize(y, scale):
    """float32 -> int8 by the float32 reciprocal of the scale:
    clamp(round_half_even(y * float32(1 / scale)), -127, 127)."""
    r = np.float32(1) / np.float32(scale)
    q = np.rint(np.asarray(y, np.float32) * r)
    return np.clip(q, -QMAX, QMAX).astype(np.int8)


def fold_bn(w, bias, bn):
    """Batch norm folded into the preceding conv (the inference
    simplification of Section 2.2): s = gamma / sqrt(var + eps),
    w' = w s, b' = (b - mean) s + beta, in float64, each rounded once to
    float32 (eps as the float32 the network description holds)."""
    g = np.asarray(bn["gamma"], np.float64)
    v = np.asarray(bn["var"], np.float64)
    s = g / np.sqrt(v + np.float64(np.float32(bn["eps"])))
    w2 = (np.asarray(w, np.float64) * s[:, None, None, None]).astype(np.float32)
    b = np.zeros(len(g)) if bias is None else np.asarray(bias, np.float64)
    b2 = ((b - np.asarray(bn["mean"], np.float64)) * s + np.asarray(bn["beta"], np.float64))
    return w2, b2.astype(np.float32)


def act_scale(x):
    """A tensor's scale: max |x| / 127 in float32 (1 for an all-zero tensor)."""
    m = np.float32(np.abs(np.asarray(x, np.float32)).max())
    return np.float32(m / np.float32(QMAX)) if m > 0 else np.float32(1.0)


def conv_node_int8(n, x, residual=None, chained=False):
    """One conv node through the integer path: (output, the input's scale).
    How x becomes int8: `chained` True: x is the float32 output of the conv
    that writes this conv's input requantized; False: quantized by division;
    or a list of (channel count, chained) parts in channel order (a
    concatenation whose parts' producers write their slices, each by its
    own rule, with the concatenation's scale)."""
    if n.bn is not None:
        w, b = fold_bn(n.w, n.bias, n.bn)
    else:
        w = np.asarray(n.w, np.float32)
        b = None if n.bias is None else np.asarray(n.bias, np.float32)
    xs = act_scale(x)
    wq, ws = quantize_filter(w)
    if isinstance(chained, list):
        xq, c0 = [], 0
        for cnt, ch in chained:
            xq.append((requantize if ch else quantize)(x[:, c0:c0 + cnt], xs))
            c0 += cnt
        assert c0 == x.shape[1]
        xq = np.concatenate(xq, axis=1)
    else:
        xq = (requantize if chained else quantize)(x, xs)
    acc = conv2d_int(xq, wq, n.stride, n.pad)
    return epilogue_f32(acc, multipliers(xs, ws), b, residual, n.act), xs


def dense_int(xq, wq):
    """Exact integer dot products acc[n, k] = sum_i xq[n, i] * wq[k, i]
    (int64: |acc| <= 127^2 * IN)."""
    return np.asarray(xq, np.int64) @ np.asarray(wq, np.int64).T


def dense_node_int8(n, x, chained=False):
    """One dense node through the integer path: (output, the input's scale).
    The weights [out][in] are quantized per output row (quantize_filter on
    [out][in][1][1]), the input (flattened) with one scale; `chained`: x is
    the float32 output of the dense layer that writes this one's input
    requantized, else it is quantized by division.  The output is the conv's
    float32 epilogue on the exact sums (bias, activation)."""
    x2 = np.asarray(x, np.float32).reshape(x.shape[0], -1)
    w = np.asarray(n.w, np.float32)
    b = None if n.bias is None else np.asarray(n.bias, np.float32)
    xs = act_scale(x2)
    wq, ws = quantize_filter(w.reshape(w.shape[0], w.shape[1], 1, 1))
    acc = dense_int((requantize if chained else quantize)(x2, xs), wq.reshape(w.shape))
    y = epilogue_f32(acc[:, :, None, None], multipliers(xs, ws), b, None, n.act)
    return y[:, :, 0, 0], xs


def run_graph_int8(graph, x=None):
    """A network description with every conv and dense layer through the
    integer path, node by node; returns (output, their input scales in node
    order)."""
    import oracle as fo
    x = graph.x if x is None else x
    vals = [None] * len(graph.nodes)
    scales = []
    uses = [[] for _ in graph.nodes]
    for i, n in enumerate(graph.nodes):
        for j in n.inputs:
            uses[j].append(i)
        if n.residual >= 0:
            uses[n.residual].append(i)

    def parts(j):
        """A concatenation's parts in channel order as (channels, requantized),
        through nested concatenations, when every part is a conv or pool
        output read by nothing but its concatenation; else None."""
        out = []
        for p in graph.nodes[j].inputs:
            op = graph.nodes[p].op
            if uses[p] != [j]:
                return None
            if op in ("conv", "maxpool", "avgpool"):
                out.append((vals[p].shape[1], op == "conv"))
            elif op == "concat":
                sub = parts(p)
                if sub is None:
                    return None
                out += sub
            else:
                return None
        return out

    def rule(j):
        """How a conv's input value j becomes int8 (conv_node_int8's chained)."""
        src = graph.nodes[j]
        if src.op == "conv":
            return True
        if src.op == "concat":
            p = parts(j)
            if p is not None:
                return p
        return False

    for i, n in enumerate(graph.nodes):
        ins = [vals[j] for j in n.inputs]
        if n.op == "input":
            v = np.asarray(x, np.float32)
        elif n.op == "conv":
            # a conv's output is the one int8 tensor all convs reading it
            # share (whatever their paddings), requantized by that conv; a
            # concatenation of conv and pool outputs read by nothing else is
            # assembled by its parts' producers, each with its own rule and
            # the concatenation's scale; any other value is quantized by its
            # own pass (a pool's output: by the pool, the same division)
            v, xs = conv_node_int8(n, ins[0], vals[n.residual] if n.residual >= 0 else None,
                                   rule(n.inputs[0]))
            scales.append(xs)
        elif n.op == "maxpool":
            v = fo.maxpool2d(ins[0], n.R, n.S, n.stride, n.pad)
        elif n.op == "avgpool":
            v = fo.avgpool2d(ins[0], n.R, n.S, n.stride, n.pad)
        elif n.op == "gap":
            v = fo.global_avgpool(ins[0])
        elif n.op == "concat":
            v = fo.concat(ins)
        elif n.op == "flatten":
            v = fo.flatten(ins[0])
        elif n.op == "dense":
            # a dense layer's output read by the next dense layer (through a
            # flatten, if any) is requantized by it; any other input is
            # quantized by division
            src = n.inputs[0]
            while graph.nodes[src].op == "flatten":
                src = graph.nodes[src].inputs[0]
            v, xs = dense_node_int8(n, ins[0], graph.nodes[src].op == "dense")
            scales.append(xs)
        elif n.op == "output":
            v = ins[0]
        else:
            raise ValueError("unknown op " + n.op)
        vals[i] = v
    return vals[-1], np.array(scales, np.float32)
