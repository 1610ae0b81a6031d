"""An independent float32 CPU pipeline (PyTorch's own CPU kernels) for the
network descriptions: the ceiling that the parity tests put on how many
elements may miss the plain element-wise clause 1e-4 (1 + |ref|) against the
oracle.  A float32 implementation's rounding error grows with the magnitude of
the summed terms, not with |ref|, so at outputs that arise from cancellation
any float32 pipeline misses the plain clause; this one says how often a
correct one does on the same inputs.

Batch norm is folded into the weights in float64 and rounded once, as the
GPU plan does, so the two differ only in their float32 arithmetic.  Test
infrastructure only; it shares nothing with the HIP path or the oracle."""
import numpy as np


def _torch():
    import torch
    return torch


def fold(n):
    """(w', b') of a conv node: w' = w s, b' = (b - mean) s + beta with
    s = gamma / sqrt(var + eps), in float64, one rounding; without batch norm
    the node's own weights and bias (or zeros)."""
    w = n.w.astype(np.float64)
    b = n.bias.astype(np.float64) if n.bias is not None else np.zeros(n.K)
    if n.bn is not None:
        p = n.bn
        s = p["gamma"].astype(np.float64) / np.sqrt(p["var"].astype(np.float64) + p["eps"])
        w = w * s.reshape(-1, 1, 1, 1)
        b = (b - p["mean"].astype(np.float64)) * s + p["beta"].astype(np.float64)
    return w.astype(np.float32), b.astype(np.float32)


def conv_layer(x, w, b, stride, pad, act, residual=None):
    """act(conv(x, w) + b + residual) in float32 on the CPU (numpy in and out)."""
    torch = _torch()
    F = torch.nn.functional
    with torch.no_grad():
        y = F.conv2d(torch.from_numpy(np.ascontiguousarray(x, np.float32)),
                     torch.from_numpy(np.ascontiguousarray(w, np.float32)),
                     torch.from_numpy(np.ascontiguousarray(b, np.float32)),
                     stride=tuple(stride), padding=tuple(pad))
        if residual is not None:
            y = y + torch.from_numpy(np.ascontiguousarray(residual, np.float32))
        if act == "relu":
            y = torch.relu(y)
    return y.numpy()


def run_graph(graph, x=None):
    """The network in float32 on the CPU, node by node; returns the output."""
    torch = _torch()
    F = torch.nn.functional
    x = graph.x if x is None else x
    vals = [None] * len(graph.nodes)
    with torch.no_grad():
        for i, n in enumerate(graph.nodes):
            ins = [vals[j] for j in n.inputs]
            if n.op == "input":
                v = torch.from_numpy(np.ascontiguousarray(x, np.float32))
            elif n.op == "conv":
                w, b = fold(n)
                v = F.conv2d(ins[0], torch.from_numpy(w), torch.from_numpy(b),
                             stride=tuple(n.stride), padding=tuple(n.pad))
                if n.residual >= 0:
                    v = v + vals[n.residual]
                if n.act == "relu":
                    v = torch.relu(v)
            elif n.op == "maxpool":
                v = F.max_pool2d(ins[0], (n.R, n.S), tuple(n.stride), tuple(n.pad))
            elif n.op == "avgpool":
                v = F.avg_pool2d(ins[0], (n.R, n.S), tuple(n.stride), tuple(n.pad),
                                 count_include_pad=False)
            elif n.op == "gap":
                v = ins[0].mean(dim=(2, 3), keepdim=True)
            elif n.op == "concat":
                v = torch.cat(ins, dim=1)
            elif n.op == "flatten":
                v = ins[0].reshape(ins[0].shape[0], -1)
            elif n.op == "dense":
                v = F.linear(ins[0], torch.from_numpy(n.w), torch.from_numpy(n.bias))
                if n.act == "relu":
                    v = torch.relu(v)
            elif n.op == "output":
                v = ins[0]
            else:
                raise ValueError("unknown op " + n.op)
            vals[i] = v
    return vals[-1].numpy()
