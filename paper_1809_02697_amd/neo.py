"""Python binding of libneo (ctypes).  Argument marshalling only: every
operation runs in the HIP kernels of ``libneo.so``; there is no fallback.

Device tensors are ``torch`` float32 CUDA (HIP) tensors; torch supplies the
memory and the current stream.  Names follow the C-ABI in ``include/neo.h``.
"""
from __future__ import annotations

import ctypes
import json
import os
import re

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libneo.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "neo.h")

OK = 0
ERR_NAMES = {-1: "NEO_ERR_INVALID_ARG", -2: "NEO_ERR_SHAPE", -3: "NEO_ERR_ALIGN",
             -4: "NEO_ERR_UNSUPPORTED", -5: "NEO_ERR_HIP", -6: "NEO_ERR_OOM", -7: "NEO_ERR_STATE"}
ACT = {"none": 0, "relu": 1}
OPS = {"input": 0, "conv": 1, "maxpool": 2, "avgpool": 3, "gap": 4, "concat": 5, "flatten": 6,
       "dense": 7, "output": 8}
PLAN_HOST_ONLY = 1
PLAN_NAIVE = 2
PLAN_HIPGRAPH = 4
PLAN_TUNE = 8
PLAN_GLOBAL_SEARCH = 16
PLAN_GROUP = 32
PLAN_FUSE_GAP = 64
PLAN_FUSE_PAIRS = 128
PLAN_FUSE_CHAINS = 256
PLAN_FUSE_POOL = 512
PLAN_WINOGRAD = 1024
PLAN_INT8 = 2048
BLOCK = 16
SEARCH_BLOCKS = (0, 4, 8, 16, 32, 64)   # layout index space of neo_layout_search


class NeoError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{ERR_NAMES.get(code, code)}: {msg}")
        self.code = code


class Epilogue(ctypes.Structure):
    _fields_ = [("act", ctypes.c_int), ("residual", ctypes.c_void_p)]


class Node(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int), ("n_inputs", ctypes.c_int),
                ("inputs", ctypes.POINTER(ctypes.c_int)),
                ("K", ctypes.c_int), ("R", ctypes.c_int), ("S", ctypes.c_int),
                ("stride_h", ctypes.c_int), ("stride_w", ctypes.c_int),
                ("pad_h", ctypes.c_int), ("pad_w", ctypes.c_int),
                ("act", ctypes.c_int), ("residual", ctypes.c_int),
                ("w", ctypes.c_void_p), ("bias", ctypes.c_void_p),
                ("bn_gamma", ctypes.c_void_p), ("bn_beta", ctypes.c_void_p),
                ("bn_mean", ctypes.c_void_p), ("bn_var", ctypes.c_void_p),
                ("bn_eps", ctypes.c_float), ("ic_bn", ctypes.c_int), ("oc_bn", ctypes.c_int)]


_lib = None


def lib():
    """Load libneo.so; raises if it has not been built (no fallback path)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_1809_02697_amd.build` (no CPU fallback exists)")
    # torch first: libneo then binds to the HIP runtime torch already mapped
    # (same soname), so the process holds one HIP runtime.  Loaded the other
    # way round, the system runtime and torch's bundled one are both mapped,
    # and the second one to initialise can fail to see the device.
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    P, I, F, S = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    sig = {
        "neo_conv2d_blocked": [P, I, I, I, I, P, I, I, I, P, I, I, I, I,
                               ctypes.POINTER(Epilogue), P, I, I, P],
        "neo_conv2d_blocked_noalloc": [P, I, I, I, I, P, I, I, I, P, I, I, I, I,
                                       ctypes.POINTER(Epilogue), P, I, I, P],
        "neo_conv2d_nchwxc": [P, I, I, I, I, I, P, I, I, I, P, I, I, I, I,
                              ctypes.POINTER(Epilogue), P, I, I, I, P],
        "neo_maxpool2d_nchwxc": [P, I, I, I, I, I, I, I, I, I, I, I, P, I, I, P],
        "neo_avgpool2d_nchwxc": [P, I, I, I, I, I, I, I, I, I, I, I, P, I, I, P],
        "neo_global_avgpool_nchwxc": [P, I, I, I, I, I, P, P],
        "neo_layout_search": [ctypes.POINTER(Node), I, I, I, I, I, I, P, P, P, P, P],
        "neo_layout_transform": [P, I, P, I, I, I, I, I, P],
        "neo_pack_filter": [P, I, I, I, I, I, I, P, P],
        "neo_winograd_filter": [P, I, I, P, P],
        "neo_conv2d_winograd": [P, I, I, I, I, P, I, P, I, I, ctypes.POINTER(Epilogue), P, I, I,
                                P],
        "neo_quantize_int8": [P, I, I, I, I, F, I, I, P, P],
        "neo_pack_dense_int8": [P, I, I, P, P, P],
        "neo_quantize_rows_int8": [P, I, I, F, P, P],
        "neo_dense_int8": [P, I, I, P, P, I, F, P, I, P, F, P, P],
        "neo_pack_filter_int8": [P, I, I, I, I, P, P, P],
        "neo_conv2d_int8": [P, I, I, I, I, P, P, I, I, I, F, P, I, I, I, I,
                            ctypes.POINTER(Epilogue), P, I, I, P],
        "neo_conv2d_int8_acc": [P, I, I, I, I, P, I, I, I, I, I, I, I, P, P],
        "neo_conv2d_int8_q": [P, I, I, I, I, P, P, I, I, I, F, P, I, I, I, I,
                              ctypes.POINTER(Epilogue), F, I, I, P, I, I, P],
        "neo_fold_bn": [P, P, P, P, P, P, F, I, I, I, I, P, P],
        "neo_maxpool2d_blocked": [P, I, I, I, I, I, I, I, I, I, I, P, I, I, P],
        "neo_avgpool2d_blocked": [P, I, I, I, I, I, I, I, I, I, I, P, I, I, P],
        "neo_global_avgpool_blocked": [P, I, I, I, I, P, P],
        "neo_dense": [P, I, I, P, I, P, I, P, P],
        "neo_plan_create": [ctypes.POINTER(Node), I, I, I, I, I, I, ctypes.c_uint,
                            ctypes.POINTER(P)],
        "neo_plan_describe": [P, ctypes.c_char_p, S],
        "neo_plan_output_shape": [P, ctypes.POINTER(I)],
        "neo_plan_conv_params": [P, I, P, P],
        "neo_run_graph": [P, P, P, P],
        "neo_run_step": [P, I, P, P, P],
        "neo_plan_calibrate_int8": [P, P, P, P],
        "neo_tune_db_save": [ctypes.c_char_p],
        "neo_tune_db_load": [ctypes.c_char_p],
        "neo_tune_db_clear": [],
        "neo_tune_db_size": [],
        "neo_plan_destroy": [P],
        "neo_last_error": [],
    }
    for name, args in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = I
    L.neo_plan_destroy.restype = None
    L.neo_tune_db_clear.restype = None
    L.neo_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def header_symbols():
    """Names of the functions declared in include/neo.h."""
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(neo_[a-z0-9_]+)\s*\(", txt)))


def last_error():
    return lib().neo_last_error().decode()


def _check(rc):
    if rc < 0:
        raise NeoError(rc, last_error())
    return rc


def _stream(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dptr(t, name="tensor"):
    if t is None:
        return None
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device (cuda) tensor")
    if t.dtype != torch.float32:
        raise TypeError(f"{name} must be float32")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _dptr_typed(t, dtype, name="tensor"):
    """_dptr for a device tensor of another element type (int8, int32)."""
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device (cuda) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _pair(v):
    return tuple(v) if isinstance(v, (tuple, list)) else (v, v)


def cblocks(C, block=BLOCK):
    return -(-C // block)


def out_size(n, k, s, p):
    return (n + 2 * p - k) // s + 1


# --------------------------------------------------------------------------------------
# Single operations
# --------------------------------------------------------------------------------------
def _need(t, n, name):
    """A device buffer the kernels index up to n floats: refuse a shorter one
    (it would be an out-of-bounds device access)."""
    if t is not None and t.numel() < n:
        raise ValueError(f"{name} holds {t.numel()} floats, the call needs {n}")


def _conv_common(fn, x, xb, C, w_packed, K, R, S, bias, stride, pad, act, residual, out,
                 y_block, y_off, y_tot, stream, blocked_abi):
    import torch
    (sh, sw), (ph, pw) = _pair(stride), _pair(pad)
    N, XB, H, W, blk = x.shape
    if blk != xb or XB != cblocks(C, xb):
        raise ValueError(f"x shape {tuple(x.shape)} is not NCHW[{xb}]c of {C} channels")
    OH, OW = out_size(H, R, sh, ph), out_size(W, S, sw, pw)
    tot = cblocks(K, y_block) if y_tot is None else y_tot
    if out is None:
        out = torch.empty((N, tot, max(OH, 0), max(OW, 0), y_block), device=x.device,
                          dtype=torch.float32)
    if OH > 0 and OW > 0:
        _need(out, N * tot * OH * OW * y_block, "out")
        _need(residual, N * cblocks(K, y_block) * OH * OW * y_block, "residual")
    _need(bias, cblocks(K) * BLOCK, "bias")
    _need(w_packed, cblocks(K) * cblocks(C) * R * S * BLOCK * BLOCK, "w_packed")
    ep = Epilogue(ACT[act] if isinstance(act, str) else int(act),
                  residual.data_ptr() if residual is not None else None)
    if residual is not None:
        _dptr(residual, "residual")
    pre = (_dptr(x, "x"),) if blocked_abi else (_dptr(x, "x"), xb)
    mid = (_dptr(out, "out"),) if blocked_abi else (_dptr(out, "out"), y_block)
    _check(fn(*pre, N, C, H, W, _dptr(w_packed, "w_packed"), K, R, S, _dptr(bias, "bias"),
              sh, sw, ph, pw, ctypes.byref(ep), *mid, y_off, tot, _stream(stream)))
    return out


def conv2d_blocked(x, C, w_packed, K, R, S, bias=None, stride=1, pad=0, act="none",
                   residual=None, out=None, y_cblk_offset=0, y_cblk_total=None, stream=None):
    """x: [N][ceil(C/16)][H][W][16]; w_packed: KCRS[16]c[16]k.  Returns out."""
    return _conv_common(lib().neo_conv2d_blocked, x, BLOCK, C, w_packed, K, R, S, bias, stride,
                        pad, act, residual, out, BLOCK, y_cblk_offset, y_cblk_total, stream, True)


def conv2d_blocked_noalloc(x, C, w_packed, K, R, S, bias=None, stride=1, pad=0, act="none",
                           residual=None, out=None, y_cblk_offset=0, y_cblk_total=None,
                           stream=None):
    """conv2d_blocked whose split-reduction partials use the library's fixed
    device array (no device allocation inside the call; ``out`` should be
    passed by a caller that cannot allocate)."""
    return _conv_common(lib().neo_conv2d_blocked_noalloc, x, BLOCK, C, w_packed, K, R, S, bias,
                        stride, pad, act, residual, out, BLOCK, y_cblk_offset, y_cblk_total,
                        stream, True)


def conv2d_nchwxc(x, C, w_packed, K, R, S, bias=None, stride=1, pad=0, act="none",
                  residual=None, out=None, y_block=BLOCK, y_blk_offset=0, y_blk_total=None,
                  stream=None):
    """x: [N][ceil(C/xb)][H][W][xb] (xb from x's last dim); output NCHW[y_block]c."""
    return _conv_common(lib().neo_conv2d_nchwxc, x, x.shape[-1], C, w_packed, K, R, S, bias,
                        stride, pad, act, residual, out, y_block, y_blk_offset, y_blk_total,
                        stream, False)


def layout_transform(src, src_block, dst_block, N, C, H, W, out=None, stream=None):
    import torch
    if out is None:
        shape = (N, C, H, W) if dst_block == 0 else (N, cblocks(C, dst_block), H, W, dst_block)
        out = torch.empty(shape, device=src.device, dtype=torch.float32)
    _check(lib().neo_layout_transform(_dptr(src, "src"), src_block, _dptr(out, "out"), dst_block,
                                      N, C, H, W, _stream(stream)))
    return out


def to_blocked(x, block=BLOCK, stream=None):
    N, C, H, W = x.shape
    return layout_transform(x, 0, block, N, C, H, W, stream=stream)


def from_blocked(xb, C, stream=None):
    N, CB, H, W, blk = xb.shape
    return layout_transform(xb, blk, 0, N, C, H, W, stream=stream)


def pack_filter(w, ic_bn=BLOCK, oc_bn=BLOCK, out=None, stream=None):
    """w: device KCRS [K][C][R][S] -> KCRS[ic_bn]c[oc_bn]k."""
    import torch
    K, C, R, S = w.shape
    if out is None:
        out = torch.empty((cblocks(K, oc_bn), cblocks(C, ic_bn), R, S, ic_bn, oc_bn),
                          device=w.device, dtype=torch.float32)
    _check(lib().neo_pack_filter(_dptr(w, "w"), K, C, R, S, ic_bn, oc_bn, _dptr(out, "out"),
                                 _stream(stream)))
    return out


def winograd_filter_floats(K, C):
    return cblocks(K) * cblocks(C) * 16 * 256


def winograd_filter(w, out=None, stream=None):
    """w: device KCRS [K][C][3][3] -> the Winograd F(2x2, 3x3) transformed
    filter G w G^T, [ceil(K/16)][ceil(C/16)][16][256]."""
    import torch
    K, C, R, S = w.shape
    if (R, S) != (3, 3):
        raise ValueError("the Winograd filter transform takes 3x3 filters")
    if out is None:
        out = torch.empty((cblocks(K), cblocks(C), 16, 256), device=w.device, dtype=torch.float32)
    _need(out, winograd_filter_floats(K, C), "out")
    _check(lib().neo_winograd_filter(_dptr(w, "w"), K, C, _dptr(out, "out"), _stream(stream)))
    return out


def conv2d_winograd(x, C, u, K, bias=None, pad=1, act="none", residual=None, out=None,
                    y_cblk_offset=0, y_cblk_total=None, stream=None):
    """3x3 stride-1 convolution by Winograd F(2x2, 3x3): x NCHW16c of C
    channels, u from winograd_filter; the rest as conv2d_blocked."""
    import torch
    ph, pw = _pair(pad)
    N, XB, H, W, blk = x.shape
    if blk != BLOCK or XB != cblocks(C):
        raise ValueError(f"x shape {tuple(x.shape)} is not NCHW16c of {C} channels")
    OH, OW = out_size(H, 3, 1, ph), out_size(W, 3, 1, pw)
    tot = cblocks(K) if y_cblk_total is None else y_cblk_total
    if out is None:
        out = torch.empty((N, tot, max(OH, 0), max(OW, 0), BLOCK), device=x.device,
                          dtype=torch.float32)
    if OH > 0 and OW > 0:
        _need(out, N * tot * OH * OW * BLOCK, "out")
        _need(residual, N * cblocks(K) * OH * OW * BLOCK, "residual")
    _need(bias, cblocks(K) * BLOCK, "bias")
    _need(u, winograd_filter_floats(K, C), "u")
    ep = Epilogue(ACT[act] if isinstance(act, str) else int(act),
                  residual.data_ptr() if residual is not None else None)
    if residual is not None:
        _dptr(residual, "residual")
    _check(lib().neo_conv2d_winograd(_dptr(x, "x"), N, C, H, W, _dptr(u, "u"), K,
                                     _dptr(bias, "bias"), ph, pw, ctypes.byref(ep),
                                     _dptr(out, "out"), y_cblk_offset, tot, _stream(stream)))
    return out


def int8_filter_bytes(K, C, R, S):
    return cblocks(K) * cblocks(C, 64) * R * S * 1024


def quantize_int8(x, C, x_scale, pad=0, out=None, stream=None):
    """x: fp32 NCHW16c of C channels -> int8 NCHW16c with the zero padding
    `pad` of the convolution that reads it stored as a halo,
    [N][CB][H + 2 ph][W + 2 pw][16], clamp(round_half_even(x / x_scale), -127, 127)."""
    import torch
    ph, pw = _pair(pad)
    N, XB, H, W, blk = x.shape
    if blk != BLOCK or XB != cblocks(C):
        raise ValueError(f"x shape {tuple(x.shape)} is not NCHW16c of {C} channels")
    shape = (N, XB, H + 2 * ph, W + 2 * pw, BLOCK)
    if out is None:
        out = torch.empty(shape, device=x.device, dtype=torch.int8)
    if out.numel() < int(np.prod(shape)):
        raise ValueError(f"out holds {out.numel()} bytes, the call needs {int(np.prod(shape))}")
    _check(lib().neo_quantize_int8(_dptr(x, "x"), N, C, H, W, float(x_scale), ph, pw,
                                   _dptr_typed(out, torch.int8, "out"), _stream(stream)))
    return out


def pack_filter_int8(w, out=None, scale=None, stream=None):
    """w: device KCRS fp32 -> (packed int8 filter, per-output-channel scales
    [ceil(K/16)*16] fp32), the scales max |w[k]| / 127."""
    import torch
    K, C, R, S = w.shape
    nb = int8_filter_bytes(K, C, R, S)
    if out is None:
        out = torch.empty(nb, device=w.device, dtype=torch.int8)
    if scale is None:
        scale = torch.empty(cblocks(K) * BLOCK, device=w.device, dtype=torch.float32)
    if out.numel() < nb:
        raise ValueError(f"out holds {out.numel()} bytes, the call needs {nb}")
    _need(scale, cblocks(K) * BLOCK, "scale")
    _check(lib().neo_pack_filter_int8(_dptr(w, "w"), K, C, R, S,
                                      _dptr_typed(out, torch.int8, "out"), _dptr(scale, "scale"),
                                      _stream(stream)))
    return out, scale


def dense_row_bytes(n):
    """Bytes of one int8 row of n values, padded to 16."""
    return -(-int(n) // BLOCK) * BLOCK


def pack_dense_int8(w, out=None, scale=None, stream=None):
    """w: device [out][in] fp32 -> (int8 rows [out][dense_row_bytes(in)],
    per-row scales [out] fp32), the scales max |w[k]| / 127."""
    import torch
    OUT, IN = w.shape
    shape = (OUT, dense_row_bytes(IN))
    if out is None:
        out = torch.empty(shape, device=w.device, dtype=torch.int8)
    if scale is None:
        scale = torch.empty(OUT, device=w.device, dtype=torch.float32)
    if out.numel() < OUT * shape[1]:
        raise ValueError(f"out holds {out.numel()} bytes, the call needs {OUT * shape[1]}")
    _need(scale, OUT, "scale")
    _check(lib().neo_pack_dense_int8(_dptr(w, "w"), OUT, IN, _dptr_typed(out, torch.int8, "out"),
                                     _dptr(scale, "scale"), _stream(stream)))
    return out, scale


def quantize_rows_int8(x, x_scale, out=None, stream=None):
    """x: device [N][in] fp32 -> int8 rows [N][dense_row_bytes(in)],
    clamp(round_half_even(x / x_scale), -127, 127), the padding 0."""
    import torch
    N, IN = x.shape
    shape = (N, dense_row_bytes(IN))
    if out is None:
        out = torch.empty(shape, device=x.device, dtype=torch.int8)
    if out.numel() < N * shape[1]:
        raise ValueError(f"out holds {out.numel()} bytes, the call needs {N * shape[1]}")
    _check(lib().neo_quantize_rows_int8(_dptr(x, "x"), N, IN, float(x_scale),
                                        _dptr_typed(out, torch.int8, "out"), _stream(stream)))
    return out


def dense_int8(xq, IN, w_rows, w_scale, OUT, x_scale, bias=None, act="none", out=None,
               y_scale=None, out_q=None, stream=None):
    """Integer dense layer: xq int8 rows [N][dense_row_bytes(IN)]
    (quantize_rows_int8), w_rows and w_scale from pack_dense_int8; fp32 output
    [N][OUT] act(acc * x_scale * w_scale[k] + bias) (out), and with y_scale
    also its int8 rows for the next dense layer (out_q, [N][dense_row_bytes(OUT)])
    -- out=False for the int8 rows only."""
    import torch
    N = xq.shape[0]
    if xq.numel() < N * dense_row_bytes(IN) or w_rows.numel() < OUT * dense_row_bytes(IN):
        raise ValueError("xq or w_rows smaller than the layer's rows")
    _need(w_scale, OUT, "w_scale")
    _need(bias, OUT, "bias")
    if out is None:
        out = torch.empty((N, OUT), device=xq.device, dtype=torch.float32)
    if out is not False:
        _need(out, N * OUT, "out")
    if y_scale is not None and out_q is None:
        out_q = torch.zeros((N, dense_row_bytes(OUT)), device=xq.device, dtype=torch.int8)
    if out_q is not None and out_q.numel() < N * dense_row_bytes(OUT):
        raise ValueError(f"out_q holds {out_q.numel()} bytes, the call needs {N * dense_row_bytes(OUT)}")
    yp = None if out is False else _dptr(out, "out")
    qp = None if out_q is None else _dptr_typed(out_q, torch.int8, "out_q")
    _check(lib().neo_dense_int8(_dptr_typed(xq, torch.int8, "xq"), N, IN,
                                _dptr_typed(w_rows, torch.int8, "w_rows"), _dptr(w_scale, "w_scale"), OUT,
                                float(x_scale), _dptr(bias, "bias"), ACT[act] if isinstance(act, str) else int(act),
                                yp, float(y_scale or 0.0), qp, _stream(stream)))
    return (None if out is False else out), out_q


def _int8_args(xq, C, w_packed, K, R, S, stride, pad):
    (sh, sw), (ph, pw) = _pair(stride), _pair(pad)
    N, XB, Hp, Wp, blk = xq.shape
    if blk != BLOCK or XB != cblocks(C):
        raise ValueError(f"xq shape {tuple(xq.shape)} is not NCHW16c of {C} channels")
    # xq carries the convolution's padding as its halo
    H, W = Hp - 2 * ph, Wp - 2 * pw
    if H < 1 or W < 1:
        raise ValueError(f"xq shape {tuple(xq.shape)} is smaller than its halo of {(ph, pw)}")
    if w_packed.numel() < int8_filter_bytes(K, C, R, S):
        raise ValueError(f"w_packed holds {w_packed.numel()} bytes, the call needs "
                         f"{int8_filter_bytes(K, C, R, S)}")
    return N, H, W, sh, sw, ph, pw, out_size(H, R, sh, ph), out_size(W, S, sw, pw)


def _int8_ptrs(xq, w_packed):
    import torch
    return _dptr_typed(xq, torch.int8, "xq"), _dptr_typed(w_packed, torch.int8, "w_packed")


def conv2d_int8(xq, C, w_packed, w_scale, K, R, S, x_scale, bias=None, stride=1, pad=0,
                act="none", residual=None, out=None, y_cblk_offset=0, y_cblk_total=None,
                stream=None):
    """Integer convolution: xq int8 NCHW16c with the halo `pad`
    (quantize_int8 with the same pad), w_packed and
    w_scale from pack_filter_int8; fp32 NCHW16c output
    act(acc * x_scale * w_scale[k] + bias + residual), the view as conv2d_blocked."""
    import torch
    N, H, W, sh, sw, ph, pw, OH, OW = _int8_args(xq, C, w_packed, K, R, S, stride, pad)
    tot = cblocks(K) if y_cblk_total is None else y_cblk_total
    if out is None:
        out = torch.empty((N, tot, max(OH, 0), max(OW, 0), BLOCK), device=xq.device,
                          dtype=torch.float32)
    if OH > 0 and OW > 0:
        _need(out, N * tot * OH * OW * BLOCK, "out")
        _need(residual, N * cblocks(K) * OH * OW * BLOCK, "residual")
    _need(bias, cblocks(K) * BLOCK, "bias")
    _need(w_scale, cblocks(K) * BLOCK, "w_scale")
    ep = Epilogue(ACT[act] if isinstance(act, str) else int(act),
                  residual.data_ptr() if residual is not None else None)
    if residual is not None:
        _dptr(residual, "residual")
    xp, wp = _int8_ptrs(xq, w_packed)
    _check(lib().neo_conv2d_int8(xp, N, C, H, W, wp, _dptr(w_scale, "w_scale"), K, R, S,
                                 float(x_scale), _dptr(bias, "bias"), sh, sw, ph, pw,
                                 ctypes.byref(ep), _dptr(out, "out"), y_cblk_offset, tot,
                                 _stream(stream)))
    return out


def conv2d_int8_q(xq, C, w_packed, w_scale, K, R, S, x_scale, y_scale, bias=None, stride=1,
                  pad=0, act="none", residual=None, out_pad=0, out=None, y_cblk_offset=0,
                  y_cblk_total=None, stream=None):
    """conv2d_int8 with its float32 output requantized for the next layer:
    int8 NCHW16c [N][y_cblk_total][OH + 2 ph'][OW + 2 pw'][16] with the halo
    `out_pad` (the next conv's padding) left as the caller made it (zeros when
    `out` is allocated here), clamp(round_half_even(y * float32(1 / y_scale)))."""
    import torch
    N, H, W, sh, sw, ph, pw, OH, OW = _int8_args(xq, C, w_packed, K, R, S, stride, pad)
    qph, qpw = _pair(out_pad)
    tot = cblocks(K) if y_cblk_total is None else y_cblk_total
    shape = (N, tot, max(OH, 0) + 2 * qph, max(OW, 0) + 2 * qpw, BLOCK)
    if out is None:
        out = torch.zeros(shape, device=xq.device, dtype=torch.int8)
    if OH > 0 and OW > 0:
        if out.numel() < int(np.prod(shape)):
            raise ValueError(f"out holds {out.numel()} bytes, the call needs {int(np.prod(shape))}")
        _need(residual, N * cblocks(K) * OH * OW * BLOCK, "residual")
    _need(bias, cblocks(K) * BLOCK, "bias")
    _need(w_scale, cblocks(K) * BLOCK, "w_scale")
    ep = Epilogue(ACT[act] if isinstance(act, str) else int(act),
                  residual.data_ptr() if residual is not None else None)
    if residual is not None:
        _dptr(residual, "residual")
    xp, wp = _int8_ptrs(xq, w_packed)
    _check(lib().neo_conv2d_int8_q(xp, N, C, H, W, wp, _dptr(w_scale, "w_scale"), K, R, S,
                                   float(x_scale), _dptr(bias, "bias"), sh, sw, ph, pw,
                                   ctypes.byref(ep), float(y_scale), qph, qpw,
                                   _dptr_typed(out, torch.int8, "out"), y_cblk_offset, tot,
                                   _stream(stream)))
    return out


def conv2d_int8_acc(xq, C, w_packed, K, R, S, stride=1, pad=0, out=None, stream=None):
    """The exact int32 sums of the integer convolution, int32 NCHW16c
    [N][ceil(K/16)][OH][OW][16] (padding channels 0)."""
    import torch
    N, H, W, sh, sw, ph, pw, OH, OW = _int8_args(xq, C, w_packed, K, R, S, stride, pad)
    if out is None:
        out = torch.empty((N, cblocks(K), max(OH, 0), max(OW, 0), BLOCK), device=xq.device,
                          dtype=torch.int32)
    if OH > 0 and OW > 0 and out.numel() < N * cblocks(K) * OH * OW * BLOCK:
        raise ValueError(f"out holds {out.numel()} values, the call needs "
                         f"{N * cblocks(K) * OH * OW * BLOCK}")
    xp, wp = _int8_ptrs(xq, w_packed)
    _check(lib().neo_conv2d_int8_acc(xp, N, C, H, W, wp, K, R, S, sh, sw, ph, pw,
                                     _dptr_typed(out, torch.int32, "out"), _stream(stream)))
    return out


def _hp(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def fold_bn(w, bias, gamma, beta, mean, var, eps):
    """Host batch-norm fold (numpy float32 in, numpy float32 out)."""
    w = np.ascontiguousarray(w, np.float32)
    K, C, R, S = w.shape
    arrs = [None if bias is None else np.ascontiguousarray(bias, np.float32)] + \
           [np.ascontiguousarray(a, np.float32) for a in (gamma, beta, mean, var)]
    w_out = np.empty_like(w)
    b_out = np.empty(K, np.float32)
    _check(lib().neo_fold_bn(_hp(w), *[_hp(a) for a in arrs], float(eps), K, C, R, S,
                             _hp(w_out), _hp(b_out)))
    return w_out, b_out


def _pool(fn, x, C, R, S, stride, pad, out, y_cblk_offset, y_cblk_total, stream, blocked=False):
    import torch
    (sh, sw), (ph, pw) = _pair(stride), _pair(pad)
    N, CB, H, W, blk = x.shape
    OH, OW = out_size(H, R, sh, ph), out_size(W, S, sw, pw)
    tot = CB if y_cblk_total is None else y_cblk_total
    if out is None:
        out = torch.empty((N, tot, max(OH, 0), max(OW, 0), blk), device=x.device,
                          dtype=torch.float32)
    if CB != cblocks(C, blk):
        raise ValueError(f"x shape {tuple(x.shape)} is not NCHW[{blk}]c of {C} channels")
    if OH > 0 and OW > 0:
        _need(out, N * tot * OH * OW * blk, "out")
    pre = (_dptr(x, "x"), blk) if blocked else (_dptr(x, "x"),)
    _check(fn(*pre, N, C, H, W, R, S, sh, sw, ph, pw, _dptr(out, "out"), y_cblk_offset,
              tot, _stream(stream)))
    return out


def maxpool2d_nchwxc(x, C, R, S, stride, pad=0, out=None, y_blk_offset=0, y_blk_total=None,
                     stream=None):
    """x: [N][ceil(C/b)][H][W][b], block b from x's last dim."""
    return _pool(lib().neo_maxpool2d_nchwxc, x, C, R, S, stride, pad, out, y_blk_offset,
                 y_blk_total, stream, blocked=True)


def avgpool2d_nchwxc(x, C, R, S, stride, pad=0, out=None, y_blk_offset=0, y_blk_total=None,
                     stream=None):
    return _pool(lib().neo_avgpool2d_nchwxc, x, C, R, S, stride, pad, out, y_blk_offset,
                 y_blk_total, stream, blocked=True)


def global_avgpool_nchwxc(x, C, out=None, stream=None):
    import torch
    N, CB, H, W, blk = x.shape
    if out is None:
        out = torch.empty((N, CB, 1, 1, blk), device=x.device, dtype=torch.float32)
    _need(out, N * CB * blk, "out")
    _check(lib().neo_global_avgpool_nchwxc(_dptr(x, "x"), blk, N, C, H, W, _dptr(out, "out"),
                                           _stream(stream)))
    return out


def maxpool2d_blocked(x, C, R, S, stride, pad=0, out=None, y_cblk_offset=0, y_cblk_total=None,
                      stream=None):
    return _pool(lib().neo_maxpool2d_blocked, x, C, R, S, stride, pad, out, y_cblk_offset,
                 y_cblk_total, stream)


def avgpool2d_blocked(x, C, R, S, stride, pad=0, out=None, y_cblk_offset=0, y_cblk_total=None,
                      stream=None):
    return _pool(lib().neo_avgpool2d_blocked, x, C, R, S, stride, pad, out, y_cblk_offset,
                 y_cblk_total, stream)


def global_avgpool_blocked(x, C, out=None, stream=None):
    import torch
    N, CB, H, W, _ = x.shape
    if out is None:
        out = torch.empty((N, CB, 1, 1, BLOCK), device=x.device, dtype=torch.float32)
    _need(out, N * CB * BLOCK, "out")
    _check(lib().neo_global_avgpool_blocked(_dptr(x, "x"), N, C, H, W, _dptr(out, "out"),
                                            _stream(stream)))
    return out


def dense(x, w, bias=None, act="none", out=None, stream=None):
    """x device [N][IN], w device [OUT][IN] -> [N][OUT]."""
    import torch
    N, IN = x.shape
    OUT = w.shape[0]
    if out is None:
        out = torch.empty((N, OUT), device=x.device, dtype=torch.float32)
    if w.numel() != OUT * IN:
        raise ValueError(f"w holds {w.numel()} floats, not {OUT} x {IN}")
    _need(out, N * OUT, "out")
    _need(bias, OUT, "bias")
    _check(lib().neo_dense(_dptr(x, "x"), N, IN, _dptr(w, "w"), OUT, _dptr(bias, "bias"),
                           ACT[act] if isinstance(act, str) else int(act), _dptr(out, "out"),
                           _stream(stream)))
    return out


def tune_db_save(path):
    return _check(lib().neo_tune_db_save(str(path).encode()))


def tune_db_load(path):
    return _check(lib().neo_tune_db_load(str(path).encode()))


def tune_db_clear():
    lib().neo_tune_db_clear()


def tune_db_size():
    return lib().neo_tune_db_size()


# --------------------------------------------------------------------------------------
# Graph plan
# --------------------------------------------------------------------------------------
def _node_array(graph, schemes=None, keep=None, with_params=True):
    """ctypes neo_node array of a network description; schemes: {conv node id:
    (ic_bn, oc_bn)}.  Host arrays referenced by the nodes are appended to keep."""
    keep = [] if keep is None else keep
    schemes = schemes or {}
    arr = (Node * len(graph.nodes))()
    for i, n in enumerate(graph.nodes):
        d = arr[i]
        d.op = OPS[n.op]
        ins = (ctypes.c_int * max(1, len(n.inputs)))(*n.inputs)
        keep.append(ins)
        d.n_inputs = len(n.inputs)
        d.inputs = ctypes.cast(ins, ctypes.POINTER(ctypes.c_int))
        d.K, d.R, d.S = n.K, n.R, n.S
        d.stride_h, d.stride_w = n.stride
        d.pad_h, d.pad_w = n.pad
        d.act = ACT[n.act]
        d.residual = n.residual
        d.ic_bn, d.oc_bn = schemes.get(i, (0, 0))
        if not with_params:
            continue

        def host(a):
            if a is None:
                return None
            a = np.ascontiguousarray(a, np.float32)
            keep.append(a)
            return ctypes.c_void_p(a.ctypes.data)

        d.w = host(n.w)
        d.bias = host(n.bias)
        if n.bn is not None:
            d.bn_gamma, d.bn_beta = host(n.bn["gamma"]), host(n.bn["beta"])
            d.bn_mean, d.bn_var = host(n.bn["mean"]), host(n.bn["var"])
            d.bn_eps = float(n.bn["eps"])
    return arr


def layout_search(graph, conv_time, xform_time, block=BLOCK, schemes=None):
    """Algorithm 2 on the host (neo_layout_search).  conv_time, xform_time:
    arrays [n_nodes][6][6] over SEARCH_BLOCKS (conv_time inf / negative = not a
    candidate).  Returns (cost, {conv node: (ic_bn, oc_bn)})."""
    L = lib()
    n = len(graph.nodes)
    ct = np.ascontiguousarray(conv_time, np.float64).reshape(n, 6, 6)
    xt = np.ascontiguousarray(xform_time, np.float64).reshape(n, 6, 6)
    ic = np.zeros(n, np.int32)
    oc = np.zeros(n, np.int32)
    cost = ctypes.c_double()
    arr = _node_array(graph, schemes, with_params=False)
    _check(L.neo_layout_search(arr, n, *graph.input_shape, block, _hp(ct), _hp(xt), _hp(ic),
                               _hp(oc), ctypes.byref(cost)))
    return cost.value, {i: (int(ic[i]), int(oc[i])) for i in range(n)
                        if graph.nodes[i].op == "conv"}


class Plan:
    """A plan built from a network description (``workloads.Graph``).
    schemes: {conv node id: (ic_bn, oc_bn)} fixing those convs' layouts."""

    def __init__(self, graph, input_shape=None, flags=0, block=BLOCK, schemes=None):
        L = lib()
        shape = tuple(input_shape or graph.input_shape)
        keep = []
        arr = _node_array(graph, schemes, keep)
        h = ctypes.c_void_p()
        _check(L.neo_plan_create(arr, len(graph.nodes), *shape, block, flags, ctypes.byref(h)))
        self._h = h
        self.flags = flags
        self.input_shape = shape
        dims = (ctypes.c_int * 4)()
        _check(L.neo_plan_output_shape(h, dims))
        self.output_shape = tuple(dims)

    @property
    def handle(self):
        if self._h is None:
            raise NeoError(-7, "plan destroyed")
        return self._h

    def describe(self):
        L = lib()
        n = _check(L.neo_plan_describe(self.handle, None, 0))
        buf = ctypes.create_string_buffer(n + 1)
        _check(L.neo_plan_describe(self.handle, buf, n + 1))
        return json.loads(buf.value.decode())

    def conv_params(self, node_id, K, C, R, S):
        wp = np.empty((cblocks(K), cblocks(C), R, S, BLOCK, BLOCK), np.float32)
        b = np.empty(cblocks(K) * BLOCK, np.float32)
        _check(lib().neo_plan_conv_params(self.handle, node_id, _hp(wp), _hp(b)))
        return wp, b

    def run(self, x, out=None, stream=None):
        """x: device NCHW input -> device output of ``output_shape``
        ([N, C] after flatten/dense, else [N, C, H, W])."""
        import torch
        if tuple(x.shape) != self.input_shape:
            raise ValueError(f"input shape {tuple(x.shape)} != plan input {self.input_shape}")
        if out is None:
            N, C, H, W = self.output_shape
            shape = (N, C) if (H, W) == (1, 1) else (N, C, H, W)
            out = torch.empty(shape, device=x.device, dtype=torch.float32)
        _need(out, int(np.prod(self.output_shape)), "out")
        _check(lib().neo_run_graph(self.handle, _dptr(x, "x"), _dptr(out, "out"),
                                   _stream(stream)))
        return out

    def calibrate_int8(self, x, out=None, stream=None):
        """NEO_PLAN_INT8: set every conv's input scale from a run on x (device
        NCHW); returns that run's output."""
        import torch
        if tuple(x.shape) != self.input_shape:
            raise ValueError(f"input shape {tuple(x.shape)} != plan input {self.input_shape}")
        if out is None:
            N, C, H, W = self.output_shape
            shape = (N, C) if (H, W) == (1, 1) else (N, C, H, W)
            out = torch.empty(shape, device=x.device, dtype=torch.float32)
        _need(out, int(np.prod(self.output_shape)), "out")
        _check(lib().neo_plan_calibrate_int8(self.handle, _dptr(x, "x"), _dptr(out, "out"),
                                             _stream(stream)))
        return out

    def run_step(self, step, x, out, stream=None):
        """Launch one step of the plan's launch list (for timing single layers)."""
        if tuple(x.shape) != self.input_shape:
            raise ValueError(f"input shape {tuple(x.shape)} != plan input {self.input_shape}")
        _need(out, int(np.prod(self.output_shape)), "out")
        _check(lib().neo_run_step(self.handle, step, _dptr(x, "x"), _dptr(out, "out"),
                                  _stream(stream)))

    def destroy(self):
        if self._h is not None:
            lib().neo_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass
