"""Integer (INT8) convolution (neo_quantize_int8, neo_pack_filter_int8,
neo_conv2d_int8, neo_conv2d_int8_acc) and dense layer (neo_pack_dense_int8,
neo_quantize_rows_int8, neo_dense_int8): argument handling on the host; on
the GPU the quantized activations, the packed filters and their scales, and
the int32 accumulators bit-exact against the oracle's integer path
(oracle.quant), and the dequantized float32 output within the rounding bound
of its epilogue (and bit-exact against the oracle's step-by-step float32
evaluation)."""
import ctypes

import numpy as np
import pytest

import oracle as orc
from oracle import quant as oq
from paper_1809_02697_amd import neo
from paper_1809_02697_amd import workloads as wl

FAKE = ctypes.c_void_p(1 << 20)   # aligned, never dereferenced: validation fails first
MIS = ctypes.c_void_p((1 << 20) + 4)


def _conv(x=FAKE, C=16, R=3, yt=1, w=FAKE, ws=FAKE, xs=1.0, pd=1, y=FAKE):
    return neo.lib().neo_conv2d_int8(x, 1, C, 8, 8, w, ws, 16, R, R, xs, None, 1, 1, pd, pd, None,
                                     y, 0, yt, None)


def test_argument_errors():
    """Validation before any device work, the entry point named in the message."""
    L = neo.lib()
    assert _conv(x=None) == -1 and "neo_conv2d_int8" in neo.last_error()
    assert _conv(w=MIS) == -3
    assert _conv(ws=None) == -1 and "w_scale" in neo.last_error()
    assert _conv(ws=MIS) == -3
    for bad in (0.0, -1.0, float("nan"), float("inf")):
        assert _conv(xs=bad) == -1 and "x_scale" in neo.last_error()
    assert _conv(yt=0) == -2
    assert _conv(pd=-1) == -1
    # 14,778 channels x 3 x 3 = 133,002 terms: 127^2 times that exceeds int32
    assert _conv(C=14778) == -4 and "133,000" in neo.last_error()
    assert L.neo_conv2d_int8_acc(FAKE, 1, 16, 8, 8, FAKE, 16, 3, 3, 1, 1, 1, 1, None, None) == -1
    assert L.neo_conv2d_int8_acc(FAKE, 1, 16, 8, 8, FAKE, 16, 3, 3, 1, 1, 1, 1, MIS, None) == -3
    assert L.neo_quantize_int8(None, 1, 16, 8, 8, 1.0, 1, 1, FAKE, None) == -1
    assert L.neo_quantize_int8(FAKE, 1, 16, 8, 8, 0.0, 1, 1, FAKE, None) == -1
    assert L.neo_quantize_int8(FAKE, 1, 16, 8, 8, 1.0, 1, 1, MIS, None) == -3
    assert L.neo_quantize_int8(FAKE, 0, 16, 8, 8, 1.0, 1, 1, FAKE, None) == -1
    assert L.neo_quantize_int8(FAKE, 1, 16, 8, 8, 1.0, -1, 1, FAKE, None) == -1
    def q(ys=0.5, yq=FAKE, qp=1):
        return L.neo_conv2d_int8_q(FAKE, 1, 16, 8, 8, FAKE, FAKE, 16, 3, 3, 1.0, None, 1, 1, 1, 1,
                                   None, ys, qp, qp, yq, 0, 1, None)
    assert q(yq=None) == -1 and "yq" in neo.last_error()
    assert q(yq=MIS) == -3
    for bad in (0.0, -2.0, float("inf"), float("nan"), 1e-45):
        assert q(ys=bad) == -1 and "y_scale" in neo.last_error()
    assert q(qp=-1) == -1
    assert L.neo_pack_filter_int8(None, 16, 16, 3, 3, FAKE, FAKE, None) == -1
    assert L.neo_pack_filter_int8(FAKE, 16, 16, 3, 3, FAKE, None, None) == -1
    assert L.neo_pack_filter_int8(FAKE, 0, 16, 3, 3, FAKE, FAKE, None) == -1


def test_dense_argument_errors():
    """The integer dense layer's calls validate before any device work."""
    L = neo.lib()
    def d(xq=FAKE, IN=64, w=FAKE, ws=FAKE, OUT=16, xs=1.0, act=0, y=FAKE, ys=0.0, yq=None):
        return L.neo_dense_int8(xq, 1, IN, w, ws, OUT, xs, None, act, y, ys, yq, None)
    assert d(xq=None) == -1 and "neo_dense_int8" in neo.last_error()
    assert d(ws=None) == -1
    assert d(y=None, yq=None) == -1 and "neither" in neo.last_error()
    assert d(xq=MIS) == -3 and d(w=MIS) == -3
    assert d(IN=0) == -1 and d(OUT=-1) == -1
    assert d(act=7) == -1
    for bad in (0.0, -1.0, float("nan"), float("inf")):
        assert d(xs=bad) == -1 and "x_scale" in neo.last_error()
    for bad in (0.0, -2.0, float("inf"), 1e-45):
        assert d(yq=FAKE, ys=bad) == -1 and "y_scale" in neo.last_error()
    # 133,145 inputs: 127^2 times that exceeds int32 (133,144 do not)
    assert d(IN=133145) == -4 and "133,144" in neo.last_error()
    assert L.neo_pack_dense_int8(None, 16, 64, FAKE, FAKE, None) == -1
    assert L.neo_pack_dense_int8(FAKE, 16, 64, MIS, FAKE, None) == -3
    assert L.neo_pack_dense_int8(FAKE, 0, 64, FAKE, FAKE, None) == -1
    assert L.neo_quantize_rows_int8(FAKE, 1, 64, 0.0, FAKE, None) == -1
    assert L.neo_quantize_rows_int8(FAKE, 1, 64, 1.0, MIS, None) == -3
    assert L.neo_quantize_rows_int8(None, 1, 64, 1.0, FAKE, None) == -1
    assert neo.dense_row_bytes(1000) == 1008 and neo.dense_row_bytes(4096) == 4096


def test_packed_filter_size():
    # ceil(K/16) * ceil(C/64) * R * S blocks of 64 lanes x 16 bytes
    assert neo.int8_filter_bytes(64, 64, 3, 3) == 4 * 1 * 9 * 1024
    assert neo.int8_filter_bytes(17, 65, 1, 7) == 2 * 2 * 7 * 1024
    assert neo.int8_filter_bytes(1, 1, 1, 1) == 1024


def test_binding_refuses_short_buffers():
    import torch
    xq = torch.zeros((1, 1, 10, 10, 16), dtype=torch.int8)     # 8 x 8 with a halo of 1
    wq = torch.zeros(neo.int8_filter_bytes(32, 16, 3, 3), dtype=torch.int8)
    with pytest.raises(ValueError, match="w_packed holds"):
        neo.conv2d_int8(xq, 16, wq[:-1], torch.ones(32), 32, 3, 3, 0.1, pad=1)
    with pytest.raises(ValueError, match="NCHW16c"):
        neo.conv2d_int8(torch.zeros((1, 2, 8, 8, 16), dtype=torch.int8), 16, wq, torch.ones(32),
                        32, 3, 3, 0.1)
    with pytest.raises(ValueError, match="halo"):
        neo.conv2d_int8(torch.zeros((1, 1, 2, 2, 16), dtype=torch.int8), 16, wq, torch.ones(32),
                        32, 3, 3, 0.1, pad=1)
    with pytest.raises(ValueError, match="out"):
        neo.conv2d_int8(xq, 16, wq, torch.ones(32), 32, 3, 3, 0.1, pad=1,
                        out=torch.zeros(2 * 8 * 8 * 16 - 1))
    with pytest.raises(ValueError, match="w_scale"):
        neo.conv2d_int8(xq, 16, wq, torch.ones(31), 32, 3, 3, 0.1, pad=1,
                        out=torch.zeros(2 * 8 * 8 * 16))
    with pytest.raises(ValueError, match="out holds"):
        neo.conv2d_int8_acc(xq, 16, wq, 32, 3, 3, pad=1,
                            out=torch.zeros(2 * 8 * 8 * 16 - 1, dtype=torch.int32))
    with pytest.raises(ValueError, match="out holds"):
        neo.pack_filter_int8(torch.zeros((32, 16, 3, 3)),
                             out=torch.zeros(100, dtype=torch.int8))
    with pytest.raises(ValueError, match="NCHW16c"):
        neo.quantize_int8(torch.zeros((1, 1, 8, 8, 16)), 17, 0.1)
    with pytest.raises(ValueError, match="out holds"):
        neo.quantize_int8(torch.zeros((1, 1, 8, 8, 16)), 16, 0.1, pad=1,
                          out=torch.zeros((1, 1, 8, 8, 16), dtype=torch.int8))


# ---- GPU -------------------------------------------------------------------------------------
def packed_filter_ref(wq):
    """The oracle's int8 KCRS filter in the library's packed order: block
    (kb, r, s, cg), lane (g, k) = 16 g + k, byte b holds
    q[16 kb + k][64 cg + 16 g + b][r][s] (zero padded)."""
    K, C, R, S = wq.shape
    KB, CG = -(-K // 16), -(-C // 64)
    p = np.zeros((KB * 16, CG * 64, R, S), np.int8)
    p[:K, :C] = wq
    # (kb, k, cg, g, b, r, s) -> (kb, r, s, cg, g, k, b)
    t = p.reshape(KB, 16, CG, 4, 16, R, S).transpose(0, 5, 6, 2, 3, 1, 4)
    return np.ascontiguousarray(t).reshape(-1)


def act_scale(x):
    """A per-tensor activation scale (the caller's calibration): max |x| / 127."""
    return np.float32(np.abs(x).max()) / np.float32(127)


def _pad16(v, K):
    p = np.zeros(-(-K // 16) * 16, np.float32)
    p[:K] = v
    return p


@pytest.fixture(scope="module")
def gpu():
    from gpu_util import torch_cuda
    torch_cuda()
    neo.lib()
    return neo


def run_int8(gpu, c, xs, raw=False, bias=True, out=None, y_off=0, y_tot=None):
    """One LayerCase (no batch norm) through the device chain: layout
    transform, activation quantization, filter packing, convolution."""
    from gpu_util import dev
    xq = gpu.quantize_int8(gpu.to_blocked(dev(c.x)), c.C, xs, pad=c.pad)
    wq, ws = gpu.pack_filter_int8(dev(c.w))
    if raw:
        return gpu.conv2d_int8_acc(xq, c.C, wq, c.K, c.R, c.S, stride=c.stride, pad=c.pad)
    res = gpu.to_blocked(dev(c.residual)) if c.epilogue == "res" else None
    act = "relu" if c.epilogue in ("relu", "res", "bias_relu") else "none"
    b = dev(_pad16(c.bias, c.K)) if bias and c.bias is not None else None
    return gpu.conv2d_int8(xq, c.C, wq, ws, c.K, c.R, c.S, xs, bias=b, stride=c.stride,
                           pad=c.pad, act=act, residual=res, out=out, y_cblk_offset=y_off,
                           y_cblk_total=y_tot)


def oracle_int8(c, xs, bias=True, images=None):
    """The oracle's integer chain: (exact accumulators, the ideal dequantized
    output, the magnitude |acc m| + |bias| + |residual| of the epilogue's
    terms, the float32 epilogue as the interface evaluates it)."""
    sel = slice(None) if images is None else images
    acc = oq.conv2d_int(oq.quantize(c.x[sel], xs), oq.quantize_filter(c.w)[0], c.stride, c.pad)
    m = oq.multipliers(xs, oq.filter_scales(c.w))
    b = c.bias if bias else None
    res = c.residual[sel] if c.epilogue == "res" else None
    act = "relu" if c.epilogue in ("relu", "res", "bias_relu") else "none"
    y = oq.dequantize(acc, m, b, res, act)
    mag = np.abs(acc * m.astype(np.float64)[None, :, None, None])
    if b is not None:
        mag = mag + np.abs(b.astype(np.float64))[None, :, None, None]
    if res is not None:
        mag = mag + np.abs(res.astype(np.float64))
    return acc, y, mag, oq.epilogue_f32(acc, m, b, res, act)


def assert_dequant_close(got, want, mag, what="", exact=None):
    """float32 epilogue: equal to the oracle's step-by-step float32 evaluation
    (`exact`), and within 6 u (|acc m| + |b| + |r|), u = 2^-24, of the ideal
    value (the int32 -> float32 conversion, the product, the bias and residual
    adds each round once, the ReLU is 1-Lipschitz, the ideal rounds once)."""
    if exact is not None:
        np.testing.assert_array_equal(got, exact, err_msg=what)
    got = np.asarray(got, np.float64)
    bound = 6 * 2.0 ** -24 * mag + 1e-30
    bad = np.abs(got - want) > bound
    assert not bad.any(), (f"{what}: {int(bad.sum())} outputs beyond the epilogue bound; max "
                           f"err {np.abs(got - want).max():.3e}")


def assert_acc_equal(acc_b, want, K, what=""):
    """Blocked int32 accumulators equal the oracle's, padding channels 0."""
    got = orc.from_blocked(acc_b, acc_b.shape[1] * 16)
    np.testing.assert_array_equal(got[:, :K], want, err_msg=what)
    assert (got[:, K:] == 0).all(), what + ": padding channels not zero"


@pytest.mark.gpu
@pytest.mark.parametrize("C,pad", [(1, (0, 0)), (16, (1, 1)), (37, (2, 1)), (64, (3, 0))])
def test_quantize_bit_exact(gpu, C, pad):
    """Round half to even on exact ties, clamping, and random values: the
    device's int8 NCHW16c equals the oracle's quantization inside the halo,
    padding lanes and the halo 0."""
    from gpu_util import dev, host
    rng = np.random.default_rng([C, 8])
    s = np.float32(0.25)
    x = rng.normal(0, 12, (2, C, 5, 7)).astype(np.float32)
    x.flat[::3] = s * (rng.integers(-140, 140, x.size)[::3] + 0.5)   # exact ties, some clamped
    q = host(gpu.quantize_int8(gpu.to_blocked(dev(x)), C, s, pad=pad))
    ph, pw = pad
    want = np.zeros((2, C, 5 + 2 * ph, 7 + 2 * pw), np.int8)
    want[:, :, ph:ph + 5, pw:pw + 7] = oq.quantize(x, s)
    np.testing.assert_array_equal(q, orc.to_blocked(want))


@pytest.mark.gpu
@pytest.mark.parametrize("K,C,R,S", [(64, 64, 3, 3), (40, 17, 3, 3), (5, 3, 7, 7), (1, 1, 1, 1),
                                     (33, 130, 1, 7), (20, 256, 1, 1)])
def test_pack_filter_bit_exact(gpu, K, C, R, S):
    from gpu_util import dev, host
    w = np.random.default_rng([K, C, R, S]).normal(0, 0.1, (K, C, R, S)).astype(np.float32)
    if K > 4:
        w[3] = 0.0                                  # an all-zero output channel: scale 1
    wq, ws = gpu.pack_filter_int8(dev(w))
    q, s = oq.quantize_filter(w)
    np.testing.assert_array_equal(host(wq), packed_filter_ref(q))
    want_s = np.ones(-(-K // 16) * 16, np.float32)
    want_s[:K] = s
    np.testing.assert_array_equal(host(ws), want_s)


ACC_CASES = [
    # C, K, R, S, stride, pad, H, W, N
    (64, 64, 1, 1, 1, 0, 7, 7, 2),          # pointwise, one channel group
    (3, 16, 3, 3, 1, 1, 9, 9, 1),           # three channels (one block, three lanes)
    (17, 40, 3, 3, 1, 1, 11, 13, 1),        # ragged C and K, ragged pixel tile
    (64, 128, 3, 3, 2, 1, 15, 15, 1),       # stride 2
    (3, 64, 7, 7, 2, 3, 32, 32, 1),         # a stem: 7x7 stride 2 pad 3
    (256, 512, 1, 1, 2, 0, 14, 14, 1),      # strided projection
    (512, 512, 3, 3, 1, 1, 7, 7, 1),        # 72 reduction steps
    (128, 192, 1, 7, 1, (0, 3), 17, 17, 1),  # Inception 1x7
    (192, 160, 7, 1, 1, (3, 0), 17, 17, 1),  # Inception 7x1
    (1, 1, 1, 1, 1, 0, 1, 1, 1),            # the degenerate case
    (48, 32, 3, 3, 1, 0, 5, 9, 3),          # valid padding, N = 3, odd step count
    (80, 96, 5, 5, 1, 2, 6, 6, 2),          # 5x5, two channel groups (the second ragged)
]


@pytest.mark.gpu
@pytest.mark.parametrize("e", ACC_CASES, ids=[f"C{e[0]}K{e[1]}{e[2]}x{e[3]}s{e[4]}p{e[5]}H{e[6]}"
                                              f"W{e[7]}N{e[8]}" for e in ACC_CASES])
def test_accumulators_bit_exact(gpu, e):
    from gpu_util import host
    C, K, R, S, st, pd, H, W, N = e
    c = wl.conv_case(C, K, R, S, st, pd, H, W, N=N, epilogue="none", with_bn=False)
    xs = act_scale(c.x)
    print(f"\n[int8] acc {e}", flush=True)
    acc, _, _, _ = oracle_int8(c, xs)
    assert_acc_equal(host(run_int8(gpu, c, xs, raw=True)), acc, K, str(e))


@pytest.mark.gpu
@pytest.mark.parametrize("C,H,sign", [(512, 4, 1), (1024, 6, -1)])
def test_accumulators_at_the_extremes(gpu, C, H, sign):
    """All inputs and weights at +-127 after quantization: sums up to
    127^2 * 9 * 1024 = 148,644,864, exact (float32 would round them)."""
    from gpu_util import host
    c = wl.conv_case(C, 16, 3, 3, 1, 1, H, H, epilogue="none", with_bn=False)
    c.x = np.full_like(c.x, sign * 1.0)
    c.w = np.ones_like(c.w)
    c.w[5] = -1.0
    xs = act_scale(c.x)
    acc, _, _, _ = oracle_int8(c, xs)
    assert np.abs(acc).max() == 127 * 127 * 9 * C
    assert_acc_equal(host(run_int8(gpu, c, xs, raw=True)), acc, 16, f"extreme C={C}")


@pytest.mark.gpu
@pytest.mark.parametrize("epi", ["none", "bias_relu", "res", "nobias"])
def test_dequantized_output(gpu, epi):
    """act(acc * s_x * s_w[k] + bias + residual) in float32 against the
    oracle's float64 epilogue, within the epilogue's rounding bound."""
    from gpu_util import host
    e = "none" if epi == "nobias" else epi
    c = wl.conv_case(64, 80, 3, 3, 1, 1, 10, 9, N=2, epilogue=e, with_bn=False,
                     out_hw=(10, 9))
    xs = act_scale(c.x)
    _, want, mag, y32 = oracle_int8(c, xs, bias=epi != "nobias")
    got = orc.from_blocked(host(run_int8(gpu, c, xs, bias=epi != "nobias")), 80)
    assert_dequant_close(got, want, mag, epi, y32)


@pytest.mark.gpu
def test_concat_view(gpu):
    """The output written into blocks [2, 5) of a 6-block buffer, the others
    untouched."""
    import torch
    from gpu_util import host
    c = wl.conv_case(24, 40, 3, 3, 1, 1, 9, 9, N=2, epilogue="relu", with_bn=False)
    xs = act_scale(c.x)
    buf = torch.full((2, 6, 9, 9, 16), 7.0, device="cuda")
    run_int8(gpu, c, xs, out=buf, y_off=2, y_tot=6)
    b = host(buf)
    _, want, mag, y32 = oracle_int8(c, xs)
    assert_dequant_close(orc.from_blocked(np.ascontiguousarray(b[:, 2:5]), 40), want, mag, "view", y32)
    assert (b[:, :2] == 7).all() and (b[:, 5:] == 7).all()


CONFIGS = [f"{fk},{fp},{wv}" for fk, fp in [(1, 1), (1, 2), (2, 1), (2, 2), (4, 2), (2, 4), (4, 4)]
           for wv in (1, 2, 4)]


@pytest.mark.gpu
@pytest.mark.parametrize("cfg", CONFIGS)
def test_every_configuration(gpu, cfg, monkeypatch):
    """Each launch configuration (forced): register tiles and waves splitting
    the reduction, on 18 steps (two channel groups, the second ragged) and on
    9 steps (odd: the two-step loop's tail), a ragged pixel tile, residual +
    ReLU; a second run gives the same bits."""
    from gpu_util import host
    monkeypatch.setenv("NEO_I8_CONFIG", cfg)
    for C, H, W, N in [(80, 13, 11, 2), (48, 7, 9, 1)]:
        c = wl.conv_case(C, 64, 3, 3, 1, 1, H, W, N=N, epilogue="res", with_bn=False,
                         out_hw=(H, W))
        xs = act_scale(c.x)
        print(f"\n[int8] forced {cfg} C={C}", flush=True)
        acc, want, mag, y32 = oracle_int8(c, xs)
        a1 = host(run_int8(gpu, c, xs, raw=True))
        assert_acc_equal(a1, acc, 64, cfg)
        np.testing.assert_array_equal(a1, host(run_int8(gpu, c, xs, raw=True)))
        assert_dequant_close(orc.from_blocked(host(run_int8(gpu, c, xs)), 64), want, mag, cfg, y32)


@pytest.mark.gpu
@pytest.mark.parametrize("cfg", ["8,2,1", "8,2,4", "8,4,1", "8,4,2"])
def test_eight_block_tiles(gpu, cfg, monkeypatch):
    """The 8-output-block tiles (K a multiple of 128): a 1x1 over four channel
    groups and a 3x3 with a ragged pixel tile and residual + ReLU, the sums
    and both outputs against the oracle (the configuration is checked to be
    one the kernel takes, so the override is not silently ignored)."""
    from gpu_util import host
    fk, fp, wv = map(int, cfg.split(","))
    monkeypatch.setenv("NEO_I8_CONFIG", cfg)
    for C, R, H, N in [(200, 1, 9, 2), (80, 3, 13, 1)]:
        c = wl.conv_case(C, 128, R, R, 1, R // 2, H, H, N=N, epilogue="res", with_bn=False,
                         out_hw=(H, H))
        assert R * R * -(-C // 64) >= wv and 8 % fk == 0
        xs = act_scale(c.x)
        acc, want, mag, y32 = oracle_int8(c, xs)
        assert_acc_equal(host(run_int8(gpu, c, xs, raw=True)), acc, 128, cfg)
        assert_dequant_close(orc.from_blocked(host(run_int8(gpu, c, xs)), 128), want, mag, cfg, y32)
        ys = act_scale(y32)
        np.testing.assert_array_equal(host(run_int8_q(gpu, c, xs, ys, (1, 1))),
                                      requant_ref(y32, ys, 128, (1, 1)), err_msg=cfg)


@pytest.mark.gpu
@pytest.mark.parametrize("lid", ["R01", "R03", "R08", "R11", "R19", "R23"])
def test_resnet50_layers_batch32_sampled(gpu, lid):
    """ResNet-50 layers at batch 32 in the launch configuration the library
    chooses: the convolution is per image, so the oracle on images 0 and 31
    checks those outputs bit for bit (accumulators) and to the epilogue bound."""
    from gpu_util import host
    _, C, K, R, st, pd, H, _, _ = {e[0]: e for e in wl.RESNET50_LAYERS}[lid]
    c = wl.conv_case(C, K, R, R, st, pd, H, H, N=32, epilogue="bias_relu", with_bn=False)
    xs = act_scale(c.x)
    print(f"\n[int8] {lid} batch 32", flush=True)
    acc_b = host(run_int8(gpu, c, xs, raw=True))[[0, 31]]
    y_b = host(run_int8(gpu, c, xs))[[0, 31]]
    acc, want, mag, y32 = oracle_int8(c, xs, images=[0, 31])
    assert_acc_equal(acc_b, acc, c.K, lid)
    assert_dequant_close(orc.from_blocked(y_b, c.K), want, mag, lid, y32)


@pytest.mark.gpu
@pytest.mark.parametrize("cfg,N", [("1,1,4", 6), ("1,1,2", 12)])
def test_workgroups_taking_several_tiles(gpu, cfg, N, monkeypatch):
    """A grid above two rounds of the chip's SIMDs: the workgroups take
    several output tiles in turn (600 tiles for 512 workgroups of 4 waves,
    1200 for 1024 of 2), accumulators and output against the oracle."""
    from gpu_util import host
    monkeypatch.setenv("NEO_I8_CONFIG", cfg)
    c = wl.conv_case(64, 16, 3, 3, 1, 1, 40, 40, N=N, epilogue="res", with_bn=False,
                     out_hw=(40, 40))
    xs = act_scale(c.x)
    acc, want, mag, y32 = oracle_int8(c, xs)
    assert_acc_equal(host(run_int8(gpu, c, xs, raw=True)), acc, 16, cfg)
    assert_dequant_close(orc.from_blocked(host(run_int8(gpu, c, xs)), 16), want, mag, cfg, y32)


# ---- int8 output: the float32 epilogue requantized into the next layer's input ----------------
def run_int8_q(gpu, c, xs, ys, out_pad, out=None, y_off=0, y_tot=None):
    from gpu_util import dev
    xq = gpu.quantize_int8(gpu.to_blocked(dev(c.x)), c.C, xs, pad=c.pad)
    wq, ws = gpu.pack_filter_int8(dev(c.w))
    res = gpu.to_blocked(dev(c.residual)) if c.epilogue == "res" else None
    act = "relu" if c.epilogue in ("relu", "res", "bias_relu") else "none"
    b = dev(_pad16(c.bias, c.K)) if c.bias is not None else None
    return gpu.conv2d_int8_q(xq, c.C, wq, ws, c.K, c.R, c.S, xs, ys, bias=b, stride=c.stride,
                             pad=c.pad, act=act, residual=res, out_pad=out_pad, out=out,
                             y_cblk_offset=y_off, y_cblk_total=y_tot)


def requant_ref(y32, ys, K, out_pad, blocks=None):
    """The oracle's requantized output in the blocked layout with its halo
    (zeros), padding channels 0."""
    q = oq.requantize(y32, ys)
    N, _, OH, OW = q.shape
    ph, pw = out_pad
    full = np.zeros((N, q.shape[1], OH + 2 * ph, OW + 2 * pw), np.int8)
    full[:, :, ph:ph + OH, pw:pw + OW] = q
    return orc.to_blocked(full)


Q_CASES = [
    # C, K, R, stride, pad, H, N, epilogue, out_pad
    (64, 64, 3, 1, 1, 14, 2, "relu", (1, 1)),       # a 3x3 feeding a 3x3
    (48, 40, 1, 1, 0, 9, 1, "none", (0, 0)),        # ragged K, signed output, no halo
    (32, 80, 3, 2, 1, 15, 3, "relu", (2, 1)),       # stride 2, uneven halo
    (64, 48, 1, 1, 0, 7, 2, "res", (1, 1)),         # residual + ReLU
]


@pytest.mark.gpu
@pytest.mark.parametrize("e", Q_CASES, ids=[f"C{e[0]}K{e[1]}r{e[2]}s{e[3]}{e[7]}q{e[8][0]}{e[8][1]}"
                                            for e in Q_CASES])
def test_requantized_output_bit_exact(gpu, e):
    """int8 output against the oracle's float32 epilogue requantized by the
    float32 reciprocal of the output scale, the halo zero; the output scale is
    the float output's max |y| / 127 (the next layer's calibration)."""
    from gpu_util import host
    C, K, R, st, pd, H, N, epi, qpad = e
    OH = (H + 2 * pd - R) // st + 1
    c = wl.conv_case(C, K, R, R, st, pd, H, H, N=N, epilogue=epi, with_bn=False, out_hw=(OH, OH))
    xs = act_scale(c.x)
    _, _, _, y32 = oracle_int8(c, xs)
    ys = act_scale(y32) if np.abs(y32).max() > 0 else np.float32(1)
    got = host(run_int8_q(gpu, c, xs, ys, qpad))
    np.testing.assert_array_equal(got, requant_ref(y32, ys, K, qpad), err_msg=str(e))


@pytest.mark.gpu
def test_requantized_view_keeps_the_rest(gpu):
    """Written into blocks [1, 4) of a 5-block int8 buffer prefilled with 7: the
    other blocks and the halo keep their bytes."""
    import torch
    from gpu_util import host
    c = wl.conv_case(24, 40, 3, 3, 1, 1, 9, 9, N=2, epilogue="relu", with_bn=False)
    xs = act_scale(c.x)
    _, _, _, y32 = oracle_int8(c, xs)
    ys = act_scale(y32)
    buf = torch.full((2, 5, 11, 11, 16), 7, dtype=torch.int8, device="cuda")
    run_int8_q(gpu, c, xs, ys, (1, 1), out=buf, y_off=1, y_tot=5)
    b = host(buf)
    want = requant_ref(y32, ys, 40, (1, 1))
    np.testing.assert_array_equal(b[:, 1:4, 1:10, 1:10], want[:, :, 1:10, 1:10])
    assert (b[:, 0] == 7).all() and (b[:, 4] == 7).all()
    inner = np.zeros(b.shape, bool)
    inner[:, :, 1:10, 1:10] = True
    assert (b[~inner] == 7).all()


@pytest.mark.gpu
@pytest.mark.parametrize("cfg", ["1,1,1", "2,2,2", "4,2,4", "4,4,1", "2,4,2"])
def test_requantized_every_tile(gpu, cfg, monkeypatch):
    from gpu_util import host
    monkeypatch.setenv("NEO_I8_CONFIG", cfg)
    c = wl.conv_case(80, 64, 3, 3, 1, 1, 13, 11, N=2, epilogue="res", with_bn=False,
                     out_hw=(13, 11))
    xs = act_scale(c.x)
    _, _, _, y32 = oracle_int8(c, xs)
    ys = act_scale(y32)
    np.testing.assert_array_equal(host(run_int8_q(gpu, c, xs, ys, (1, 2))),
                                  requant_ref(y32, ys, 64, (1, 2)), err_msg=cfg)


@pytest.mark.gpu
def test_two_layer_int8_chain(gpu):
    """conv 1 (3x3, int8 output with conv 2's halo) -> conv 2 (3x3) reading it
    directly: conv 2's sums against the oracle's chain, bit for bit."""
    from gpu_util import dev, host
    c1 = wl.conv_case(32, 48, 3, 3, 1, 1, 12, 10, N=2, epilogue="bias_relu", with_bn=False)
    rng = np.random.default_rng(44)
    w2 = rng.normal(0, np.sqrt(2 / (48 * 9)), (64, 48, 3, 3)).astype(np.float32)
    xs = act_scale(c1.x)
    _, _, _, y32 = oracle_int8(c1, xs)
    ys = act_scale(y32)
    # oracle chain: requantize, then the integer conv of layer 2
    want = oq.conv2d_int(oq.requantize(y32, ys), oq.quantize_filter(w2)[0], 1, 1)
    # device chain
    q1 = run_int8_q(gpu, c1, xs, ys, (1, 1))
    wq2, _ = gpu.pack_filter_int8(dev(w2))
    acc2 = gpu.conv2d_int8_acc(q1, 48, wq2, 64, 3, 3, stride=1, pad=1)
    assert_acc_equal(host(acc2), want, 64, "chain")


# ---- integer dense layer -----------------------------------------------------------------
@pytest.mark.gpu
@pytest.mark.parametrize("N,IN,OUT", [(1, 1000, 10), (3, 37, 1000), (20, 512, 64), (40, 4096, 17)])
def test_dense_int8_against_the_oracle(gpu, N, IN, OUT):
    """The packed rows and scales, the quantized input rows (padding 0), the
    float32 output with and without ReLU and its requantized rows, bit-exact
    against the oracle's integer dense layer (quantize_filter per row,
    dense_int, epilogue_f32, requantize); 40 images take two launches."""
    from gpu_util import dev, host
    rng = np.random.default_rng(N * 7919 + IN + OUT)
    x = rng.uniform(-1, 1, (N, IN)).astype(np.float32)
    w = (rng.standard_normal((OUT, IN)) * np.sqrt(2.0 / IN)).astype(np.float32)
    b = rng.normal(0, 0.1, OUT).astype(np.float32)
    xs = oq.act_scale(x)
    wq, ws = oq.quantize_filter(w.reshape(OUT, IN, 1, 1))
    wq = wq.reshape(OUT, IN)
    rows, scale = neo.pack_dense_int8(dev(w))
    r = host(rows)
    np.testing.assert_array_equal(r[:, :IN], wq)
    assert (r[:, IN:] == 0).all()
    np.testing.assert_array_equal(host(scale), ws)
    xq = neo.quantize_rows_int8(dev(x), xs)
    q = host(xq)
    np.testing.assert_array_equal(q[:, :IN], oq.quantize(x, xs))
    assert (q[:, IN:] == 0).all()
    acc = oq.dense_int(oq.quantize(x, xs), wq)
    for act in ("none", "relu"):
        y, _ = neo.dense_int8(xq, IN, rows, scale, OUT, xs, bias=dev(b), act=act)
        ref = oq.epilogue_f32(acc[:, :, None, None], oq.multipliers(xs, ws), b, None, act)[:, :, 0, 0]
        np.testing.assert_array_equal(host(y), ref)
    ys = oq.act_scale(ref)
    y2, yq = neo.dense_int8(xq, IN, rows, scale, OUT, xs, bias=dev(b), act="relu", y_scale=ys)
    np.testing.assert_array_equal(host(y2), ref)
    got = host(yq)
    np.testing.assert_array_equal(got[:, :OUT], oq.requantize(ref, ys))
    assert (got[:, OUT:] == 0).all()
    # the int8 rows alone
    _, yq2 = neo.dense_int8(xq, IN, rows, scale, OUT, xs, bias=dev(b), act="relu", out=False, y_scale=ys)
    np.testing.assert_array_equal(host(yq2), got)


@pytest.mark.gpu
def test_dense_int8_extreme_sums(gpu):
    """Every value +-127 over 25,088 inputs (VGG-16's first dense layer): the
    sums reach 127^2 * 25,088 = 404,654,592 and stay exact."""
    from gpu_util import dev, host
    IN, OUT, N = 25088, 32, 2
    x = np.ones((N, IN), np.float32)
    x[1] = -1.0
    w = np.ones((OUT, IN), np.float32)
    w[1::2] = -1.0
    rows, scale = neo.pack_dense_int8(dev(w))
    xq = neo.quantize_rows_int8(dev(x), 1.0 / 127)
    y, _ = neo.dense_int8(xq, IN, rows, scale, OUT, np.float32(1.0 / 127))
    acc = oq.dense_int(oq.quantize(x, np.float32(1.0 / 127)), oq.quantize_filter(w.reshape(OUT, IN, 1, 1))[0]
                       .reshape(OUT, IN))
    assert int(np.abs(acc).max()) == 127 * 127 * IN
    ref = oq.epilogue_f32(acc[:, :, None, None], oq.multipliers(np.float32(1.0 / 127), host(scale)))[:, :, 0, 0]
    np.testing.assert_array_equal(host(y), ref)
