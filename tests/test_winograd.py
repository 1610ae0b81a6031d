"""Winograd F(2x2, 3x3) convolution (neo_winograd_filter, neo_conv2d_winograd):
argument handling on the host, and on the GPU parity with the oracle's direct
convolution on seeded inputs -- configuration 1, the ResNet-50 and VGG-16 3x3
stride-1 layers, ragged and degenerate shapes, every launch configuration."""
import ctypes

import numpy as np
import pytest

import oracle as orc
from paper_1809_02697_amd import neo
from paper_1809_02697_amd import workloads as wl

FAKE = ctypes.c_void_p(1 << 20)   # aligned, never dereferenced: validation fails first
MIS = ctypes.c_void_p((1 << 20) + 4)


def _call(x=FAKE, C=16, H=8, pd=(1, 1), yt=1, u=FAKE):
    return neo.lib().neo_conv2d_winograd(x, 1, C, H, 8, u, 16, None, pd[0], pd[1], None, FAKE, 0,
                                         yt, None)


def test_argument_errors():
    """Validation before any device work, the entry point named in the message."""
    assert _call(x=None) == -1 and "neo_conv2d_winograd" in neo.last_error()
    assert _call(u=MIS) == -3
    assert _call(C=0) == -1
    assert _call(C=4) == -4 and "4 input channels" in neo.last_error()
    assert _call(H=2, pd=(0, 0)) == -2          # OH = 0
    assert _call(pd=(-1, 1)) == -1
    assert _call(yt=0) == -2
    L = neo.lib()
    assert L.neo_winograd_filter(None, 16, 16, FAKE, None) == -1
    assert L.neo_winograd_filter(FAKE, 0, 16, FAKE, None) == -1


def test_binding_refuses_short_buffers():
    import torch
    x = torch.zeros((1, 1, 8, 8, 16))
    u = torch.zeros((2, 1, 16, 256))
    with pytest.raises(ValueError, match="u holds"):
        neo.conv2d_winograd(x, 16, u[:1], 32, out=torch.zeros((1, 2, 8, 8, 16)))
    with pytest.raises(ValueError, match="out"):
        neo.conv2d_winograd(x, 16, u, 32, out=torch.zeros(2 * 8 * 8 * 16 - 1))
    with pytest.raises(ValueError, match="residual"):
        neo.conv2d_winograd(x, 16, u, 32, residual=torch.zeros(7), out=torch.zeros((1, 2, 8, 8, 16)))
    with pytest.raises(ValueError, match="3x3"):
        neo.winograd_filter(torch.zeros((16, 16, 1, 1)))
    with pytest.raises(ValueError, match="NCHW16c"):
        neo.conv2d_winograd(torch.zeros((1, 2, 8, 8, 16)), 16, u, 32)


# ---- GPU -------------------------------------------------------------------------------------
G = np.array([[1, 0, 0], [0.5, 0.5, 0.5], [0.5, -0.5, 0.5], [0, 0, 1]])


def wino_filter_ref(w):
    """G w G^T in float64 per (k, c), rounded once, in the kernel's element
    blocks [kb][cb][e][(c%16)/4 * 16 + k%16][c%4]."""
    K, C = w.shape[:2]
    KB, CB = -(-K // 16), -(-C // 16)
    U = np.einsum("ir,kcrs,js->kcij", G, w.astype(np.float64), G).astype(np.float32)
    Up = np.zeros((KB * 16, CB * 16, 4, 4), np.float32)
    Up[:K, :C] = U
    # (kb, kk, cb, cq, ci, i, j) -> (kb, cb, i, j, cq, kk, ci)
    t = Up.reshape(KB, 16, CB, 4, 4, 4, 4).transpose(0, 2, 5, 6, 3, 1, 4)
    return np.ascontiguousarray(t).reshape(KB, CB, 16, 256)


@pytest.fixture(scope="module")
def gpu():
    from gpu_util import torch_cuda
    torch_cuda()
    neo.lib()
    return neo


def run_wino(gpu, c, out=None, y_off=0, y_tot=None):
    """One LayerCase through the Winograd path: fold (host), the filter
    transform (device), the convolution.  Returns the NCHW16c output."""
    from gpu_util import dev
    assert (c.R, c.S) == (3, 3) and tuple(c.stride) == (1, 1)
    if c.bn is not None:
        w, b = gpu.fold_bn(c.w, c.bias, c.bn["gamma"], c.bn["beta"], c.bn["mean"], c.bn["var"],
                           c.bn["eps"])
    else:
        w, b = c.w, c.bias
    bp = None
    if b is not None:
        bpad = np.zeros(-(-c.K // 16) * 16, np.float32)
        bpad[:c.K] = b
        bp = dev(bpad)
    u = gpu.winograd_filter(dev(w))
    xb = gpu.to_blocked(dev(c.x))
    res = gpu.to_blocked(dev(c.residual)) if c.epilogue == "res" else None
    act = "relu" if c.epilogue in ("relu", "res", "bias_relu") else "none"
    return gpu.conv2d_winograd(xb, c.C, u, c.K, bias=bp, pad=c.pad, act=act, residual=res,
                               out=out, y_cblk_offset=y_off, y_cblk_total=y_tot)


@pytest.mark.gpu
@pytest.mark.parametrize("K,C", [(64, 64), (40, 17), (5, 3), (1, 1), (33, 80)])
def test_filter_transform(gpu, K, C):
    from gpu_util import dev, host
    w = np.random.default_rng([K, C]).normal(0, 0.1, (K, C, 3, 3)).astype(np.float32)
    got = host(gpu.winograd_filter(dev(w)))
    want = wino_filter_ref(w)
    # float64 sums of float32 values rounded once: equal up to the rounding
    # of the last bit when the order of the sums differs
    np.testing.assert_allclose(got, want, rtol=2.0 ** -23, atol=1e-30)
    assert ((got == 0) == (want == 0)).all()    # the padding of K and C exactly zero


@pytest.mark.gpu
def test_config1(gpu):
    """Configuration 1 (3x3, 64 -> 64, 56x56, bias + ReLU) in NCHW after the
    round trip, against the oracle."""
    from gpu_util import assert_close, host
    g = wl.single_conv(0)
    n = g.nodes[1]
    c = wl.LayerCase("cfg1", 64, 64, 3, 3, (1, 1), (1, 1), 56, 56, 1, "bias_relu", 1, g.x, n.w,
                     n.bias, None, None)
    y = host(neo.from_blocked(run_wino(gpu, c), 64))
    assert_close(y, orc.run_graph(g), "winograd config 1")


@pytest.mark.gpu
@pytest.mark.parametrize("lid", ["R03", "R11", "R17", "R23"])
def test_resnet50_3x3_layers(gpu, lid):
    from gpu_util import assert_close, host
    case = {c.id: c for c in wl.resnet50_layer_sweep(1)}[lid]
    yb = host(run_wino(gpu, case))
    assert_close(orc.from_blocked(yb, case.K), orc.layer_forward(case), lid)
    lanes = yb.transpose(0, 1, 4, 2, 3).reshape(1, -1, *yb.shape[2:4])[:, case.K:]
    assert (lanes == 0).all()


EDGE = [
    # C, K, pad, H, W, N, epilogue
    (5, 7, 1, 9, 11, 2, "relu"),        # ragged C and K, odd output (ragged last tiles), N = 2
    (17, 40, 1, 15, 13, 1, "relu"),     # C one past a block
    (64, 64, 0, 10, 7, 1, "relu"),      # valid padding: 8 x 5 output
    (32, 48, 2, 6, 5, 1, "none"),       # pad 2: the patch's border rows are padding
    (16, 16, 1, 1, 1, 1, "relu"),       # 1x1 input: one tile, three quarters clipped
    (48, 32, 1, 2, 3, 3, "none"),       # tiny maps, N = 3
    (64, 256, 1, 7, 7, 3, "res"),       # residual, N = 3
    (80, 96, 1, 17, 17, 1, "relu"),     # Inception 17x17 width, C = 80
    (256, 256, 1, 14, 14, 2, "res"),
    (512, 512, 1, 7, 7, 1, "relu"),
]


@pytest.mark.gpu
@pytest.mark.parametrize("e", EDGE, ids=[f"C{e[0]}K{e[1]}p{e[2]}H{e[3]}W{e[4]}N{e[5]}{e[6]}"
                                         for e in EDGE])
def test_edge_cases(gpu, e):
    from gpu_util import assert_close, host
    C, K, pd, H, W, N, epi = e
    OH, OW = H + 2 * pd - 2, W + 2 * pd - 2
    c = wl.conv_case(C, K, 3, 3, 1, pd, H, W, N=N, epilogue=epi, out_hw=(OH, OW))
    print(f"\n[winograd] {e}", flush=True)
    y = orc.from_blocked(host(run_wino(gpu, c)), K)
    assert_close(y, orc.layer_forward(c), str(e))


@pytest.mark.gpu
def test_concat_view(gpu):
    """The output written into blocks [2, 2 + ceil(K/16)) of a 6-block buffer,
    the other blocks untouched."""
    import torch
    from gpu_util import assert_close, host
    c = wl.conv_case(24, 40, 3, 3, 1, 1, 9, 9, N=2, epilogue="relu")
    buf = torch.full((2, 6, 9, 9, 16), 7.0, device="cuda")
    run_wino(gpu, c, out=buf, y_off=2, y_tot=6)
    b = host(buf)
    assert_close(orc.from_blocked(np.ascontiguousarray(b[:, 2:5]), 40), orc.layer_forward(c), "view")
    assert (b[:, :2] == 7).all() and (b[:, 5:] == 7).all()


CONFIGS = ["1,1,1,1", "1,1,1,2", "1,1,1,4", "1,1,1,8", "2,1,1,1", "2,1,1,4", "1,2,1,1", "1,2,1,4",
           "1,1,2,4", "1,1,4,2", "2,1,3,1", "1,2,5,2", "1,1,5,1"]


@pytest.mark.gpu
@pytest.mark.parametrize("cfg", CONFIGS)
def test_every_configuration(gpu, cfg, monkeypatch):
    """Each launch configuration (forced): register tiles, waves splitting the
    channel blocks, splits across workgroups with the reduction kernel, on a
    case with several tile groups, a ragged tile group, five channel blocks
    (uneven splits) and residual + ReLU; a second run gives the same bits."""
    from gpu_util import assert_close, host
    monkeypatch.setenv("NEO_WINO_CONFIG", cfg)
    c = wl.conv_case(80, 64, 3, 3, 1, 1, 13, 11, N=2, epilogue="res", out_hw=(13, 11))
    print(f"\n[winograd] forced {cfg}", flush=True)
    y1 = host(run_wino(gpu, c))
    y2 = host(run_wino(gpu, c))
    np.testing.assert_array_equal(y1, y2)
    assert_close(orc.from_blocked(y1, 64), orc.layer_forward(c), cfg)


@pytest.mark.gpu
def test_vgg16_layer(gpu):
    """A VGG-16 3x3 layer (256 -> 256 at 56x56, batch 1), against the oracle."""
    from gpu_util import assert_close, host
    c = wl.conv_case(256, 256, 3, 3, 1, 1, 56, 56, N=1, epilogue="relu", with_bn=False)
    assert_close(orc.from_blocked(host(run_wino(gpu, c)), 256), orc.layer_forward(c), "vgg 256")


# ---- the plan (NEO_PLAN_WINOGRAD) ---------------------------------------------------------------
def _host_desc(g, flags):
    p = neo.Plan(g, flags=flags | neo.PLAN_HOST_ONLY)
    d = p.describe()
    p.destroy()
    return d


def _algos(d):
    return [s["conv"]["algo"] for s in d["steps"] if s["kind"] == "conv"]


def test_planner_marks_the_3x3_stride1_convs():
    """Untuned, every 3x3 stride-1 conv launched alone with more than 4 input
    channels runs the Winograd kernel; the rest, and every conv of a plan
    without the flag, the direct kernel."""
    g = wl.resnet50(1)
    d = _host_desc(g, neo.PLAN_WINOGRAD)
    want = sum(1 for n in g.nodes if n.op == "conv" and (n.R, n.S) == (3, 3) and n.stride == (1, 1))
    assert want == 13                       # 3 + 4 - 1 + 6 - 1 + 3 - 1 bottlenecks at stride 1
    assert _algos(d).count("winograd") == want
    for s in d["steps"]:
        if s["kind"] == "conv" and s["conv"]["algo"] == "winograd":
            c = s["conv"]
            assert (c["R"], c["S"], tuple(c["stride"]), c["ic_bn"], c["oc_bn"]) == (3, 3, (1, 1), 16, 16)
    assert set(_algos(_host_desc(g, 0))) == {"direct"}
    v = _host_desc(wl.vgg16(1), neo.PLAN_WINOGRAD)
    assert _algos(v).count("winograd") == 12   # every conv but the 3-channel stem
    # convs fused into another launch keep their own kernel
    f = _host_desc(g, neo.PLAN_WINOGRAD | neo.PLAN_FUSE_PAIRS | neo.PLAN_FUSE_CHAINS)
    assert _algos(f).count("winograd") == want - 3


def test_results_file_wino_entries(tmp_path):
    """A Winograd entry round-trips through the results file; one naming a
    configuration the kernel does not take for its shape fails the load."""
    neo.tune_db_clear()
    good = tmp_path / "good.txt"
    good.write_text("wino gfx950 32 256 14 14 256 1 1 2 1 1 2 59.25\n")
    assert neo.tune_db_load(good) == 1 and neo.tune_db_size() == 1
    out = tmp_path / "out.txt"
    assert neo.tune_db_save(out) == 1
    assert out.read_text().split() == good.read_text().split()
    bad = tmp_path / "bad.txt"
    bad.write_text("wino gfx950 1 64 8 8 16 1 1 2 1 1 1 5.0\n")     # fk 2 > the one output block
    with pytest.raises(neo.NeoError):
        neo.tune_db_load(bad)
    neo.tune_db_clear()


@pytest.mark.gpu
def test_plan_vgg16_b1_all_winograd(gpu):
    """VGG-16 batch 1 with its twelve 3x3 stride-1 convs on the Winograd kernel
    (untuned), against the oracle's logits."""
    from gpu_util import assert_close_network, dev, host, oracle_output
    g = wl.vgg16(1)
    p = gpu.Plan(g, flags=gpu.PLAN_WINOGRAD)
    assert _algos(p.describe()).count("winograd") == 12
    y = host(p.run(dev(g.x)))
    p.destroy()
    ref = oracle_output(g)
    assert_close_network(y, ref, "vgg16 b1 winograd", graph=g)
    assert (np.argmax(y, 1) == np.argmax(ref, 1)).all()


@pytest.mark.gpu
@pytest.mark.parametrize("model,N", [("resnet50", 32), ("vgg16", 32)])
def test_plan_tuned_batch32(gpu, model, N):
    """Batch 32, tuned: the local search keeps the Winograd kernel where it
    measures faster; all 32 images against the oracle, two runs bit-identical,
    and a plan rebuilt from the saved results makes the same choices."""
    import os
    import tempfile
    import torch
    from gpu_util import assert_close_network, dev, host, oracle_output
    g = wl.MODELS[model](N)
    gpu.tune_db_clear()
    p = gpu.Plan(g, flags=gpu.PLAN_WINOGRAD | gpu.PLAN_TUNE)
    d = p.describe()
    algos = _algos(d)
    print(f"\n{model} b{N}: {algos.count('winograd')} of {len(algos)} convs by Winograd", flush=True)
    x = dev(g.x)
    out = torch.empty((N, 1000), device="cuda")
    p.run(x, out)
    y = host(out)
    p.run(x, out)
    np.testing.assert_array_equal(host(out), y)
    p.destroy()
    with tempfile.TemporaryDirectory() as tmp:
        path = os.path.join(tmp, "db.txt")
        gpu.tune_db_save(path)
        gpu.tune_db_clear()
        gpu.tune_db_load(path)
        p2 = gpu.Plan(g, flags=gpu.PLAN_WINOGRAD | gpu.PLAN_TUNE)
        assert _algos(p2.describe()) == algos
        p2.destroy()
    ref = oracle_output(g)
    assert_close_network(y, ref, f"{model} b{N} winograd tuned", graph=g)
    for i in range(N):
        assert_close_network(y[i:i + 1], ref[i:i + 1], f"{model} b{N} winograd image {i}")


@pytest.mark.gpu
def test_tuned_plan_compares_even_with_stored_direct_configs(gpu, tmp_path):
    """A tuned plan times the Winograd kernel for every 3x3 stride-1 conv also
    when the results database already holds the direct configurations (from
    an earlier plan), and runs it only where it measured faster."""
    from gpu_util import dev, host, oracle_output, assert_close_network
    g = wl.resnet50(1)
    gpu.tune_db_clear()
    gpu.Plan(g, flags=gpu.PLAN_TUNE).destroy()          # direct configurations stored
    p = gpu.Plan(g, flags=gpu.PLAN_TUNE | gpu.PLAN_WINOGRAD)
    path = tmp_path / "db.txt"
    gpu.tune_db_save(path)
    wino = {tuple(int(v) for v in l.split()[2:9]): float(l.split()[-1])
            for l in open(path) if l.startswith("wino ")}
    assert len(wino) == 4                                 # R03, R11, R17, R23
    direct = {}
    for l in open(path):
        f = l.split()
        if f[0] == "gfx950" and f[6:12] == ["3", "3", "1", "1", "1", "1"] and f[12] == "1":
            direct[(int(f[1]), int(f[2]), int(f[3]), int(f[4]), int(f[5]), 1, 1)] = float(f[-1])
    for s in p.describe()["steps"]:
        if s["kind"] == "conv" and (s["conv"]["R"], s["conv"]["stride"][0]) == (3, 1):
            c = s["conv"]
            key = (c["N"], c["C"], c["H"], c["W"], c["K"], 1, 1)
            assert (c["algo"] == "winograd") == (wino[key] < direct[key]), (key, wino[key], direct[key])
    y = host(p.run(dev(g.x)))
    p.destroy()
    assert_close_network(y, oracle_output(g), "resnet50 b1 tuned winograd", graph=g)
    gpu.tune_db_clear()


def _gap_graph():
    b = wl._Builder("gap3x3", (1, 32, 9, 9), np.random.Generator(np.random.PCG64(5)))
    c1 = b.conv(0, 48, 3, pad=1, name="c1")
    c2 = b.conv(c1, 64, 3, pad=1, name="c2")
    gp = b.gap(c2)
    fl = b.flatten(gp, 64)
    b.output(b.dense(fl, 10, name="fc"))
    return b.finish(lambda rng: wl._f32(rng.uniform(-1.0, 1.0, size=(1, 32, 9, 9))))


def test_planner_keeps_a_pool_folded_conv_direct():
    """A 3x3 stride-1 conv whose output the global pool reads, folded into it
    (NEO_PLAN_FUSE_GAP), writes channel sums, which only the direct kernel
    does: it stays direct under NEO_PLAN_WINOGRAD."""
    g = _gap_graph()
    d = _host_desc(g, neo.PLAN_WINOGRAD | neo.PLAN_FUSE_GAP)
    convs = [s["conv"] for s in d["steps"] if s["kind"] == "conv"]
    assert [c.get("gap_sums", False) for c in convs] == [False, True]
    assert [c["algo"] for c in convs] == ["winograd", "direct"]


@pytest.mark.gpu
def test_plan_winograd_with_pool_fold(gpu):
    """The plan above on the GPU, untuned and tuned, against the oracle."""
    from gpu_util import assert_close, dev, host
    g = _gap_graph()
    ref = orc.run_graph(g)
    for fl in (gpu.PLAN_WINOGRAD | gpu.PLAN_FUSE_GAP, gpu.PLAN_WINOGRAD | gpu.PLAN_FUSE_GAP | gpu.PLAN_TUNE):
        p = gpu.Plan(g, flags=fl)
        y = host(p.run(dev(g.x)))
        p.destroy()
        assert_close(y.reshape(ref.shape), ref, f"gap-folded plan, flags {fl}")
