"""Integer inference of whole networks through the plan (NEO_PLAN_INT8,
neo_plan_calibrate_int8) against the oracle's integer network executor
(oracle.quant.run_graph_int8).

Every int8 layer's arithmetic is fixed exactly (quantization by float32
division, or by the float32 reciprocal where the producing conv writes the
input's int8 copy itself; exact integer sums; the float32 epilogue one rounding per
operation; max pools exact; average pools the exact mean rounded once), so
the calibrated input scales of all convs must equal the oracle's bit for
bit: each is the maximum of a tensor that both sides computed identically.
Only the global average pool and the dense layers that follow the last conv
sum floats in different orders, so the logits are held to the network
tolerance."""
import ctypes

import numpy as np
import pytest

from oracle import quant as oq
from paper_1809_02697_amd import neo
from paper_1809_02697_amd import workloads as wl


def test_host_plan_and_flags():
    g = wl.resnet50(1)
    p = neo.Plan(g, flags=neo.PLAN_HOST_ONLY | neo.PLAN_INT8)
    d = p.describe()
    convs = [s for s in d["steps"] if s["kind"] == "conv"]
    assert len(convs) == 53 and len(d["steps"]) == 57
    assert all(s["conv"]["algo"] == "int8" and not s["conv"]["int8"]["calibrated"] for s in convs)
    assert not any(s["kind"].startswith("conv_") for s in d["steps"])     # no fused steps
    # one int8 copy per (value, padding): 49 for 53 convs (each stage's input
    # is shared by its reduce and projection convs); every conv output that
    # convs read is written as a copy by its producer (47; 12 of them, the
    # outputs of identity-shortcut blocks, also in float32 for the residual),
    # so only the network input and the max pool's output are quantized by a
    # pass of their own
    q = [s["conv"]["int8"] for s in convs]
    assert len({x["input_copy"] for x in q}) == 49
    assert sum(x["quantizes_input"] for x in q) == 2
    assert sum(x["writes_copy"] >= 0 for x in q) == 47
    assert sum(x["writes_copy"] >= 0 and x["writes_f32"] for x in q) == 12
    L = neo.lib()
    FAKE = ctypes.c_void_p(1 << 20)
    assert L.neo_plan_calibrate_int8(p.handle, FAKE, FAKE, None) == -7   # host-only: NEO_ERR_STATE
    p.destroy()
    for extra in (neo.PLAN_GROUP, neo.PLAN_FUSE_PAIRS, neo.PLAN_WINOGRAD, neo.PLAN_NAIVE,
                  neo.PLAN_GLOBAL_SEARCH):
        with pytest.raises(RuntimeError, match="NEO_PLAN_INT8"):
            neo.Plan(g, flags=neo.PLAN_HOST_ONLY | neo.PLAN_INT8 | extra)
    with pytest.raises(RuntimeError, match="NEO_PLAN_INT8"):
        neo.Plan(g, flags=neo.PLAN_HOST_ONLY | neo.PLAN_INT8, block=32)
    # a float32 plan refuses calibration
    p = neo.Plan(wl.tiny_graph(), flags=neo.PLAN_HOST_ONLY)
    assert L.neo_plan_calibrate_int8(p.handle, FAKE, FAKE, None) == -7
    p.destroy()


# ---- GPU -------------------------------------------------------------------------------------
@pytest.fixture(scope="module")
def gpu():
    from gpu_util import torch_cuda
    torch_cuda()
    neo.lib()
    return neo


def plan_scales(d):
    """{conv node id: its calibrated input scale} from a plan description."""
    return {s["node"]: np.float32(s["conv"]["int8"]["x_scale"]) for s in d["steps"]
            if s["kind"] == "conv"}


def run_int8_plan(gpu, g, flags=0):
    """Build, calibrate on the network's own input, run again: (calibration
    output, run output, scales by conv node, plan)."""
    from gpu_util import dev, host
    p = gpu.Plan(g, flags=gpu.PLAN_INT8 | flags)
    x = dev(g.x)
    y_cal = host(p.calibrate_int8(x))
    d = p.describe()
    assert all(s["conv"]["int8"]["calibrated"] for s in d["steps"] if s["kind"] == "conv")
    y = host(p.run(x))
    return y_cal, y, plan_scales(d), p


@pytest.mark.gpu
@pytest.mark.parametrize("name,N", [("vgg_tiny", 2), ("resnet50", 1), ("resnet50", 2), ("vgg16", 1),
                                    ("inception_v3", 1)])
def test_int8_network_against_the_oracle(gpu, name, N):
    """All conv input scales bit-exact against the oracle's integer network;
    the logits within the network tolerance of the oracle's (top-1 equal);
    the calibration run and a later run bit-identical; a replayed graph too."""
    from gpu_util import assert_close_network, dev, host
    g = wl.vgg_like_tiny(N=N) if name == "vgg_tiny" else wl.MODELS[name](N)
    print(f"\n[int8 plan] {name} N={N}", flush=True)
    y_cal, y, scales, p = run_int8_plan(gpu, g)
    p.destroy()
    ref, ref_scales = oq.run_graph_int8(g)
    conv_ids = g.node_ids("conv")
    assert sorted(scales) == conv_ids
    got = np.array([scales[i] for i in conv_ids], np.float32)
    mism = np.nonzero(got != ref_scales)[0]
    assert len(mism) == 0, f"{len(mism)} of {len(got)} scales differ, first at conv {mism[:3]}"
    np.testing.assert_array_equal(y, y_cal)
    ref = ref.reshape(y.shape)
    assert_close_network(y, ref, f"{name} int8 b{N}")
    assert (np.argmax(y, 1) == np.argmax(ref, 1)).all()
    # graph replay: the same launches, the same bits
    pg = gpu.Plan(g, flags=gpu.PLAN_INT8 | gpu.PLAN_HIPGRAPH)
    x = dev(g.x)
    pg.calibrate_int8(x)
    y1 = host(pg.run(x))
    y2 = host(pg.run(x))
    pg.destroy()
    np.testing.assert_array_equal(y1, y)
    np.testing.assert_array_equal(y2, y)
    # how far integer inference moves the float32 network (reported, not a gate)
    f32 = __import__("oracle").run_graph(g).reshape(y.shape)
    e = np.linalg.norm((y - f32).ravel()) / np.linalg.norm(f32.ravel())
    print(f"[int8 plan] {name} N={N}: rel L2 against the float32 network {e:.3e}, top-1 agreement "
          f"{(np.argmax(y, 1) == np.argmax(f32, 1)).mean():.2f}")


@pytest.mark.gpu
def test_tuned_int8_plan_gives_the_same_bits(gpu):
    """The local search picks other tiles and wave splits; the integer sums
    are exact and the epilogue the same, so the output is bit-identical."""
    from gpu_util import dev, host
    g = wl.resnet50(1)
    _, y, _, p = run_int8_plan(gpu, g)
    p.destroy()
    pt = gpu.Plan(g, flags=gpu.PLAN_INT8 | gpu.PLAN_TUNE | gpu.PLAN_HIPGRAPH)
    d = pt.describe()
    assert all(s["conv"]["tuned"] for s in d["steps"] if s["kind"] == "conv")
    tiles = {tuple(s["conv"]["int8"]["tile"]) + (s["conv"]["int8"]["waves"],)
             for s in d["steps"] if s["kind"] == "conv"}
    x = dev(g.x)
    pt.calibrate_int8(x)
    yt = host(pt.run(x))
    pt.destroy()
    print(f"\n[int8 plan] tuned: {len(tiles)} distinct configurations")
    np.testing.assert_array_equal(yt, y)


@pytest.mark.gpu
def test_int8_plan_runs_only_after_calibration(gpu):
    from gpu_util import dev
    g = wl.vgg_like_tiny()
    p = gpu.Plan(g, flags=gpu.PLAN_INT8)
    with pytest.raises(RuntimeError, match="calibrate"):
        p.run(dev(g.x))
    p.destroy()


@pytest.mark.gpu
def test_recalibration_on_another_input(gpu):
    """Calibrating again on a scaled input sets the scales from that input
    (the oracle on the same input agrees), and the captured graph is rebuilt."""
    from gpu_util import dev, host
    g = wl.vgg_like_tiny()
    p = gpu.Plan(g, flags=gpu.PLAN_INT8 | gpu.PLAN_HIPGRAPH)
    p.calibrate_int8(dev(g.x))
    y_a = host(p.run(dev(g.x)))
    x2 = (g.x * np.float32(3.0)).astype(np.float32)
    p.calibrate_int8(dev(x2))
    s2 = plan_scales(p.describe())
    y_b = host(p.run(dev(x2)))
    p.destroy()
    ref_b, ref_s2 = oq.run_graph_int8(g, x2)
    np.testing.assert_array_equal(np.array([s2[i] for i in g.node_ids("conv")], np.float32), ref_s2)
    assert not np.array_equal(y_a, y_b)
    from gpu_util import assert_close_network
    assert_close_network(y_b, ref_b.reshape(y_b.shape), "recalibrated")


def test_results_file_int8_lines(tmp_path):
    """An "int8" line of the results file loads (and is saved back) when it
    names a configuration the kernel takes for its shape; others are refused."""
    neo.tune_db_clear()
    arch = "gfx950"
    good = tmp_path / "good.txt"
    good.write_text(f"int8 {arch} 1 64 56 56 64 3 3 1 1 1 1 0 4 2 1 12.5\n"
                    f"int8 {arch} 32 256 14 14 256 3 3 1 1 1 1 3 2 4 2 11.25\n")
    assert neo.tune_db_load(str(good)) == 2 and neo.tune_db_size() == 2
    out = tmp_path / "saved.txt"
    neo.tune_db_save(str(out))
    assert sorted(l for l in out.read_text().splitlines() if l.startswith("int8 ")) == \
        sorted(good.read_text().splitlines())
    for bad in (f"int8 {arch} 1 64 56 56 64 3 3 1 1 1 1 0 3 2 1 12.5",     # no 3-block tile
                f"int8 {arch} 1 64 56 56 48 3 3 1 1 1 1 0 4 2 1 12.5",     # 3 blocks: fk 4 does not divide
                f"int8 {arch} 1 64 56 56 64 3 3 1 1 1 1 1 4 2 1 12.5",     # output mode 1
                f"int8 {arch} 1 64 56 56 64 3 3 1 1 1 1 0 4 2 8 12.5"):    # 8 waves
        f = tmp_path / "bad.txt"
        f.write_text(bad + "\n")
        with pytest.raises(RuntimeError, match="malformed"):
            neo.tune_db_load(str(f))
    neo.tune_db_clear()
