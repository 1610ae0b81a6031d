"""Integer inference of whole networks through the plan (NEO_PLAN_INT8,
neo_plan_calibrate_int8) against the oracle's integer network executor
(oracle.quant.run_graph_int8).

Every int8 layer's arithmetic is fixed exactly (quantization by float32
division, or by the float32 reciprocal where the producing conv or dense
layer writes the input's int8 copy itself; exact integer sums; the float32
epilogue one rounding per operation; max pools exact; average pools and the
global average pool the exact mean rounded once), so the calibrated input
scales of all convs and dense layers must equal the oracle's bit for bit --
each is the maximum of a tensor that both sides computed identically -- and
so must the logits."""
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
    # (the stem reads the network input directly: no NCHW -> NCHW16c step)
    assert len(convs) == 53 and len(d["steps"]) == 56
    assert all(s["conv"]["algo"] == "int8" and not s["conv"]["int8"]["calibrated"] for s in convs)
    assert not any(s["kind"].startswith("conv_") for s in d["steps"])     # no fused steps
    # one int8 copy per value: 49 for 53 convs (each stage's input is shared
    # by its reduce and projection convs); every conv output that convs read
    # is written as a copy by its producer (47; 12 of them, the outputs of
    # identity-shortcut blocks, also in float32 for the residual), and the
    # max pool writes its output's copy (int8 only), so only the network
    # input is quantized by a pass of its own
    q = [s["conv"]["int8"] for s in convs]
    assert len({x["input_copy"] for x in q}) == 49
    assert sum(x["quantizes_input"] for x in q) == 1 and q[0]["quantizes_input"]
    # the 7x7 stem over 3 channels runs as a 1x1 conv over its input's im2col
    # rows (147 channels: 3 reduction steps of 64 instead of 49), quantized
    # straight from the NCHW network input
    assert [x.get("im2col", False) for x in q] == ["nchw"] + [False] * 52
    assert sum(x["writes_copy"] >= 0 for x in q) == 47
    assert sum(x["writes_copy"] >= 0 and x["writes_f32"] for x in q) == 12
    pool = [s for s in d["steps"] if s["kind"] == "maxpool"][0]
    assert pool["int8"]["writes_copy"] >= 0 and not pool["int8"]["writes_f32"]
    # (the stem's 3.2 MB output is pooled in float32: below 16 MiB)
    assert "reads_int8" not in pool["int8"]
    L = neo.lib()
    FAKE = ctypes.c_void_p(1 << 20)
    assert L.neo_plan_calibrate_int8(p.handle, FAKE, FAKE, None) == -7   # host-only: NEO_ERR_STATE
    p.destroy()
    for extra in (neo.PLAN_FUSE_PAIRS, neo.PLAN_WINOGRAD, neo.PLAN_NAIVE, neo.PLAN_GLOBAL_SEARCH):
        with pytest.raises(RuntimeError, match="NEO_PLAN_INT8"):
            neo.Plan(g, flags=neo.PLAN_HOST_ONLY | neo.PLAN_INT8 | extra)
    with pytest.raises(RuntimeError, match="NEO_PLAN_INT8"):
        neo.Plan(g, flags=neo.PLAN_HOST_ONLY | neo.PLAN_INT8, block=32)
    # a float32 plan refuses calibration
    p = neo.Plan(wl.tiny_graph(), flags=neo.PLAN_HOST_ONLY)
    assert L.neo_plan_calibrate_int8(p.handle, FAKE, FAKE, None) == -7
    p.destroy()


def conv_steps(d):
    """(step index, conv description) of every conv, group members included."""
    out = []
    for i, s in enumerate(d["steps"]):
        if s["kind"] == "conv":
            out.append((i, s["conv"]))
        elif s["kind"] == "conv_group":
            out.extend((i, m["conv"]) for m in s["members"])
    return out


@pytest.mark.parametrize("name", ["resnet50", "inception_v3"])
def test_host_grouped_int8_plan(name):
    """NEO_PLAN_INT8 | NEO_PLAN_GROUP: independent integer convs share
    launches (pools ride along), every conv is still planned once, and each
    copy that no conv writes is quantized once, by its first reader in the
    grouped order (members of one launch count as one position: the launch
    runs its members' passes first)."""
    g = wl.MODELS[name](1)
    p0 = neo.Plan(g, flags=neo.PLAN_HOST_ONLY | neo.PLAN_INT8)
    d0 = p0.describe()
    p0.destroy()
    p = neo.Plan(g, flags=neo.PLAN_HOST_ONLY | neo.PLAN_INT8 | neo.PLAN_GROUP)
    d = p.describe()
    p.destroy()
    cs = conv_steps(d)
    assert sorted(c["int8"]["input_copy"] for _, c in cs) == sorted(s["conv"]["int8"]["input_copy"]
                                                                  for s in d0["steps"] if s["kind"] == "conv")
    groups = [s for s in d["steps"] if s["kind"] == "conv_group"]
    assert groups and all(s["algo"] == "int8" and 2 <= len(s["members"]) + ("pool" in s) for s in groups)
    for s in groups:
        assert all(m["conv"]["int8"]["tile"] == s["tile"] and m["conv"]["int8"]["waves"] == s["waves"]
                   for m in s["members"])
    # the same copies are written by the same convs and pools; passes only
    # where no conv or pool writes
    writers = {c["int8"]["writes_copy"] for _, c in cs if c["int8"]["writes_copy"] >= 0}
    for s in d["steps"]:
        for p_ in [s] + ([s["pool"]] if "pool" in s else []):
            if "int8" in p_ and "writes_copy" in p_["int8"] and "input_copy" not in p_["int8"]:
                writers.add(p_["int8"]["writes_copy"])
    first = {}
    for i, c in cs:
        first.setdefault(c["int8"]["input_copy"], i)
    for i, c in cs:
        q = c["int8"]["input_copy"]
        want = q not in writers and i == first[q]
        if c["int8"]["quantizes_input"]:
            assert want
    passes = [c["int8"]["input_copy"] for _, c in cs if c["int8"]["quantizes_input"]]
    assert len(passes) == len(set(passes)) == len({c["int8"]["input_copy"] for _, c in cs} - writers)
    n_launch = len(d["steps"]) + len(passes)
    n_launch0 = len(d0["steps"]) + sum(s["conv"]["int8"]["quantizes_input"] for s in d0["steps"]
                                       if s["kind"] == "conv")
    print(f"\n[int8 group] {name}: {n_launch0} -> {n_launch} launches, {len(groups)} groups")
    assert n_launch < n_launch0
    if name == "inception_v3":
        # one pass, the input's; the 4 values read by a 1x3 and a 3x1 conv
        # have one copy, halo (1, 1), written by their producer; the pools
        # write their own outputs' copies; the 10 concatenations convs read
        # are assembled by their parts (one through two nested ones)
        assert len(groups) == 27 and sum("pool" in s for s in groups) == 11 and len(passes) == 1
        slices = {}
        for s in d["steps"]:
            for w in ([s["conv"]["int8"]] if s["kind"] == "conv" else
                      [m["conv"]["int8"] for m in s.get("members", [])] +
                      ([s["pool"]["int8"]] if "int8" in s.get("pool", {}) else []) +
                      ([s["int8"]] if s["kind"] in ("maxpool", "avgpool") and "int8" in s else [])):
                if "writes_slice" in w:
                    slices.setdefault(w["writes_copy"], []).append(w["writes_slice"])
        assert len(slices) == 10
        for parts in slices.values():      # the parts tile the copy's blocks in order
            parts.sort()
            assert parts[0][0] == 0 and len({t for _, t in parts}) == 1
            assert all(a[0] < b[0] for a, b in zip(parts, parts[1:]))


# ---- GPU -------------------------------------------------------------------------------------
@pytest.fixture(scope="module")
def gpu():
    from gpu_util import torch_cuda
    torch_cuda()
    neo.lib()
    return neo


def plan_scales(d):
    """{conv or dense node id: its calibrated input scale} from a plan
    description (group members included)."""
    out = {}
    for s in d["steps"]:
        for m in [s] if s["kind"] == "conv" else s.get("members", []) if s["kind"] == "conv_group" else []:
            out[m["node"]] = np.float32(m["conv"]["int8"]["x_scale"])
        if s["kind"] == "dense" and "int8" in s["dense"]:
            out[s["node"]] = np.float32(s["dense"]["int8"]["x_scale"])
    return out


def int8_ids(g):
    """The node ids of a network's int8 layers (convs and dense layers), in node order."""
    return sorted(g.node_ids("conv") + g.node_ids("dense"))


def run_int8_plan(gpu, g, flags=0):
    """Build, calibrate on the network's own input, run again: (calibration
    output, run output, scales by conv node, plan)."""
    from gpu_util import dev, host
    p = gpu.Plan(g, flags=gpu.PLAN_INT8 | flags)
    x = dev(g.x)
    y_cal = host(p.calibrate_int8(x))
    d = p.describe()
    assert all(c["int8"]["calibrated"] for _, c in conv_steps(d))
    y = host(p.run(x))
    return y_cal, y, plan_scales(d), p


STEMS = [  # (C, R, S, stride, pad, H, W, N, im2col)
    (3, 7, 7, 2, 3, 37, 41, 2, True),     # ResNet's stem: 147 channels, ragged last block
    (3, 3, 3, 2, 0, 29, 29, 1, True),     # Inception's: 27 channels
    (17, 3, 3, 1, 1, 15, 13, 2, True),    # two input blocks: 153 channels
    (5, 5, 3, 1, (2, 1), 19, 9, 3, True),
    (40, 3, 3, 1, 1, 11, 11, 1, False),   # 360 channels: 6 steps against 9, not taken
    (3, 1, 1, 1, 0, 9, 9, 1, False),      # a 1x1 conv: nothing to gain
]


@pytest.mark.parametrize("C,R,S,stride,pad,H,W,N,i2c", STEMS)
def test_host_im2col_choice(C, R, S, stride, pad, H, W, N, i2c):
    """An integer conv runs over its input's im2col rows exactly when that at
    least halves its 64-channel reduction steps."""
    g = wl.stem_graph(N=N, C=C, H=H, W=W, K=32, R=R, S=S, stride=stride, pad=pad)
    p = neo.Plan(g, flags=neo.PLAN_HOST_ONLY | neo.PLAN_INT8)
    d = p.describe()
    (_, c), = conv_steps(d)
    p.destroy()
    assert c["int8"].get("im2col", False) == ("nchw" if i2c else False) and c["int8"]["quantizes_input"]
    # the network input's blocked copy only when the direct conv reads it
    # (besides the exit of the pool's output to NCHW)
    assert sum(s["kind"] == "transform" for s in d["steps"]) == (1 if i2c else 2)


@pytest.mark.gpu
@pytest.mark.parametrize("C,R,S,stride,pad,H,W,N,i2c", STEMS)
def test_im2col_stem_against_the_oracle(gpu, C, R, S, stride, pad, H, W, N, i2c):
    """The stem through the im2col rows (or the direct path) bit-exact
    against the oracle's integer conv: the same int8 inputs, the same integer
    sums, the same float32 epilogue."""
    from gpu_util import dev, host
    print(f"\n[int8 stem] C={C} R={R} S={S} stride={stride} pad={pad} {H}x{W} N={N}", flush=True)
    g = wl.stem_graph(N=N, C=C, H=H, W=W, K=32, R=R, S=S, stride=stride, pad=pad)
    y_cal, y, scales, p = run_int8_plan(gpu, g)
    (_, c), = conv_steps(p.describe())
    p.destroy()
    assert bool(c["int8"].get("im2col", False)) == i2c
    ref, ref_scales = oq.run_graph_int8(g)
    assert np.array_equal(np.array([scales[i] for i in int8_ids(g)], np.float32), ref_scales)
    np.testing.assert_array_equal(y, ref.reshape(y.shape))
    np.testing.assert_array_equal(y_cal, y)


def pooled_stem_graph(N=8, H=128, W=128):
    """A 3x3 stem (32 channels, 16.8 MB of float32 output at batch 8), a max
    pool and a 1x1 conv reading the pool: the stem's output is pooled in
    int8."""
    b = wl._Builder("pooled_stem", (N, 3, H, W), np.random.Generator(np.random.PCG64(12)))
    x = b.conv(0, 32, 3, pad=1, name="stem")
    x = b.pool("maxpool", x, 3, 2, 1, name="pool")
    b.output(b.conv(x, 16, 1, name="c1"))
    return b.finish(wl._normal_input((N, 3, H, W)))


def test_host_int8_pool_input():
    p = neo.Plan(pooled_stem_graph(), flags=neo.PLAN_HOST_ONLY | neo.PLAN_INT8)
    d = p.describe()
    p.destroy()
    (_, stem), _ = conv_steps(d)
    pool = [s for s in d["steps"] if s["kind"] == "maxpool"][0]
    assert pool["int8"]["reads_int8"] == stem["int8"]["writes_copy"] >= 0 and not stem["int8"]["writes_f32"]
    p = neo.Plan(pooled_stem_graph(N=7), flags=neo.PLAN_HOST_ONLY | neo.PLAN_INT8)   # 14.7 MB: float32
    assert "reads_int8" not in [s for s in p.describe()["steps"] if s["kind"] == "maxpool"][0]["int8"]
    p.destroy()


@pytest.mark.gpu
def test_int8_pool_input_against_the_oracle(gpu):
    """The stem requantized by division with the pool's scale, the max pool
    over bytes: the oracle's bits (its pool quantizes the float32 maxima)."""
    print("\n[int8 pool] pooled stem N=8", flush=True)
    g = pooled_stem_graph()
    y_cal, y, scales, p = run_int8_plan(gpu, g)
    p.destroy()
    ref, ref_scales = oq.run_graph_int8(g)
    assert np.array_equal(np.array([scales[i] for i in int8_ids(g)], np.float32), ref_scales)
    np.testing.assert_array_equal(y, ref.reshape(y.shape))
    np.testing.assert_array_equal(y_cal, y)


def two_stems_graph(N=2, H=21, W=19):
    """Two small-channel convs reading the network input (a 7x7 and a 3x3,
    both im2col), concatenated: the input's blocked copy has two readers, so
    both passes read it instead of the NCHW input."""
    b = wl._Builder("two_stems", (N, 3, H, W), np.random.Generator(np.random.PCG64(11)))
    a = b.conv(0, 32, 7, stride=2, pad=3, name="s7")
    c = b.conv(0, 16, 3, stride=2, pad=1, name="s3")
    b.output(b.concat([a, c], name="cat"))
    return b.finish(wl._normal_input((N, 3, H, W)))


def test_host_im2col_from_the_blocked_input():
    p = neo.Plan(two_stems_graph(), flags=neo.PLAN_HOST_ONLY | neo.PLAN_INT8)
    d = p.describe()
    p.destroy()
    assert [c["int8"].get("im2col") for _, c in conv_steps(d)] == ["blocked", "blocked"]


@pytest.mark.gpu
def test_im2col_from_the_blocked_input_against_the_oracle(gpu):
    print("\n[int8 stem] two stems from the blocked input", flush=True)
    g = two_stems_graph()
    y_cal, y, scales, p = run_int8_plan(gpu, g)
    p.destroy()
    ref, ref_scales = oq.run_graph_int8(g)
    assert np.array_equal(np.array([scales[i] for i in int8_ids(g)], np.float32), ref_scales)
    np.testing.assert_array_equal(y, ref.reshape(y.shape))
    np.testing.assert_array_equal(y_cal, y)


@pytest.mark.gpu
@pytest.mark.parametrize("name,N", [("tiny", 2), ("vgg_tiny", 2), ("vgg_tiny", 20), ("resnet50", 1),
                                    ("resnet50", 2), ("vgg16", 1), ("inception_v3", 1)])
def test_int8_network_against_the_oracle(gpu, name, N):
    """All conv and dense input scales and the logits bit-exact against the
    oracle's integer network; the calibration run and a later run
    bit-identical; a replayed graph too.  (The small net at batch 20 takes
    the dense kernel's four-rows-per-wave path, in a launch of 16 images
    and one of 4, with a ragged last row group of 10 outputs.)"""
    from gpu_util import dev, host
    g = (wl.vgg_like_tiny(N=N) if name == "vgg_tiny" else wl.tiny_graph() if name == "tiny" else
         wl.MODELS[name](N))
    print(f"\n[int8 plan] {name} N={N}", flush=True)
    y_cal, y, scales, p = run_int8_plan(gpu, g)
    p.destroy()
    ref, ref_scales = oq.run_graph_int8(g)
    ids = int8_ids(g)
    assert sorted(scales) == ids
    got = np.array([scales[i] for i in ids], np.float32)
    mism = np.nonzero(got != ref_scales)[0]
    assert len(mism) == 0, f"{len(mism)} of {len(got)} scales differ, first at conv {mism[:3]}"
    np.testing.assert_array_equal(y, y_cal)
    ref = ref.reshape(y.shape)
    np.testing.assert_array_equal(y, ref)
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
@pytest.mark.parametrize("name,N", [("vgg_tiny", 2), ("resnet50", 1), ("inception_v3", 1),
                                    ("inception_v3", 2)])
def test_grouped_int8_plan_gives_the_same_bits(gpu, name, N):
    """Convs in one launch compute what they compute alone (exact sums, the
    same epilogue, the pools' own arithmetic), so the grouped plan's scales
    equal the oracle's and its outputs the ungrouped plan's, bit for bit;
    graph replays too; the tuned grouped plan (groups kept, split or
    dissolved by the local search) as well."""
    from gpu_util import dev, host
    g = wl.vgg_like_tiny(N=N) if name == "vgg_tiny" else wl.MODELS[name](N)
    print(f"\n[int8 group] {name} N={N}", flush=True)
    _, y, scales, p = run_int8_plan(gpu, g)
    p.destroy()
    for flags in (gpu.PLAN_GROUP | gpu.PLAN_HIPGRAPH, gpu.PLAN_GROUP | gpu.PLAN_TUNE | gpu.PLAN_HIPGRAPH):
        y_cal, yg, sg, pg = run_int8_plan(gpu, g, flags)
        d = pg.describe()
        yr = host(pg.run(dev(g.x)))
        pg.destroy()
        n_groups = sum(s["kind"] == "conv_group" for s in d["steps"])
        print(f"[int8 group] flags {flags}: {n_groups} groups, {len(d['steps'])} steps", flush=True)
        assert sg == scales
        np.testing.assert_array_equal(yg, y)
        np.testing.assert_array_equal(y_cal, y)
        np.testing.assert_array_equal(yr, y)
    if name != "vgg_tiny":
        _, ref_scales = oq.run_graph_int8(g)
        np.testing.assert_array_equal(np.array([scales[i] for i in int8_ids(g)], np.float32), ref_scales)


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
    np.testing.assert_array_equal(np.array([s2[i] for i in int8_ids(g)], np.float32), ref_s2)
    assert not np.array_equal(y_a, y_b)
    np.testing.assert_array_equal(y_b, ref_b.reshape(y_b.shape))


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


def test_results_file_int8_group_lines(tmp_path):
    """An "i8group" line (n members with their output modes, m pools, the
    configuration) loads and saves back when the configuration suits every
    member; others are refused."""
    neo.tune_db_clear()
    arch = "gfx950"
    a = "1 64 35 35 64 1 1 1 1 0 0 0"      # 1x1, float32 output
    b = "1 64 35 35 48 1 1 1 1 0 0 2"      # 1x1 to 48 channels, int8 copy (3 blocks: fk 1)
    pool = "0 1 64 35 35 3 3 1 1 1 1 16 2" # 3x3 average pool, block 16, int8 output
    good = tmp_path / "good.txt"
    good.write_text(f"i8group {arch} 2 1 {a} {b} {pool} 1 2 1 7.5\n"
                    f"i8group {arch} 2 0 {a} {b} 1 1 1 6.25\n")
    assert neo.tune_db_load(str(good)) == 2 and neo.tune_db_size() == 2
    out = tmp_path / "saved.txt"
    neo.tune_db_save(str(out))
    assert sorted(l for l in out.read_text().splitlines() if l.startswith("i8group ")) == \
        sorted(good.read_text().splitlines())
    for bad in (f"i8group {arch} 2 1 {a} {b} {pool} 2 2 1 7.5",             # fk 2: 48 channels
                f"i8group {arch} 2 1 {a} {b} 0 1 64 35 35 3 3 1 1 1 1 8 2 1 1 1 7.5",  # block 8
                f"i8group {arch} 2 1 {a} {b} 0 1 64 35 35 3 3 1 1 1 1 16 1 1 1 1 7.5",  # pool mode 1
                f"i8group {arch} 2 2 {a} {b} {pool} {pool} 1 1 1 7.5",     # two pools
                f"i8group {arch} 5 0 {a} {a} {a} {a} {a} 1 1 1 7.5",       # five members
                f"i8group {arch} 1 0 1 64 35 35 64 1 1 1 1 0 0 1 1 1 1 7.5",  # output mode 1
                f"i8group {arch} 2 0 {a} {b} 1 1 2"):                       # no time
        f = tmp_path / "bad.txt"
        f.write_text(bad + "\n")
        with pytest.raises(RuntimeError, match="malformed"):
            neo.tune_db_load(str(f))
    neo.tune_db_clear()
