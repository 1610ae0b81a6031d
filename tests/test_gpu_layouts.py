"""GPU parity of the per-tensor layouts (NCHW[x]c with x = 4..64) that the
global layout search (Section 3.3.2) chooses between: the convolution with
its input in NCHW[ic_bn]c and output in NCHW[oc_bn]c, the layout-tolerant
pools, the transforms between any two blocks, and whole plans with mixed
schemes -- each against the oracle, and bit-identical to the 16-channel
result where the arithmetic is the same."""
import numpy as np
import pytest

import oracle as orc
from oracle import search as S
from paper_1809_02697_amd import workloads as wl

from gpu_util import assert_close, assert_close_network, dev, host, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def neo():
    torch_cuda()
    from paper_1809_02697_amd import neo as n
    n.lib()
    return n


def _prep(neo, c):
    """Fold (host), pack (device), padded bias for one LayerCase."""
    if c.bn is not None:
        w, b = neo.fold_bn(c.w, c.bias, c.bn["gamma"], c.bn["beta"], c.bn["mean"], c.bn["var"],
                           c.bn["eps"])
    else:
        w, b = c.w, c.bias
    bp = None
    if b is not None:
        bpad = np.zeros(-(-c.K // 16) * 16, np.float32)
        bpad[:c.K] = b
        bp = dev(bpad)
    return neo.pack_filter(dev(w)), bp


def run_xy(neo, c, xb, yb):
    """The case with its input in NCHW[xb]c and its output (and residual) in
    NCHW[yb]c; returns the NCHW[yb]c device output."""
    wp, bp = _prep(neo, c)
    x = neo.layout_transform(dev(c.x), 0, xb, *c.x.shape)
    res = None
    if c.epilogue == "res":
        res = neo.layout_transform(dev(c.residual), 0, yb, *c.residual.shape)
    act = "relu" if c.epilogue in ("relu", "res", "bias_relu") else "none"
    return neo.conv2d_nchwxc(x, c.C, wp, c.K, c.R, c.S, bias=bp, stride=c.stride, pad=c.pad,
                             act=act, residual=res, y_block=yb)


CASES = [
    # C, K, R, stride, pad, H, N, epilogue, (xb, yb) pairs
    (64, 64, 3, 1, 1, 14, 1, "relu", [(16, 32), (32, 16), (32, 32), (64, 64), (16, 64), (64, 32)]),
    (48, 40, 3, 2, 1, 13, 2, "res", [(32, 32), (64, 64), (32, 16), (16, 64)]),   # ragged C, K
    (256, 128, 1, 2, 0, 15, 1, "none", [(32, 64), (64, 16)]),                    # strided 1x1
    (96, 48, 1, 1, 0, 9, 3, "res", [(32, 32), (64, 16), (16, 32)]),
    (3, 64, 7, 2, 3, 40, 1, "relu", [(4, 16), (4, 32), (8, 64), (16, 32), (64, 16), (1, 16)]),  # stem
    (3, 20, 3, 1, 1, 12, 2, "relu", [(4, 32), (4, 64), (1, 32)]),                # stem, ragged K
    # NCHW input (block 1) with 1 and 4 channels; a residual
    (1, 16, 3, 1, 1, 10, 2, "relu", [(1, 16), (4, 16)]),
    (4, 24, 5, 2, 2, 11, 1, "res", [(1, 16), (1, 32), (8, 16)]),
]


@pytest.mark.parametrize("case", CASES, ids=[f"C{c[0]}K{c[1]}_{c[2]}x{c[2]}s{c[3]}" for c in CASES])
def test_conv_blocks_match_oracle_and_block16(neo, case):
    C, K, R, st, pd, H, N, epi, pairs = case
    OH = orc.out_size(H, R, st, pd)
    c = wl.conv_case(C, K, R, R, st, pd, H, H, N=N, epilogue=epi, out_hw=(OH, OH))
    ref = orc.layer_forward(c)
    base = orc.from_blocked(host(run_xy(neo, c, 16, 16)), K)
    assert_close(base, ref, "16/16")
    for xb, yb in pairs:
        yblk = host(run_xy(neo, c, xb, yb))
        assert yblk.shape[-1] == yb
        y = orc.from_blocked(yblk, K)
        np.testing.assert_array_equal(y, base, err_msg=f"{xb}/{yb}")
        # padding lanes of the last output block are +0.0
        lanes = yblk.transpose(0, 1, 4, 2, 3).reshape(N, -1, OH, OH)[:, K:]
        assert (lanes == 0).all() and not np.signbit(lanes).any(), f"{xb}/{yb} padding"


@pytest.mark.parametrize("cfg", ["1,1,3,2", "2,2,2,1", "4,1,4,4", "1,2,1,8"])
def test_conv_blocks_split_and_tiles(neo, cfg, monkeypatch):
    """Forced launch configurations (split reductions write the zero padding
    of the last output block in the reduce pass)."""
    monkeypatch.setenv("NEO_CONV_CONFIG", cfg)
    c = wl.conv_case(80, 40, 3, 3, 1, 1, 9, 9, N=2, epilogue="res", out_hw=(9, 9))
    ref = orc.layer_forward(c)
    for xb, yb in [(16, 64), (32, 32), (64, 16)]:
        y = host(run_xy(neo, c, xb, yb))
        assert_close(orc.from_blocked(y, 40), ref, f"{cfg} {xb}/{yb}")
        lanes = y.transpose(0, 1, 4, 2, 3).reshape(2, -1, 9, 9)[:, 40:]
        assert (lanes == 0).all()


@pytest.mark.parametrize("cfg", ["1,1,3,2", "2,2,2,1", "4,1,4,4", "1,4,1,1"])
def test_conv_nchw_input_split_and_tiles(neo, cfg, monkeypatch):
    """The stem reading NCHW directly (block 1) under forced launch
    configurations, split reductions included, against the oracle and
    bit-identical to its NCHW4c input."""
    monkeypatch.setenv("NEO_CONV_CONFIG", cfg)
    c = wl.conv_case(3, 40, 7, 7, 2, 3, 23, 19, N=2, epilogue="relu", out_hw=(12, 10))
    ref = orc.layer_forward(c)
    y4 = orc.from_blocked(host(run_xy(neo, c, 4, 16)), 40)
    y1 = orc.from_blocked(host(run_xy(neo, c, 1, 16)), 40)
    assert_close(y1, ref, f"{cfg} NCHW input")
    np.testing.assert_array_equal(y1, y4)


def test_conv_block_slice_offsets(neo):
    """y_blk_offset / total in blocks of y_block: only the slice is written."""
    torch = torch_cuda()
    c = wl.conv_case(32, 64, 3, 3, 1, 1, 8, 8, epilogue="relu", with_bn=False)
    ref = orc.layer_forward(c)
    wp, bp = _prep(neo, c)
    x = neo.layout_transform(dev(c.x), 0, 32, *c.x.shape)
    out = torch.full((1, 4, 8, 8, 32), 7.0, device="cuda")
    neo.conv2d_nchwxc(x, 32, wp, 64, 3, 3, bias=bp, stride=1, pad=1, act="relu", out=out,
                      y_block=32, y_blk_offset=1, y_blk_total=4)
    o = host(out)
    assert (o[:, [0, 3]] == 7.0).all()
    assert_close(orc.from_blocked(o[:, 1:3], 64), ref, "slice")


def test_conv_block_errors(neo):
    c = wl.conv_case(32, 16, 3, 3, 1, 1, 8, 8, epilogue="relu", with_bn=False)
    wp, bp = _prep(neo, c)
    x8 = neo.layout_transform(dev(c.x), 0, 8, *c.x.shape)
    with pytest.raises(neo.NeoError) as e:
        neo.conv2d_nchwxc(x8, 32, wp, 16, 3, 3, bias=bp, pad=1)   # 8 only on the stem path
    assert e.value.code == -4
    x16 = neo.layout_transform(dev(c.x), 0, 16, *c.x.shape)
    with pytest.raises(neo.NeoError) as e:
        neo.conv2d_nchwxc(x16, 32, wp, 16, 3, 3, bias=bp, pad=1, y_block=8)
    assert e.value.code == -4


# ---- pools and transforms at every block ------------------------------------------------------
@pytest.mark.parametrize("blk", [4, 8, 32, 64])
def test_pools_every_block(neo, blk):
    for kind, R, st, pd, C, H, N in [("max", 3, 2, 1, 40, 13, 2), ("avg", 3, 1, 1, 72, 9, 1),
                                     ("max", 2, 2, 0, 64, 10, 1), ("avg", 5, 2, 2, 20, 11, 1)]:
        x = np.random.default_rng(C * H + blk).uniform(-1, 1, (N, C, H, H)).astype(np.float32)
        xb = neo.layout_transform(dev(x), 0, blk, N, C, H, H)
        x16 = neo.to_blocked(dev(x))
        if kind == "max":
            y, y16 = neo.maxpool2d_nchwxc(xb, C, R, R, st, pd), neo.maxpool2d_blocked(x16, C, R, R, st, pd)
            ref = orc.maxpool2d(x, R, R, st, pd)
        else:
            y, y16 = neo.avgpool2d_nchwxc(xb, C, R, R, st, pd), neo.avgpool2d_blocked(x16, C, R, R, st, pd)
            ref = orc.avgpool2d(x, R, R, st, pd)
        got = orc.from_blocked(host(y), C)
        np.testing.assert_array_equal(got, orc.from_blocked(host(y16), C))
        assert_close(got, ref, f"{kind} {blk}")


@pytest.mark.parametrize("blk", [4, 8, 16, 32, 64])
@pytest.mark.parametrize("N,C,H,W", [(1, 2048, 7, 7), (2, 40, 5, 3), (1, 20, 8, 8), (3, 192, 2, 3)])
def test_global_avgpool_every_block(neo, blk, N, C, H, W):
    x = np.random.default_rng(C + blk).uniform(-1, 1, (N, C, H, W)).astype(np.float32)
    y = host(neo.global_avgpool_nchwxc(neo.layout_transform(dev(x), 0, blk, N, C, H, W), C))
    y16 = host(neo.global_avgpool_blocked(neo.to_blocked(dev(x)), C))
    got = orc.from_blocked(y, C)
    np.testing.assert_array_equal(got, orc.from_blocked(y16, C))   # same summation order
    np.testing.assert_array_equal(got, orc.global_avgpool(x))      # the exact mean, rounded once


BLOCK_PAIRS = [(a, b) for a in (0, 4, 8, 16, 32, 64) for b in (0, 4, 8, 16, 32, 64) if a != b]


@pytest.mark.parametrize("sb,db", BLOCK_PAIRS)
def test_transform_every_pair_bit_exact(neo, sb, db):
    for N, C, H, W in [(2, 37, 5, 6), (1, 64, 3, 3), (1, 3, 7, 4)]:
        x = np.random.default_rng(sb * 97 + db + C).uniform(-1, 1, (N, C, H, W)).astype(np.float32)
        src = x if sb == 0 else orc.to_blocked(x, sb)
        out = host(neo.layout_transform(dev(src), sb, db, N, C, H, W))
        np.testing.assert_array_equal(out, x if db == 0 else orc.to_blocked(x, db))
        if db:
            lanes = out.transpose(0, 1, 4, 2, 3).reshape(N, -1, H, W)[:, C:]
            assert not np.signbit(lanes).any()


# ---- plans with mixed schemes ----------------------------------------------------------------
def _schemes(g, rng):
    shapes = S.infer_shapes(g)
    out = {}
    for v in S.conv_nodes(g):
        C, K = shapes[g.nodes[v].inputs[0]][1], g.nodes[v].K
        ics = [1, 4, 8, 16, 32] if C <= 4 else [b for b in (16, 32, 64) if C % b == 0 or b == 16]
        ocs = [b for b in (16, 32, 64) if K % b == 0 or b == 16]
        out[v] = (int(rng.choice(ics)), int(rng.choice(ocs)))
    return out


@pytest.mark.parametrize("builder,seed", [(wl.tiny_graph, 0), (wl.tiny_graph, 1),
                                          (wl.vgg_like_tiny, 2), (lambda: wl.resnet50(1), 3),
                                          (lambda: wl.inception_v3(1), 4)])
def test_mixed_scheme_plan_is_bit_identical(neo, builder, seed):
    """Untuned plans choose launch configurations by a cost model that ignores
    the blocks, so any scheme assignment computes exactly the same numbers as
    the one-block plan; both match the oracle."""
    neo.tune_db_clear()          # configurations from the cost model only
    g = builder()
    x = dev(g.x)
    p16 = neo.Plan(g)
    y16 = host(p16.run(x))
    p16.destroy()
    sch = _schemes(g, np.random.default_rng(seed))
    p = neo.Plan(g, schemes=sch)
    d = p.describe()
    y = host(p.run(x))
    p.destroy()
    np.testing.assert_array_equal(y, y16)
    assert d["n_transforms"] >= 1
    ref = orc.run_graph(g)
    assert_close_network(y.reshape(ref.shape), ref, g.name, graph=g)


@pytest.mark.parametrize("block", [32, 64])
def test_fixed_block_plan(neo, block):
    neo.tune_db_clear()
    g = wl.resnet50(1)
    x = dev(g.x)
    p16 = neo.Plan(g)
    y16 = host(p16.run(x))
    p16.destroy()
    p = neo.Plan(g, block=block, flags=neo.PLAN_HIPGRAPH)
    y = host(p.run(x))
    y2 = host(p.run(x))
    p.destroy()
    np.testing.assert_array_equal(y, y16)
    np.testing.assert_array_equal(y2, y16)


@pytest.mark.parametrize("builder", [wl.tiny_graph, lambda: wl.resnet50(1)])
def test_global_search_plan(neo, builder):
    """NEO_PLAN_GLOBAL_SEARCH: measured schemes and transforms, the program's
    choice, a plan that matches the oracle, and a predicted cost no worse than
    the one-block plan's under the same measurements."""
    g = builder()
    p = neo.Plan(g, flags=neo.PLAN_GLOBAL_SEARCH | neo.PLAN_HIPGRAPH)
    d = p.describe()
    y = host(p.run(dev(g.x)))
    p.destroy()
    s = d["search"]
    assert s["schemes_measured"] >= len(S.conv_nodes(g))
    assert 0 < s["cost_us"] <= s["fixed_block_cost_us"] + 1e-9
    convs = [st for st in d["steps"] if st["kind"] == "conv"]
    assert all(c["conv"]["tuned"] for c in convs)
    print(f"\n{g.name}: search {s}, schemes "
          f"{sorted(set((c['conv']['ic_bn'], c['conv']['oc_bn']) for c in convs))}, "
          f"transforms {d['n_transforms']}")
    ref = orc.run_graph(g)
    assert_close_network(y.reshape(ref.shape), ref, g.name, graph=g)
