"""GPU parity of whole networks through neo_run_graph (the layout plan of
Section 3.2) against the oracle's reference graph executor."""
import numpy as np
import pytest

import oracle as orc
from paper_1809_02697_amd import workloads as wl

import torch_ref
from gpu_util import (assert_close, assert_close_conditioned, assert_close_network,
                      assert_strict_ceiling, dev, host, oracle_output, strict_violations,
                      torch_cuda)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def neo():
    torch_cuda()
    from paper_1809_02697_amd import neo as n
    n.lib()
    return n


def run_plan(neo, g, flags=0, x=None):
    p = neo.Plan(g, flags=flags)
    y = host(p.run(dev(g.x if x is None else x)))
    p.destroy()
    return y


@pytest.mark.parametrize("builder", [wl.tiny_graph, wl.vgg_like_tiny])
def test_small_graphs(neo, builder):
    g = builder()
    ref = orc.run_graph(g)
    y = run_plan(neo, g)
    assert_close(y.reshape(ref.shape), ref, g.name)


@pytest.mark.parametrize("builder", [wl.tiny_graph, wl.vgg_like_tiny])
def test_naive_plan_bit_identical(neo, builder):
    """Eliminating the transforms does not change a single bit (the transforms
    are exact permutations and the kernels are the same)."""
    g = builder()
    np.testing.assert_array_equal(run_plan(neo, g), run_plan(neo, g, neo.PLAN_NAIVE))


def test_plan_reusable_and_output_shape(neo):
    g = wl.tiny_graph()
    p = neo.Plan(g)
    assert p.output_shape == (2, 10, 1, 1)
    a = host(p.run(dev(g.x)))
    b = host(p.run(dev(g.x)))
    np.testing.assert_array_equal(a, b)
    p.destroy()


def _teacher_forced_convs(neo, g):
    """Every conv node of g on the GPU, fed the oracle's own input (and
    residual), with the plan's folded and packed parameters.  The magnitude of
    the terms of each output (for the conditioned bound) is the oracle's
    convolution of |x| with |w'| plus |b'| and |residual|.  The same layer in
    an independent float32 CPU pipeline, on the same operands, counts how many
    elements a correct float32 implementation misses the plain clause at."""
    vals = orc.run_graph(g, keep=True)
    p = neo.Plan(g)
    worst, strict, strict_f32 = 0.0, 0, 0
    for i, n in enumerate(g.nodes):
        if n.op != "conv":
            continue
        x = vals[n.inputs[0]]
        C = x.shape[1]
        wp, b = p.conv_params(i, n.K, C, n.R, n.S)
        res = vals[n.residual] if n.residual >= 0 else None
        yb = neo.conv2d_blocked(neo.to_blocked(dev(x)), C, dev(wp), n.K, n.R, n.S, bias=dev(b),
                                stride=n.stride, pad=n.pad, act=n.act,
                                residual=neo.to_blocked(dev(res)) if res is not None else None)
        y = orc.from_blocked(host(yb), n.K)
        w_abs = np.abs(_unpack(wp, n.K, C, n.R, n.S))
        cond = orc.conv2d(np.abs(x), w_abs, n.stride, n.pad).astype(np.float64)
        cond += np.abs(b[:n.K]).reshape(1, -1, 1, 1)
        if res is not None:
            cond += np.abs(res)
        e, sv = assert_close_conditioned(y, vals[i], cond, C * n.R * n.S, n.name)
        w_f, b_f = torch_ref.fold(n)
        y_f = torch_ref.conv_layer(x, w_f, b_f, n.stride, n.pad, n.act, res)
        worst, strict = max(worst, e), strict + sv
        strict_f32 += strict_violations(y_f, vals[i])
    p.destroy()
    return worst, strict, strict_f32


def _unpack(wp, K, C, R, S):
    """KCRS[16]c[16]k -> KCRS (inverse of the closed-form packing map)."""
    KB, CB = wp.shape[:2]
    return wp.transpose(0, 5, 1, 4, 2, 3).reshape(KB * 16, CB * 16, R, S)[:K, :C]


@pytest.mark.parametrize("model", ["resnet50", "vgg16", "inception_v3"])
def test_teacher_forced_layers(neo, model):
    g = wl.MODELS[model](1)
    w, strict, strict_f32 = _teacher_forced_convs(neo, g)
    print(f"\n{model}: worst per-layer rel L2 {w:.2e}; elements beyond 1e-4(1+|ref|): {strict} "
          f"(float32 CPU pipeline: {strict_f32})")
    assert_strict_ceiling(strict, strict_f32, f"{model} teacher-forced layers")


def _gate_network(y, ref, g, what):
    """rel L2 and the output-scale floor, the plain-clause count under the
    float32 pipeline's ceiling (assert_close_network), and top-1 agreement."""
    e, strict = assert_close_network(y, ref, what, graph=g)
    assert (np.argmax(y, 1) == np.argmax(ref, 1)).all(), what + ": top-1 differs"
    return e, strict


@pytest.mark.parametrize("model", ["resnet50", "vgg16", "inception_v3"])
def test_end_to_end_batch1(neo, model):
    g = wl.MODELS[model](1)
    ref = oracle_output(g)
    _gate_network(run_plan(neo, g), ref, g, f"{model} b1")


@pytest.mark.parametrize("model", ["resnet50", "vgg16"])
def test_end_to_end_batch32(neo, model):
    """Batch 32 on the GPU, all 32 images against the oracle's batch-32 output
    (computed once per seed and cached)."""
    g = wl.MODELS[model](32)
    y = run_plan(neo, g)
    ref = oracle_output(g)
    _gate_network(y, ref, g, f"{model} b32")
    for i in range(32):     # each image at its own scale, too
        assert_close_network(y[i:i + 1], ref[i:i + 1], f"{model} b32 image {i}")


def test_tuned_fused_resnet50_batch32(neo):
    """The batch-32 ResNet-50 plan the bench times (tuned, every fusion, graph
    replay): all 32 images against the oracle, two replays bit-identical."""
    torch = torch_cuda()
    g = wl.MODELS["resnet50"](32)
    fl = (neo.PLAN_TUNE | neo.PLAN_HIPGRAPH | neo.PLAN_GROUP | neo.PLAN_FUSE_GAP |
          neo.PLAN_FUSE_PAIRS | neo.PLAN_FUSE_CHAINS)
    p = neo.Plan(g, flags=fl)
    x = dev(g.x)
    out = torch.empty((32, 1000), device="cuda")
    p.run(x, out)
    y = host(out)
    p.run(x, out)
    np.testing.assert_array_equal(host(out), y)
    p.destroy()
    ref = oracle_output(g)
    _gate_network(y, ref, g, "fused resnet50 b32")
    for i in range(32):
        assert_close_network(y[i:i + 1], ref[i:i + 1], f"fused resnet50 b32 image {i}")


def test_naive_plan_bit_identical_resnet50(neo):
    g = wl.resnet50(1)
    np.testing.assert_array_equal(run_plan(neo, g), run_plan(neo, g, neo.PLAN_NAIVE))


def test_hipgraph_replay_bit_identical(neo):
    """Graph replays (several, with eager work and synchronizations between
    them) give exactly the eager result; a new output pointer recaptures."""
    torch = torch_cuda()
    g = wl.tiny_graph()
    eager = run_plan(neo, g)
    p = neo.Plan(g, flags=neo.PLAN_HIPGRAPH)
    x = dev(g.x)
    for i in range(4):
        y = p.run(x)                      # fresh output tensor: recapture each time
        torch.ones(1000, device="cuda").sum()
        np.testing.assert_array_equal(host(y), eager)
    out = torch.empty_like(y)
    for i in range(3):
        out.fill_(-1.0)
        p.run(x, out)
        np.testing.assert_array_equal(host(out), eager)
    p.destroy()


def test_tuned_plan_matches_oracle_and_fills_db(neo, tmp_path):
    """Local search at plan creation: every conv workload timed and stored;
    the tuned plan still matches the oracle; the database persists."""
    neo.tune_db_clear()
    g = wl.tiny_graph()
    p = neo.Plan(g, flags=neo.PLAN_TUNE | neo.PLAN_HIPGRAPH)
    d = p.describe()
    convs = [s for s in d["steps"] if s["kind"] == "conv"]
    assert all(s["conv"]["tuned"] for s in convs)
    n_shapes = len({tuple(sorted((k, str(v)) for k, v in s["conv"].items()
                                 if k not in ("tile", "split", "waves", "tuned", "y_off", "y_tot",
                                              "act", "bias"))) for s in convs})
    assert neo.tune_db_size() == n_shapes
    y = host(p.run(dev(g.x)))
    assert_close(y.reshape(-1, 10), orc.run_graph(g), "tuned tiny")
    p.destroy()
    path = tmp_path / "db.txt"
    assert neo.tune_db_save(path) == n_shapes
    neo.tune_db_clear()
    assert neo.tune_db_load(path) == n_shapes
    p2 = neo.Plan(g)                       # untuned flags: configurations come from the db
    assert all(s["conv"]["tuned"] for s in p2.describe()["steps"] if s["kind"] == "conv")
    p2.destroy()


def test_tuned_resnet50_end_to_end(neo):
    g = wl.resnet50(1)
    p = neo.Plan(g, flags=neo.PLAN_TUNE)
    y = host(p.run(dev(g.x)))
    p.destroy()
    _gate_network(y, oracle_output(g), g, "tuned resnet50 b1")


def test_bench_headline_plan_matches_oracle(neo):
    """The plan bench.py times for ResNet-50 batch 1 -- global search, horizontal
    fusion, tuned, the faster of the searched and one-block plans and of graph
    replay and stream launches -- against the oracle, run several times; the
    same plan in the other launch mode gives the same bits."""
    import os
    import sys
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import bench
    torch = torch_cuda()
    g = wl.resnet50(1)
    p, info = bench.headline_plan(neo, g, None, torch)
    assert info["launch"] in ("graph", "stream")
    d = p.describe()
    x = dev(g.x)
    out = torch.empty((1, 1000), device="cuda")
    ref = oracle_output(g)
    first = None
    for _ in range(3):
        p.run(x, out)
        y = host(out)
        first = y if first is None else first
        np.testing.assert_array_equal(y, first)
    p.destroy()
    base = (neo.PLAN_TUNE | neo.PLAN_GROUP | neo.PLAN_FUSE_GAP | neo.PLAN_FUSE_PAIRS |
            neo.PLAN_FUSE_CHAINS | neo.PLAN_FUSE_POOL)
    other = neo.Plan(g, flags=base | (0 if d["hipgraph"] else neo.PLAN_HIPGRAPH),
                     schemes=bench.plan_schemes(d))
    assert bench.same_steps(other.describe(), d)
    out.fill_(0.0)
    other.run(x, out)
    np.testing.assert_array_equal(host(out), first)
    other.destroy()
    _gate_network(first, ref, g, f"bench headline plan ({info['kept']}, {info['launch']})")
