"""NEO_PLAN_FUSE_GAP: a global average pool folded into the conv before it
(which then writes per-16-pixel channel sums) and the dense layers after it
(which read their mean).  Host checks of when the fold applies; GPU parity
against the oracle and the unfolded plan."""
import numpy as np
import pytest

import oracle as orc
from paper_1809_02697_amd import neo
from paper_1809_02697_amd import workloads as wl

import nets


def _plan(g, flags=0):
    p = neo.Plan(g, flags=neo.PLAN_HOST_ONLY | neo.PLAN_FUSE_GAP | flags)
    d = p.describe()
    p.destroy()
    return d


def head_graph(K=40, hw=5, N=1, extra_reader=False, seed=21):
    """stem -> conv (K channels, hw x hw) -> global pool -> flatten -> dense;
    optionally a second reader of the conv's output."""
    b = wl._Builder("head", (N, 24, hw + 2, hw + 2), np.random.Generator(np.random.PCG64(seed)))
    x = b.conv(0, 32, 3, name="stem")
    c = b.conv(x, K, 1, name="c")
    s = b.gap(c)
    if extra_reader:
        z = b.gap(b.conv(c, 16, 1, name="z"))
        s = b.concat([s, z], name="cat")
        s = b.flatten(s, K + 16)
    else:
        s = b.flatten(s, K)
    b.output(b.dense(s, 10, name="fc"))
    return b.finish(lambda rng: rng.normal(0, 1, (N, 24, hw + 2, hw + 2)).astype(np.float32))


def test_resnet50_folds_its_pool():
    g = nets.resnet50()
    d = _plan(g, neo.PLAN_GROUP)
    assert not any(s["kind"] == "gap" for s in d["steps"])
    last = [s for s in d["steps"] if s["kind"] == "conv"][-1]
    assert last["conv"].get("gap_sums") and last["conv"]["N"] == 1
    dense = [s for s in d["steps"] if s["kind"] == "dense"]
    assert len(dense) == 1 and dense[0]["dense"]["gap_parts"] == 4    # ceil(7 * 7 / 16)
    assert dense[0]["in"] == last["out"]                                # and so runs after it
    assert d["steps"].index(dense[0]) > d["steps"].index(last)


@pytest.mark.parametrize("build", [lambda: nets.inception_v3(),     # the pool reads a concat
                                   lambda: wl.resnet50(2),            # two images
                                   lambda: head_graph(extra_reader=True)])
def test_pool_kept_where_the_fold_does_not_apply(build):
    d = _plan(build())
    assert any(s["kind"] == "gap" for s in d["steps"])
    assert not any(s.get("conv", {}).get("gap_sums") for s in d["steps"])


def test_without_the_flag_nothing_folds():
    p = neo.Plan(nets.resnet50(), flags=neo.PLAN_HOST_ONLY)
    d = p.describe()
    p.destroy()
    assert sum(s["kind"] == "gap" for s in d["steps"]) == 1


# ---- GPU ---------------------------------------------------------------------------------
@pytest.fixture(scope="module")
def gneo():
    from gpu_util import torch_cuda
    torch_cuda()
    neo.lib()
    return neo


def _run(g, flags):
    from gpu_util import dev, host
    p = neo.Plan(g, flags=flags)
    d = p.describe()
    y = host(p.run(dev(g.x)))
    p.destroy()
    return y, d


@pytest.mark.gpu
@pytest.mark.parametrize("K,hw", [(40, 5), (64, 4), (16, 9), (2048, 7)])
def test_folded_pool_matches_oracle(gneo, K, hw):
    """Ragged K (padding channels), one and several partial rows, a row of
    one pixel (hw = 9: 81 = 5 * 16 + 1)."""
    from gpu_util import assert_close, rel_l2
    g = head_graph(K, hw)
    ref = orc.run_graph(g)
    y, d = _run(g, neo.PLAN_FUSE_GAP)
    assert not any(s["kind"] == "gap" for s in d["steps"])
    assert_close(y.reshape(ref.shape), ref, f"folded pool K={K} {hw}x{hw}")
    y0, _ = _run(g, 0)
    assert rel_l2(y, y0) <= 1e-6


@pytest.mark.gpu
def test_resnet50_folded_tuned_replayed(gneo):
    """The headline configuration's flags (tuned, fused, replayed) with the
    pool folded: every replay equals the first, and matches the oracle."""
    from gpu_util import assert_close_network, dev, host, rel_l2, torch_cuda
    torch = torch_cuda()
    g = wl.resnet50(1)
    ref = orc.run_graph(g)
    flags = neo.PLAN_TUNE | neo.PLAN_GROUP | neo.PLAN_FUSE_GAP | neo.PLAN_HIPGRAPH
    p = neo.Plan(g, flags=flags)
    x = dev(g.x)
    out = torch.empty((1, 1000), device="cuda")
    first = None
    for _ in range(3):
        out.fill_(-1.0)
        p.run(x, out)
        torch.ones(1000, device="cuda").sum()
        y = host(out)
        first = y if first is None else first
        np.testing.assert_array_equal(y, first)
    p.destroy()
    assert_close_network(first, ref, "resnet50 folded pool", graph=g)
    y0, _ = _run(g, neo.PLAN_TUNE | neo.PLAN_GROUP)
    assert rel_l2(first, y0) <= 1e-6
