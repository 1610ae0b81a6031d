"""GPU tests of neo_conv2d_blocked_noalloc, the convolution entry point that
allocates nothing (its split-reduction partials live in the library's fixed
device array): the same results as neo_conv2d_blocked, call after call."""
import numpy as np
import pytest

import oracle as orc
from paper_1809_02697_amd import workloads as wl

from gpu_util import assert_close, dev, host, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def neo():
    torch_cuda()
    from paper_1809_02697_amd import neo as n
    n.lib()
    return n


def _operands(neo, c):
    w, b = neo.fold_bn(c.w, c.bias, c.bn["gamma"], c.bn["beta"], c.bn["mean"], c.bn["var"],
                       c.bn["eps"])
    bpad = np.zeros(-(-c.K // 16) * 16, np.float32)
    bpad[:c.K] = b
    res = neo.to_blocked(dev(c.residual)) if c.epilogue == "res" else None
    act = "relu" if c.epilogue in ("relu", "res") else "none"
    return neo.to_blocked(dev(c.x)), neo.pack_filter(dev(w)), dev(bpad), res, act


def _both(neo, torch, c):
    """(no-alloc output, allocating entry point's output), each into a buffer
    pre-filled with NaN, as host NCHW arrays."""
    x, wp, bp, res, act = _operands(neo, c)
    outs = []
    for fn in (neo.conv2d_blocked_noalloc, neo.conv2d_blocked):
        OH = (c.H + 2 * c.pad[0] - c.R) // c.stride[0] + 1
        OW = (c.W + 2 * c.pad[1] - c.S) // c.stride[1] + 1
        out = torch.full((c.N, -(-c.K // 16), OH, OW, 16), float("nan"), device="cuda")
        fn(x, c.C, wp, c.K, c.R, c.S, bias=bp, stride=c.stride, pad=c.pad, act=act,
           residual=res, out=out)
        outs.append(orc.from_blocked(host(out), c.K))
    return outs


# (C, K, R, stride, pad, H, N, epilogue, forced "fk,fp,split,waves" or None)
CALLS = [
    (512, 512, 3, 1, 1, 14, 1, "relu", "1,1,4,4"),   # a large split first ...
    (256, 200, 3, 2, 1, 13, 2, "relu", "2,1,2,4"),   # ... then a smaller, ragged one
    (1024, 256, 1, 1, 0, 14, 1, "relu", "1,1,8,2"),
    (512, 2048, 1, 1, 0, 7, 1, "res", "2,2,3,1"),
]


def test_noalloc_matches_allocating_entry_point(neo, monkeypatch):
    """Two or more calls in a row, later ones smaller: bit-identical to
    neo_conv2d_blocked under the same launch configuration, and within the
    float32 tolerance of the oracle."""
    torch = torch_cuda()
    for C, K, R, st, pd, H, N, epi, cfg in CALLS:
        c = wl.conv_case(C, K, R, R, st, pd, H, H, N=N, epilogue=epi,
                         out_hw=(H, H) if epi == "res" else None)
        monkeypatch.setenv("NEO_CONV_CONFIG", cfg)
        got, want = _both(neo, torch, c)
        what = f"{C}->{K} {R}x{R}/s{st} H{H} N{N} {cfg}"
        print(f"\n[noalloc] {what}", flush=True)
        np.testing.assert_array_equal(got, want, err_msg=what)
        assert_close(got, orc.layer_forward(c), what)


def test_noalloc_default_configuration(neo, monkeypatch):
    """Without a forced configuration (the cost model's choice), twice."""
    torch = torch_cuda()
    monkeypatch.delenv("NEO_CONV_CONFIG", raising=False)
    for C, K, R, st, pd, H in [(512, 512, 3, 2, 1, 14), (64, 64, 3, 1, 1, 56)]:
        c = wl.conv_case(C, K, R, R, st, pd, H, H)
        got, want = _both(neo, torch, c)
        np.testing.assert_array_equal(got, want)
        assert_close(got, orc.layer_forward(c), f"{C}->{K} default")


def test_noalloc_rejects_partials_above_the_array(neo, monkeypatch):
    """A split whose partials exceed the fixed array (4 splits x 8 images x 16
    channel blocks x 56 x 56 pixels x 64 B = 103 MB) is refused before any
    launch: the output keeps its contents."""
    torch = torch_cuda()
    c = wl.conv_case(64, 256, 3, 3, 1, 1, 56, 56, N=8)
    x, wp, bp, _, _ = _operands(neo, c)
    out = torch.full((8, 16, 56, 56, 16), 3.0, device="cuda")
    monkeypatch.setenv("NEO_CONV_CONFIG", "1,1,4,4")
    with pytest.raises(neo.NeoError) as e:
        neo.conv2d_blocked_noalloc(x, 64, wp, 256, 3, 3, bias=bp, stride=1, pad=1, out=out)
    assert e.value.code == -4 and "scratch" in str(e.value)
    assert bool((out == 3.0).all())
