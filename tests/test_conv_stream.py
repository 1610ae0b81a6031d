"""The streaming pointwise kernel (a launch configuration with fp = 0): in
plans whose results file names it for a conv, against the oracle and, bit for
bit, against the tile kernel with one wave and no split."""
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


def _line(arch, N, C, H, W, K, cfg):
    # arch N C H W K R S sh sw ph pw wmfma xb yb fk fp split waves us
    return f"{arch} {N} {C} {H} {W} {K} 1 1 1 1 0 0 1 16 16 {cfg} 1.0\n"


def _run(neo, g, cfgs, tmp_path):
    """The plan of g with each conv's configuration forced through a results
    file: {conv node: "fk fp split waves"}."""
    neo.tune_db_clear()
    N, C, H, W = g.input_shape
    path = tmp_path / "db.txt"
    with open(path, "w") as f:
        for n, cfg in cfgs.items():
            f.write(_line("gfx950", N, C, H, W, g.nodes[n].K, cfg))
    assert neo.tune_db_load(path) == len(cfgs)
    p = neo.Plan(g)
    d = p.describe()
    y = host(p.run(dev(g.x)))
    p.destroy()
    neo.tune_db_clear()
    return y, d


CASES = [
    # N, C, H, W, K, residual, stream configurations "fk fp split waves"
    (2, 64, 56, 56, 64, False, ["4 0 1 1", "2 0 1 2", "1 0 1 4", "4 0 1 8"]),
    (1, 64, 56, 56, 256, True, ["4 0 1 2", "2 0 1 1"]),
    (3, 48, 9, 7, 40, True, ["1 0 1 1", "1 0 1 8"]),      # ragged channels and pixels
    (2, 128, 28, 28, 512, True, ["2 0 1 2", "1 0 1 4"]),  # 8 input blocks
]


@pytest.mark.parametrize("case", CASES, ids=["64-64", "64-256res", "ragged", "128-512res"])
def test_stream_matches_tile_kernel_and_oracle(neo, case, tmp_path):
    N, C, H, W, K, res, cfgs = case
    g = wl.pointwise_graph(N=N, C=C, H=H, W=W, K=K, residual=res)
    conv = [i for i, n in enumerate(g.nodes) if n.op == "conv"][-1]
    ref = orc.run_graph(g)
    base = {i: "1 1 1 1" for i, n in enumerate(g.nodes) if n.op == "conv"}
    y_tile, _ = _run(neo, g, base, tmp_path)
    assert_close(y_tile, ref, "tile kernel")
    for cfg in cfgs:
        print(f"\n[stream] {case[:6]} {cfg}", flush=True)
        y, d = _run(neo, g, {**base, conv: cfg}, tmp_path)
        st = [s for s in d["steps"] if s["kind"] == "conv" and s["node"] == conv][0]
        assert st["conv"]["tile"][1] == 0 and st["conv"]["tuned"], st["conv"]
        np.testing.assert_array_equal(y, y_tile)
        assert_close(y, ref, f"stream {cfg}")


def test_stream_rejected_where_it_does_not_apply(neo, tmp_path):
    """A results file naming the streaming kernel for a filter in the ABI's
    order is refused; one naming it with fk not dividing the output blocks is
    loaded but not used (the conv runs the tile kernel's cost-model choice)."""
    N, C, H, W, K = 1, 64, 8, 8, 48
    path = tmp_path / "db.txt"
    with open(path, "w") as f:
        f.write(_line("gfx950", N, C, H, W, K, "2 0 1 1").replace(" 1 16 16 ", " 0 16 16 "))
    with pytest.raises(neo.NeoError):
        neo.tune_db_load(path)   # fp = 0 with wmfma = 0
    g = wl.pointwise_graph(N=N, C=C, H=H, W=W, K=K)
    y, d = _run(neo, g, {1: "2 0 1 1"}, tmp_path)
    st = [s for s in d["steps"] if s["kind"] == "conv"][0]["conv"]
    assert st["tile"][1] > 0 and not st["tuned"]
    assert_close(y, orc.run_graph(g), "fallback")
