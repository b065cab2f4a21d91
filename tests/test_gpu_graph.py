"""The block forward captured once in a HIP graph and replayed: every replay,
with eager forwards and synchronizations in between, gives the eager output
bit for bit (the forward is deterministic and keeps no state between calls
that a replay could miss: queue heads, slice counters and the status word are
rebuilt by its own kernels)."""

import numpy as np
import pytest

from paper_2505_05799_amd import mxmoe as M
from paper_2505_05799_amd import workloads as W
from tests.gpuhelp import say, torch_mod, upload_inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["tiny", "mix"])
def test_graph_replay_matches_eager(name):
    torch = torch_mod()
    if name == "tiny":
        blk = W.make_block("tiny")
    else:
        sch = [(W.W4G128,) * 3, (W.W8A8, W.W8A8, W.W2G128), (W.W4A4,) * 3, (W.MXFP4,) * 3,
               (W.W4A4G128, W.W4A4G128, W.W3G128), (W.W16,) * 3, (W.FP8, W.FP8, W.W8A8)]
        blk = W.random_small_block(5, T=300, H=256, F=384, E=6, k=2, n_shared=1, F_shared=256, act="bf16",
                                   schemes=sch, skew=1.0)
    mb = M.MoEBlock(blk)
    x, ids, w = upload_inputs(blk)
    y_eager = mb.forward(x, ids, w)
    torch.cuda.synchronize()
    ref = y_eager.clone()
    y = torch.empty_like(x)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        mb.forward(x, ids, w, y=y)          # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        mb.forward(x, ids, w, y=y)
    for rep in range(3):
        y.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), ref.view(torch.int16)), f"replay {rep}"
        mb.forward(x, ids, w)                # eager work between replays
        torch.cuda.synchronize()
    say(f"graph {name}: 3 replays bit-exact")
