"""The no-allocation forward (mxmoe_moe_forward_noalloc) against the
forward with a caller workspace (mxmoe_moe_forward), through the C ABI: two
calls in a row on the library's scratch array, the second with fewer tokens,
each bit for bit equal to the workspace forward on the same inputs (both run
the same kernels on the same plan), and a block too large for the array is
rejected before anything is enqueued."""

import numpy as np
import pytest

from oracle import mxmoe_oracle as O
from paper_2505_05799_amd import mxmoe as M
from paper_2505_05799_amd import workloads as W
from tests.gpuhelp import say, torch_mod, upload_inputs
from tests.stagewise import check_pure

pytestmark = pytest.mark.gpu


def _pair(blk, T):
    """Inputs of the first T tokens of blk (same weights)."""
    sub = W.Block(blk.cfg.scaled(T), blk.seed, np.ascontiguousarray(blk.x[:T]),
                  np.ascontiguousarray(blk.topk_ids[:T]), np.ascontiguousarray(blk.topk_w[:T]), blk.linears)
    return sub


@pytest.mark.parametrize("name", ["tiny", "mixed_bf16"])
def test_noalloc_matches_workspace_forward(name):
    torch = torch_mod()
    if name == "tiny":
        blk = W.make_block("tiny")
        sizes = (64, 17)
    else:
        sch = [(W.W4G128,) * 3, (W.W8A8, W.W8A8, W.W2G128), (W.W4A4,) * 3, (W.MXFP4,) * 3,
               (W.W4A4G128, W.W4A4G128, W.W3G128), (W.W16,) * 3, (W.FP8, W.FP8, W.W8A8)]
        blk = W.random_small_block(23, T=300, H=256, F=384, E=6, k=2, n_shared=1, F_shared=256, act="bf16",
                                   schemes=sch, skew=1.0)
        sizes = (300, 5)
    mb = M.MoEBlock(blk)
    for T in sizes:
        sub = _pair(blk, T)
        x, ids, w = upload_inputs(sub)
        y_ref = mb.forward(x, ids, w)
        torch.cuda.synchronize()
        y = torch.full_like(x, float("nan"))
        mb.forward_noalloc(x, ids, w, y=y)
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), y_ref.view(torch.int16)), f"{name} T={T}"
        ref = O.moe_forward(sub.x, sub.topk_ids, sub.topk_w, sub.linears, sub.cfg.E, sub.cfg.act)
        ratio = check_pure(M.act_numpy(y, sub.cfg.act), ref["y"], sub.cfg.act, f"noalloc {name} T={T}")
        say(f"noalloc {name} T={T}: equal to the workspace forward; worst err / (1e-2 rowmax) {ratio:.4f}")


def test_noalloc_rejects_blocks_beyond_the_array():
    torch = torch_mod()
    blk = W.random_small_block(3, T=8, H=256, F=256, E=4, k=2, act="bf16", schemes=[(W.W8A8,) * 3] * 4)
    mb = M.MoEBlock(blk, T_max=8)
    lib = M.load_library()
    import ctypes as C
    T_big = 1
    while lib.mxmoe_workspace_bytes(C.byref(mb.B), T_big) <= M.NOALLOC_SCRATCH_BYTES:
        T_big *= 2
    x = torch.zeros((T_big, 256), dtype=torch.bfloat16, device="cuda")
    ids = torch.zeros((T_big, 2), dtype=torch.int32, device="cuda")
    ids[:, 1] = 1
    w = torch.ones((T_big, 2), dtype=torch.float32, device="cuda")
    y = torch.full_like(x, 7.0)
    st = lib.mxmoe_moe_forward_noalloc(C.byref(mb.B), M._ptr(mb.table), T_big, M._ptr(x), M._ptr(ids), M._ptr(w),
                                       M._ptr(y), M._stream_ptr(None))
    torch.cuda.synchronize()
    assert st == M.ERR_WORKSPACE
    assert bool((y == 7.0).all())        # nothing was enqueued
    say(f"noalloc: T={T_big} rejected (workspace above {M.NOALLOC_SCRATCH_BYTES >> 20} MiB)")
