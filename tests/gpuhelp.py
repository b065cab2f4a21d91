"""Shared helpers of the GPU parity tests (imported by tests only)."""

import sys

from paper_2505_05799_amd import mxmoe as M

def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def torch_mod():
    import torch
    assert torch.cuda.is_available(), "GPU test run without a GPU"
    return torch


def upload_inputs(block, device="cuda"):
    torch = torch_mod()
    x = M.act_tensor(block.x, block.cfg.act, device)
    ids = torch.from_numpy(block.topk_ids.copy()).to(device)
    w = torch.from_numpy(block.topk_w.copy()).to(device)
    return x, ids, w
