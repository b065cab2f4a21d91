"""Shared helpers of the GPU parity tests (imported by tests only)."""

import os
import sys
import time

import numpy as np

from oracle import mxmoe_oracle as O
from paper_2505_05799_amd import mxmoe as M
from paper_2505_05799_amd import workloads as W

# Block outputs: per token row t, |y - r| <= REL_TOL * max_h |r[t, h]| + slack[t, h],
# where slack bounds the effect of a8/a4 activation codes of the down projection
# whose rounding decision depends on fp32-vs-fp64 accumulation (see the oracle).
REL_TOL = 1e-2


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


def compare_block(y_np, ref, act, what=""):
    """Returns (worst bound ratio, number of rows with slack) and asserts the tolerance."""
    yv = O.act_values(y_np, act)
    r = ref["y"]
    slack = ref["slack"] if ref["slack"] is not None else np.zeros_like(r)
    scale = np.abs(r).max(axis=1, keepdims=True)
    err = np.abs(yv - r)
    bound = REL_TOL * scale + slack
    bad = err > bound
    ratio = float((err / np.maximum(REL_TOL * scale, 1e-30)).max()) if r.size else 0.0
    if bad.any():
        t, h = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {int(bad.sum())} outputs out of tolerance; first t={t} h={h} "
                             f"gpu={yv[t, h]!r} ref={r[t, h]!r} rowmax={scale[t, 0]!r} slack={slack[t, h]!r}")
    return ratio, int((slack > 0).any(axis=1).sum())
