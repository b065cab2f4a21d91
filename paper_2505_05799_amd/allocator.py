"""Hardware-aware bit-width allocation (Sec. 4.2, Eq. 3-7).

For one MoE block, pick a scheme for every linear block (expert i, linear j)
from a candidate set S to minimize L^r * T^(1-r) subject to the packed weight
bytes staying within a budget M (Eq. 7), where

* L = sum Delta[i, j, k(i, j)]: Delta[i, j, k] is the output distortion
  ||O_hat - O||_2 of the block when only linear block (i, j) is quantized with
  scheme k (Eq. 5-6);
* T = (1/P) sum over linear blocks of n_tiles * c_t, the runtime model of
  `tile_cost` (tile configurations follow the kernel's choice from the rows);
* the memory of a linear block is its packed size under the scheme.

Gate and up of an expert share one scheme in this engine (they run in one
tile), so the linear blocks are (expert, gate+up) and (expert, down).

Delta comes from the library's own forward on a calibration batch: with every
routed expert's linear block j in scheme k and everything else 16-bit, the
per-(token, slot) down rows the forward leaves in its workspace hold
w_ts * Expert_e(x_t) for each slot separately, so the distortion that
quantizing (i, j) alone causes is read off the slots routed to expert i
(shared experts: their own slots).  One forward per (j, k) covers all experts.

The solver is a dynamic program over (memory, time) on a grid: for each grid
cell the least L, then the best L^r T^(1-r) over the cells within the memory
budget; the chosen assignment is re-evaluated exactly.  Memory is rounded up
to the grid (the budget is never exceeded), time to the nearest cell.
"""

from __future__ import annotations

import argparse
import json
import math
import sys
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np


@dataclass
class Problem:
    """Per linear block b and candidate c: loss L[b, c], time T[b, c] (ns of
    serial tile time), memory W[b, c] (bytes); budget M bytes; exponent r."""
    L: np.ndarray
    T: np.ndarray
    W: np.ndarray
    M: float
    r: float
    allowed: Optional[np.ndarray] = None   # bool [b, c]; None = all

    def objective(self, choice: Sequence[int]) -> Tuple[float, float, float, float]:
        idx = np.arange(len(choice))
        ch = np.asarray(choice)
        l = float(self.L[idx, ch].sum())
        t = float(self.T[idx, ch].sum())
        w = float(self.W[idx, ch].sum())
        return l ** self.r * t ** (1.0 - self.r), l, t, w


def solve(p: Problem, mem_cells: int = 256, time_cells: int = 256) -> Tuple[List[int], dict]:
    """Assignment (candidate index per linear block) minimizing L^r T^(1-r)
    under sum W <= M.  Raises ValueError when no assignment fits the budget."""
    nb, nc = p.L.shape
    ok = np.ones((nb, nc), bool) if p.allowed is None else p.allowed.copy()
    wmin = np.where(ok, p.W, np.inf).min(axis=1)
    if wmin.sum() > p.M * (1 + 1e-12):
        raise ValueError("no assignment fits the memory budget")
    # memory grid over what may be spent above the per-block minimum; rounded up
    spare = p.M - wmin.sum()
    extra = np.where(ok, p.W - wmin[:, None], 0.0)
    mq = max(spare, 1e-9) / mem_cells
    wcell = np.where(ok, np.ceil(extra / mq - 1e-9), 0).astype(np.int64)
    # time grid over the reachable range, rounded to nearest
    tmin = np.where(ok, p.T, np.inf).min(axis=1)
    tmax = np.where(ok, p.T, -np.inf).max(axis=1)
    span = max(float((tmax - tmin).sum()), 1e-9)
    tq = span / time_cells
    tcell = np.where(ok, np.rint((p.T - tmin[:, None]) / tq), 0).astype(np.int64)
    INF = np.inf
    best = np.full((mem_cells + 1, time_cells + 1), INF)
    best[0, 0] = 0.0
    pick = np.zeros((nb, mem_cells + 1, time_cells + 1), np.int16)
    for b in range(nb):
        nxt = np.full_like(best, INF)
        arg = np.zeros(best.shape, np.int16)
        for c in range(nc):
            if not ok[b, c]:
                continue
            dw, dt = int(wcell[b, c]), int(tcell[b, c])
            if dw > mem_cells or dt > time_cells:
                continue
            cand = np.full_like(best, INF)
            cand[dw:, dt:] = best[: mem_cells + 1 - dw, : time_cells + 1 - dt] + p.L[b, c]
            better = cand < nxt
            nxt[better] = cand[better]
            arg[better] = c
        best = nxt
        pick[b] = arg
    if not np.isfinite(best).any():
        raise ValueError("no assignment fits the memory budget on the grid")
    # objective on the grid cells (time at the cell's value), then backtrack
    tvals = tmin.sum() + np.arange(time_cells + 1) * tq
    with np.errstate(invalid="ignore", divide="ignore"):
        obj = np.where(np.isfinite(best), np.maximum(best, 0.0) ** p.r * np.maximum(tvals, 1e-30)[None, :] ** (1 - p.r),
                       INF)
    cands = np.argsort(obj, axis=None)[:64]
    best_choice, best_val = None, INF
    for flat in cands:
        if not np.isfinite(obj.flat[flat]):
            break
        wi, ti = np.unravel_index(flat, obj.shape)
        choice = [0] * nb
        for b in range(nb - 1, -1, -1):
            c = int(pick[b, wi, ti])
            choice[b] = c
            wi -= int(wcell[b, c])
            ti -= int(tcell[b, c])
        val, l, t, w = p.objective(choice)
        if w <= p.M * (1 + 1e-12) and val < best_val:
            best_choice, best_val = choice, val
    if best_choice is None:
        raise ValueError("no assignment fits the memory budget")
    val, l, t, w = p.objective(best_choice)
    return best_choice, {"objective": val, "L": l, "T_ns": t, "W_bytes": w}


def brute_force(p: Problem) -> Tuple[List[int], float]:
    """Exhaustive search (small problems only)."""
    import itertools
    nb, nc = p.L.shape
    best, arg = math.inf, None
    for choice in itertools.product(range(nc), repeat=nb):
        if p.allowed is not None and not all(p.allowed[b, c] for b, c in enumerate(choice)):
            continue
        val, l, t, w = p.objective(choice)
        if w <= p.M * (1 + 1e-12) and val < best:
            best, arg = val, list(choice)
    return arg, best


# ----------------------------------------------------------------------------
# problem construction for a block (GPU for Delta)
# ----------------------------------------------------------------------------


def sensitivity(cfg, candidates, calib_tokens: int = 1024, seed: int = 0, log=print) -> np.ndarray:
    """Delta [G, 2, |S|]: block output distortion when linear block (i, j) alone
    (j = 0 gate+up, 1 down) takes candidate k, everything else 16-bit, on a
    calibration batch of the block's synthetic inputs."""
    import torch
    from . import mxmoe as M
    from . import workloads as W
    G = cfg.E + cfg.n_shared
    T = min(calib_tokens, cfg.T)
    base = W.make_block(cfg, seed=seed, T=T, with_weights=False)
    ws16 = W.make_block(W.BlockConfig(**{**cfg.__dict__, "alloc": lambda e, r: (W.W16,) * 3,
                                        "shared_alloc": (W.W16,) * 3}), seed=seed, T=T)
    x = M.act_tensor(base.x, cfg.act)
    ids = torch.from_numpy(base.topk_ids.copy()).cuda()
    w = torch.from_numpy(base.topk_w.copy()).cuda()
    S = cfg.k + cfg.n_shared

    def slots(block):
        mb = M.MoEBlock(block, T_max=T)
        mb.forward(x, ids, w, skip_combine=True, fp32_slots=True)   # differences need the fp32 rows
        torch.cuda.synchronize()
        s = mb.ws_view("slots", torch.float32, T * S * cfg.H, T).reshape(T, S, cfg.H).double().cpu().numpy()
        del mb
        return s

    ref = slots(ws16)
    owner = np.concatenate([base.topk_ids, np.tile(np.arange(cfg.E, G), (T, 1))], axis=1)  # [T, S] expert per slot
    delta = np.zeros((G, 2, len(candidates)))
    for j in range(2):
        for ci, s in enumerate(candidates):
            def alloc(e, r, s=s, j=j):
                return (s, s, W.W16) if j == 0 else (W.W16, W.W16, s)
            c2 = W.BlockConfig(**{**cfg.__dict__, "alloc": alloc,
                                  "shared_alloc": alloc(0, 0)})
            blk = W.make_block(c2, seed=seed, T=T)
            d = slots(blk) - ref
            e2 = (d * d).sum(axis=2)                        # [T, S]
            for g in range(G):
                delta[g, j, ci] = math.sqrt(float(e2[owner == g].sum()))
            log(f"[allocator] Delta for linear block {'gate+up' if j == 0 else 'down'} in {s.name}: "
                f"mean {delta[:, j, ci].mean():.4g}")
    return delta


def block_problem(cfg, candidates, table, delta: np.ndarray, budget_bits: float, r: float,
                  counts: Optional[Sequence[int]] = None, seed: int = 0) -> Tuple[Problem, list]:
    """The allocation problem of one block: linear blocks (g, j) in order
    g = 0..G-1, j = 0 (gate+up), 1 (down)."""
    from . import workloads as W
    G = cfg.E + cfg.n_shared
    if counts is None:
        ids, _ = W.make_routing(cfg, seed)
        counts = np.bincount(ids.ravel(), minlength=cfg.E)
    nb, nc = 2 * G, len(candidates)
    L = np.zeros((nb, nc))
    Tm = np.zeros((nb, nc))
    Wm = np.zeros((nb, nc))
    params = 0
    blocks = []
    for g in range(G):
        m = int(counts[g]) if g < cfg.E else cfg.T
        F = cfg.F if g < cfg.E else cfg.F_shared
        for j in range(2):
            b = 2 * g + j
            blocks.append((g, j))
            for c, s in enumerate(candidates):
                L[b, c] = delta[g, j, c]
                if j == 0:
                    Tm[b, c] = table.linear_ns(m, F, cfg.H, 0, s)
                    Wm[b, c] = 2 * W.QLinear(s, F, cfg.H, None).nbytes_packed
                else:
                    Tm[b, c] = table.linear_ns(m, cfg.H, F, 1, s)
                    Wm[b, c] = W.QLinear(s, cfg.H, F, None).nbytes_packed
            params += (2 if j == 0 else 1) * F * cfg.H
    M = budget_bits * params / 8.0
    return Problem(L, Tm / table.P, Wm, M, r), blocks


def allocation_to_alloc(cfg, candidates, choice, blocks):
    """(expert -> (gate, up, down) schemes, shared schemes) from a solution."""
    G = cfg.E + cfg.n_shared
    sch = [[None, None, None] for _ in range(G)]
    for (g, j), c in zip(blocks, choice):
        s = candidates[c]
        if j == 0:
            sch[g][0] = sch[g][1] = s
        else:
            sch[g][2] = s
    return [tuple(x) for x in sch]


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--workload", default="qwen15_w5a5")
    ap.add_argument("--candidates", default="w8a8,w4a4,w4a4g128")
    ap.add_argument("--budget-bits", type=float, default=5.25)
    ap.add_argument("--r", type=float, default=0.75)
    ap.add_argument("--calib-tokens", type=int, default=1024)
    ap.add_argument("--table", default=None)
    ap.add_argument("--out", default=None, help="write the allocation as JSON")
    ap.add_argument("--evaluate", action="store_true",
                    help="run the allocation, each candidate used uniformly, and the workload's own allocation "
                         "on the GPU; one JSON line each")
    a = ap.parse_args()
    from . import tile_cost
    from . import workloads as W
    cfg = W.CONFIGS[a.workload]
    cands = [W.SCHEME_BY_NAME[n] for n in a.candidates.split(",")]
    table = tile_cost.CostTable.load(a.table or tile_cost.DEFAULT_TABLE)
    log = lambda *x: print(*x, file=sys.stderr, flush=True)
    delta = sensitivity(cfg, cands, a.calib_tokens, log=log)
    prob, blocks = block_problem(cfg, cands, table, delta, a.budget_bits, a.r)
    choice, info = solve(prob)
    sch = allocation_to_alloc(cfg, cands, choice, blocks)
    rec = {"workload": cfg.name, "budget_bits": a.budget_bits, "r": a.r, "candidates": a.candidates,
           **{k: (round(v, 6) if isinstance(v, float) else v) for k, v in info.items()},
           "avg_bits": round(8 * info["W_bytes"] / (prob.M * 8 / a.budget_bits), 3),
           "schemes": [[s.name for s in t] for t in sch]}
    print(json.dumps(rec), flush=True)
    if a.out:
        with open(a.out, "w") as fh:
            json.dump(rec, fh, indent=1)
    if a.evaluate:
        G = cfg.E + cfg.n_shared
        params = sum((2 + 1) * (cfg.F if g < cfg.E else cfg.F_shared) * cfg.H for g in range(G))
        runs = [("allocated", sch)] + [(f"uniform {s.name}", [(s, s, s)] * G) for s in cands]
        runs.append(("workload's own", W.schemes_of(cfg)))
        for name, schemes in runs:
            meas = tile_cost.measure_block(cfg, schemes)
            byts = sum(2 * W.QLinear(t[0], cfg.F if g < cfg.E else cfg.F_shared, cfg.H, None).nbytes_packed
                       + W.QLinear(t[2], cfg.H, cfg.F if g < cfg.E else cfg.F_shared, None).nbytes_packed
                       for g, t in enumerate(schemes))
            loss = None
            if all(t[0] in cands and t[2] in cands for t in schemes):
                loss = sum(delta[g, 0, cands.index(t[0])] + delta[g, 1, cands.index(t[2])]
                           for g, t in enumerate(schemes))
            model = table.block_ns(cfg, meas["counts"], schemes)
            print(json.dumps({"run": name, "packed_bits": round(8 * byts / params, 3),
                              "L": None if loss is None else round(float(loss), 4),
                              "gemm_ms": round(meas["gate_up_ms"] + meas["down_ms"], 4),
                              "gemm_model_ms": round((model[0] + model[1]) / 1e6, 4),
                              "forward_ms": round(meas["forward_ms"], 4)}), flush=True)


if __name__ == "__main__":
    main()
