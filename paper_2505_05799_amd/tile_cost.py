"""Tile costs and the runtime model of the allocator (Sec. 4.2.2, runtime cost
modelling).

The paper decomposes each linear block into tiles, profiles the cost c_t of a
tile of every candidate configuration ahead of time, and estimates a block's
execution time as the serial time of all its tiles over the number of
parallel workers P (valid when tiles far outnumber workers):

    T = (1 / P) * sum over linear blocks of n_tiles * c_t

Here a worker is one slot of the persistent Group-GEMM grid (two workgroups
per CU, P = 2 * 256), and a tile is one unsliced output tile of the kernel:
BM rows x BN channels over the whole K (phase 0 covers gate and up together).
A tile's cost depends on how many row tiles of its group share its weights
through L2 (mt, the group's row tiles), so the table holds, per (phase,
scheme, configuration), three coefficients of

    c_t(K, mt) = a + (K / 128) * (bs + bu / mt)     (ns)

`profile()` measures c_t on the GPU as D * P / n_tiles, where D is the
duration of a Group-GEMM launch over n_tiles >= 4 P equal tiles, at two
reduction depths, with one row tile per group (mt = 1) for every
configuration and also with 8 row tiles per group for the largest
configuration of the scheme (the only one a group of more rows takes), and
fits a, bs, bu.  The same table, in picoseconds, prices the tiles of the
run-time plan on the GPU (`device_table`, mxmoe_set_tile_costs).  It is stored
as JSON beside this module.

    python -m paper_2505_05799_amd.tile_cost --out paper_2505_05799_amd/tile_costs_mi355x.json
"""

from __future__ import annotations

import argparse
import heapq
import json
import math
import os
import sys
import time
from typing import Dict, List, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
DEFAULT_TABLE = os.path.join(HERE, "tile_costs_mi355x.json")

N_CFG = 4
BM = (16, 32, 64, 128)
BN = ((256, 256, 128, 128), (512, 512, 256, 256))   # [phase][configuration]
P_SLOTS = 512                                        # persistent grid: 2 workgroups x 256 CUs
LAUNCH_NS = 6600.0        # an empty persistent Group-GEMM launch (measured on MI355X)
SLICE_NS = 4000.0         # a sliced tile's partial-sum hand-off (3-6 us measured)


def pick_cfg(m: int, scheme, phase: int = 0) -> int:
    """The kernel's run-time choice from the group's rows (w4a4-g128 and mxfp4
    stop at 64, fp8 outside the down phase)."""
    c = 0 if m <= 16 else (1 if m <= 32 else (2 if m <= 64 else 3))
    capped = scheme.a_group > 0 or (getattr(scheme, "fmt", 0) == 2 and phase != 1)
    if scheme.a_bits < 16 and capped and c == 3:
        c = 2
    return c


def n_tiles(m: int, n: int, phase: int, cfg: int) -> int:
    """Unsliced output tiles of a group with m rows and n output channels."""
    if m <= 0:
        return 0
    return -(-m // BM[cfg]) * -(-n // BN[phase][cfg])


class CostTable:
    """c_t(K, mt) = a + K / 128 * (bs + bu / mt) in ns per tile, per (phase,
    scheme name, configuration); entries of two values [a, b] mean bu = 0."""

    def __init__(self, data: dict):
        self.data = data
        self.P = int(data.get("P", P_SLOTS))
        self.slice_ns = float(data.get("slice_ns", SLICE_NS))

    @classmethod
    def load(cls, path: str = DEFAULT_TABLE) -> "CostTable":
        with open(path) as fh:
            return cls(json.load(fh))

    def coef(self, phase: int, scheme, cfg: int):
        e = self.data["cost"][str(phase)][scheme.name][cfg]
        return (float(e[0]), float(e[1]), float(e[2]) if len(e) > 2 else 0.0)

    def tile_ns(self, phase: int, scheme, cfg: int, k: int, mt: int = 1) -> float:
        a, bs, bu = self.coef(phase, scheme, cfg)
        return a + (k / 128.0) * (bs + bu / max(mt, 1))

    def linear_ns(self, m: int, n: int, k: int, phase: int, scheme) -> float:
        """Serial tile time of one linear block (phase 0: gate and up together)."""
        if m <= 0:
            return 0.0
        c = pick_cfg(m, scheme, phase)
        return n_tiles(m, n, phase, c) * self.tile_ns(phase, scheme, c, k, -(-m // BM[c]))

    def block_ns(self, cfg, counts: Sequence[int], schemes) -> List[float]:
        """Modelled Group-GEMM time per phase, T = sum c_t / P, for a block
        configuration, routed counts per expert and (gate, up, down) schemes."""
        out = [0.0, 0.0]
        for e, sch in enumerate(schemes):
            m = int(counts[e]) if e < cfg.E else cfg.T
            F = cfg.F if e < cfg.E else cfg.F_shared
            out[0] += self.linear_ns(m, F, cfg.H, 0, sch[0])
            out[1] += self.linear_ns(m, cfg.H, F, 1, sch[2])
        return [v / self.P for v in out]

    def block_makespan_ns(self, cfg, counts: Sequence[int], schemes) -> List[float]:
        """Modelled Group-GEMM time per phase as the paper defines it before its
        approximation, T = max over workers of the worker's summed tile costs,
        with the tiles dealt the way the kernel deals them: each group's tiles
        sliced along K by the kernel's rule (the fewest slices, at most 8 of at
        least 6 k blocks, whose cost is within half the mean work per worker,
        else the cheapest tile's slices as long as the phase keeps at most one
        tile per worker, up to the first group refused for that), longest first, each to the least loaded of the P
        workers; a sliced tile pays the table's slice hand-off, and the launch
        LAUNCH_NS.  Where tiles far outnumber workers this equals sum c_t / P."""
        out = []
        for ph in (0, 1):
            groups = []
            for e, sch in enumerate(schemes):
                m = int(counts[e]) if e < cfg.E else cfg.T
                if m <= 0:
                    continue
                F = cfg.F if e < cfg.E else cfg.F_shared
                n, k = (F, cfg.H) if ph == 0 else (cfg.H, F)
                scheme = sch[0] if ph == 0 else sch[2]
                c = pick_cfg(m, scheme, ph)
                a, bs, bu = self.coef(ph, scheme, c)
                mt = -(-m // BM[c])
                groups.append((n_tiles(m, n, ph, c), a, bs + bu / mt, k // 128))
            work = sum(nt * max(a + b * kb, 1e-3) for nt, a, b, kb in groups)
            theta = work / self.P / 2.0
            unsliced = sum(g[0] for g in groups)
            added = 0
            stopped = False
            tiles = []
            for nt, a, b, kb in groups:
                smax = max(1, min(8, kb // 6))
                cost = lambda sl: max(a + b * (-(-kb // sl)), 1e-3) + (self.slice_ns if sl > 1 else 0.0)
                best, cbest, fallback = 1, None, True
                for sl in range(1, smax + 1):
                    cs = cost(sl)
                    if cs <= theta:
                        best, fallback = sl, False
                        break
                    if cbest is None or cs < cbest:
                        best, cbest = sl, cs
                if fallback and best > 1 and unsliced + added + nt * (best - 1) > self.P:
                    stopped = True
                if fallback and stopped:
                    best = 1
                added += nt * (best - 1)
                tiles += [cost(best)] * (nt * best)
            tiles.sort(reverse=True)
            heap = [(0.0, i) for i in range(self.P)]
            for c in tiles:
                t, i = heapq.heappop(heap)
                heapq.heappush(heap, (t + c, i))
            out.append(max(t for t, _ in heap) + LAUNCH_NS)
        return out

    def device_table(self) -> np.ndarray:
        """The table as the run-time plan takes it (mxmoe_set_tile_costs): int32
        [phase][scheme][configuration][a, bs, bu, h] in ps, schemes in the
        order of ALL_SCHEMES (the library's kind ids), each value rounded to the
        nearest ps and clamped to the int32 range (bs, bu, h to >= 0; a, a fit's
        intercept, may be negative); h is the slice hand-off.
        Schemes absent from the table get the largest cost, so that a missing
        profile shows as a slow tile rather than a free one."""
        from . import workloads as W
        out = np.zeros((2, len(W.ALL_SCHEMES), N_CFG, 4), dtype=np.int64)
        h = int(round(self.slice_ns * 1000.0))
        for ph in (0, 1):
            for i, s in enumerate(W.ALL_SCHEMES):
                for c in range(N_CFG):
                    if s.name in self.data["cost"][str(ph)]:
                        a, bs, bu = self.coef(ph, s, c)
                        out[ph, i, c] = [round(a * 1000.0), round(bs * 1000.0), round(bu * 1000.0), h]
                    else:
                        out[ph, i, c] = [2_000_000_000, 0, 0, h]
        out[..., 1:] = np.clip(out[..., 1:], 0, 2**31 - 1)
        out[..., 0] = np.clip(out[..., 0], -2**31, 2**31 - 1)
        return out.astype(np.int32)


# ----------------------------------------------------------------------------
# profiling (GPU)
# ----------------------------------------------------------------------------


def _device_linear(scheme, n: int, k: int, gen, dev: str = "cuda"):
    """A QLinear whose codes / scales / zeros are random tensors (on `dev`) of
    the scheme's formats (timing does not depend on the values)."""
    import torch
    from . import workloads as W
    s = scheme
    if s.w_bits == 16:
        w = (torch.randn((n, k), generator=gen, device=dev) * 0.02).to(torch.bfloat16).view(torch.int16)
        return W.QLinear(s, n, k, w)
    if s.weight_only:
        qm = (1 << s.w_bits) - 1
        codes = torch.randint(0, qm + 1, (n, k), generator=gen, device=dev, dtype=torch.int32).to(torch.uint8)
        scales = (torch.rand((n, k // 128), generator=gen, device=dev) * 0.01 + 0.001).to(torch.float16)
        zeros = torch.randint(0, qm + 1, (n, k // 128), generator=gen, device=dev).to(torch.float16)
        return W.QLinear(s, n, k, codes, scales.view(torch.int16), zeros.view(torch.int16))
    if s.fmt == 1:   # mxfp4: e2m1 codes 0..15, E8M0 bytes per 32 near 2^-7
        codes = torch.randint(0, 16, (n, k), generator=gen, device=dev, dtype=torch.int32).to(torch.uint8)
        scales = torch.randint(118, 124, (n, k // 32), generator=gen, device=dev, dtype=torch.int32).to(torch.uint8)
        return W.QLinear(s, n, k, codes, scales)
    if s.fmt == 2:   # fp8: finite e4m3 bytes (magnitude codes 0..0x7E, either sign)
        mag = torch.randint(0, 0x7F, (n, k), generator=gen, device=dev, dtype=torch.int32)
        sgn = torch.randint(0, 2, (n, k), generator=gen, device=dev, dtype=torch.int32) * 0x80
        scales = torch.rand(n, generator=gen, device=dev) * 0.01 + 0.001
        return W.QLinear(s, n, k, (mag | sgn).to(torch.uint8), scales)
    qm = (1 << (s.w_bits - 1)) - 1
    codes = torch.randint(-qm, qm + 1, (n, k), generator=gen, device=dev, dtype=torch.int32).to(torch.int8)
    if s.w_group > 0:
        scales = (torch.rand((n, k // 128), generator=gen, device=dev) * 0.01 + 0.001).to(torch.float16)
        return W.QLinear(s, n, k, codes, scales.view(torch.int16))
    scales = torch.rand(n, generator=gen, device=dev) * 0.01 + 0.001
    return W.QLinear(s, n, k, codes, scales)


REUSE_ROWS = 8   # row tiles per group in the weight-sharing probe


def _probe(scheme, phase: int, k: int, cfgs: Sequence[int], reps: int, n_sets: int = 8, reuse: int = 1,
           log=print):
    """Launch durations (ms) of the profiled phase for each configuration, with
    `reuse` row tiles per group."""
    import torch
    from . import mxmoe as M
    from . import workloads as W
    # the profiled phase has N = 8192 output channels and reduction depth k;
    # with one row tile per group 64 (gate|up) or 128 (down) experts, with
    # several 16 experts, so that every launch holds >= 4 P tiles
    H, F = (k, 8192) if phase == 0 else (8192, k)
    E = 16 if reuse > 1 else (64 if phase == 0 else 128)
    T_max = E * 128 * reuse
    cfg = W.BlockConfig(f"probe_{scheme.name}_p{phase}_k{k}_r{reuse}", T=T_max, H=H, F=F, E=E, k=1, n_shared=0,
                        F_shared=0, act="bf16", zipf_s=None, alloc=lambda e, r: (scheme,) * 3)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(1234 + phase * 7 + k + reuse)
    # n_sets distinct weight sets, dealt to the experts in turn: the working set
    # (several hundred MB at least) stays well above what the caches hold
    sets = []
    for _ in range(n_sets):
        lins = [_device_linear(scheme, F, H, gen), _device_linear(scheme, F, H, gen), _device_linear(scheme, H, F, gen)]
        sets.append([M.PackedLinear(q, "bf16") for q in lins])
    torch.cuda.synchronize()
    for ps in sets:
        for p in ps:
            p.release_sources()
    blk = W.Block(cfg, 0, np.zeros((0, H), np.uint16), np.zeros((0, 1), np.int32), np.zeros((0, 1), np.float32))
    mb = M.MoEBlock(blk, T_max=T_max, packed=[sets[e % n_sets] for e in range(E)])
    x = (torch.randn((T_max, H), generator=gen, device="cuda")).to(torch.bfloat16)
    out = {}
    ev = M.PhaseEvents()
    for c in cfgs:
        m = BM[c] * reuse
        T = E * m
        ids = (torch.arange(T, device="cuda", dtype=torch.int32) // m).reshape(T, 1).contiguous()
        w = torch.ones((T, 1), dtype=torch.float32, device="cuda")
        xs = x[:T].contiguous()
        for _ in range(2):
            mb.forward(xs, ids, w, skip_combine=True)
        torch.cuda.synchronize()
        d = []
        for _ in range(reps):
            mb.forward(xs, ids, w, skip_combine=True, events=ev)
            torch.cuda.synchronize()
            d.append(ev.elapsed_ms()[1 if phase == 0 else 3])
        nt = E * n_tiles(m, F if phase == 0 else H, phase, c)
        out[c] = (float(np.median(d)), nt)
        log(f"[tile_cost] {scheme.name} phase {phase} K {k} cfg {c} row tiles {reuse}: "
            f"{out[c][0]:.4f} ms over {nt} tiles")
    del mb, sets
    torch.cuda.empty_cache()
    return out


def profile(schemes=None, k_lo: int = 1024, k_hi: int = 4096, reps: int = 5, log=print) -> dict:
    """Per (phase, scheme, configuration) [a, bs, bu]: every configuration is
    timed with one row tile per group at K = k_lo and k_hi, giving a and the
    slope b1 = bs + bu; the scheme's largest configuration also with
    REUSE_ROWS row tiles per group, giving the slope bR = bs + bu / REUSE_ROWS,
    so bu = (b1 - bR) R / (R - 1) (>= 0) and bs = b1 - bu; a is the mean of the
    two fits' intercepts.  Smaller configurations hold one row tile per group
    whatever the rows, so they keep bs = b1, bu = 0."""
    from . import workloads as W
    schemes = list(schemes or W.ALL_SCHEMES)
    R = REUSE_ROWS
    kb_lo, kb_hi = k_lo / 128.0, k_hi / 128.0
    table = {"P": P_SLOTS, "k_points": [k_lo, k_hi], "reuse_rows": R, "slice_ns": SLICE_NS,
             "unit": "ns per tile; c_t(K, mt) = a + K / 128 * (bs + bu / mt)",
             "cost": {"0": {}, "1": {}}, "raw": {"0": {}, "1": {}}}
    for s in schemes:
        for phase in (0, 1):
            top = pick_cfg(1 << 20, s, phase)            # kinds capped at 64-row tiles stop at 2
            cfgs = list(range(top + 1))
            lo = _probe(s, phase, k_lo, cfgs, reps, log=log)
            hi = _probe(s, phase, k_hi, cfgs, reps, log=log)
            rlo = _probe(s, phase, k_lo, [top], reps, reuse=R, log=log)
            rhi = _probe(s, phase, k_hi, [top], reps, reuse=R, log=log)
            per_tile = lambda r, c: r[c][0] * 1e6 * P_SLOTS / r[c][1]
            ab, raw = [], []
            for c in range(N_CFG):
                cc = min(c, top)
                c1, c2 = per_tile(lo, cc), per_tile(hi, cc)
                b1 = (c2 - c1) / (kb_hi - kb_lo)
                a1 = c1 - b1 * kb_lo
                if cc == top:
                    r1, r2 = per_tile(rlo, top), per_tile(rhi, top)
                    bR = (r2 - r1) / (kb_hi - kb_lo)
                    aR = r1 - bR * kb_lo
                    bu = max(0.0, (b1 - bR) * R / (R - 1))
                    bs = b1 - bu
                    a = 0.5 * (a1 + aR)
                    raw.append([round(c1, 1), round(c2, 1), round(r1, 1), round(r2, 1)])
                else:
                    bs, bu, a = b1, 0.0, a1
                    raw.append([round(c1, 1), round(c2, 1)])
                ab.append([round(a, 1), round(bs, 2), round(bu, 2)])
            table["cost"][str(phase)][s.name] = ab
            table["raw"][str(phase)][s.name] = raw
    return table


def measure_block(cfg, schemes=None, reps: int = 10, seed: int = 0):
    """Measured Group-GEMM launch durations (ms, mean of `reps` forwards) of a
    block configuration, with its own or the given per-expert schemes; also the
    whole forward (ms) and the routed counts."""
    import torch
    from . import mxmoe as M
    from . import workloads as W
    if schemes is not None:
        sch = list(schemes)
        cfg = W.BlockConfig(**{**cfg.__dict__, "alloc": lambda e, r: sch[e], "shared_alloc": sch[-1]})
    blk = W.make_block(cfg, seed=seed)
    mb = M.MoEBlock(blk)
    x = M.act_tensor(blk.x, cfg.act)
    ids = torch.from_numpy(blk.topk_ids.copy()).cuda()
    w = torch.from_numpy(blk.topk_w.copy()).cuda()
    for _ in range(3):
        mb.forward(x, ids, w)
    torch.cuda.synchronize()
    ev = [M.PhaseEvents() for _ in range(reps)]
    for i in range(reps):
        mb.forward(x, ids, w, events=ev[i])
    torch.cuda.synchronize()
    ph = np.array([e.elapsed_ms() for e in ev]).mean(axis=0)
    counts = np.bincount(blk.topk_ids.ravel(), minlength=cfg.E)
    del mb
    torch.cuda.empty_cache()
    return {"gate_up_ms": float(ph[1]), "down_ms": float(ph[3]), "forward_ms": float(ph.sum()),
            "counts": counts.tolist(), "schemes": [tuple(s) for s in W.schemes_of(cfg, seed)]}


def validate(table: CostTable, names: Sequence[str], log=print) -> List[dict]:
    """Modelled against measured Group-GEMM launch time on block configurations."""
    from . import workloads as W
    out = []
    for n in names:
        cfg = W.CONFIGS[n]
        meas = measure_block(cfg)
        model = table.block_ns(cfg, meas["counts"], meas["schemes"])
        mk = table.block_makespan_ns(cfg, meas["counts"], meas["schemes"])
        rec = {"workload": n, "gate_up_ms": round(meas["gate_up_ms"], 4), "gate_up_model_ms": round(model[0] / 1e6, 4),
               "gate_up_makespan_ms": round(mk[0] / 1e6, 4),
               "down_ms": round(meas["down_ms"], 4), "down_model_ms": round(model[1] / 1e6, 4),
               "down_makespan_ms": round(mk[1] / 1e6, 4)}
        log(f"[tile_cost] validate {json.dumps(rec)}")
        out.append(rec)
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--out", default=DEFAULT_TABLE)
    ap.add_argument("--schemes", default="", help="comma-separated scheme names (default: all)")
    ap.add_argument("--reps", type=int, default=5)
    ap.add_argument("--validate", default="mixtral,dsv2lite,qwen15_uniform,qwen15_mixed,qwen15_w5a5",
                    help="workloads whose measured launch times are compared with the model ('' = none)")
    ap.add_argument("--validate-only", action="store_true", help="keep the stored costs, redo the validation")
    ap.add_argument("--merge", action="store_true",
                    help="profile only --schemes and keep the stored costs of every other scheme")
    a = ap.parse_args()
    from . import workloads as W
    log = lambda *x: print(*x, file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    if a.validate_only:
        table = CostTable.load(a.out).data
    else:
        schemes = [W.SCHEME_BY_NAME[n] for n in a.schemes.split(",") if n] or None
        new = profile(schemes, reps=a.reps, log=log)
        cmd = "python -m paper_2505_05799_amd.tile_cost" + (f" --schemes {a.schemes}" if a.schemes else "")
        if a.merge and schemes:
            table = CostTable.load(a.out).data
            for key in ("cost", "raw"):
                for ph in ("0", "1"):
                    table[key][ph].update(new[key][ph])
            prev = table.get("command", "")
            step = cmd + " --merge"
            if step not in prev.split("; then "):
                table["command"] = (prev + "; then " if prev else "") + step
        else:
            table = new
            table["command"] = cmd
    names = [n for n in a.validate.split(",") if n]
    if names:
        table["validation"] = validate(CostTable(table), names, log=log)
    with open(a.out, "w") as fh:
        json.dump(table, fh, indent=1)
    print(f"[tile_cost] wrote {a.out} in {time.perf_counter() - t0:.0f}s", file=sys.stderr)


if __name__ == "__main__":
    main()
