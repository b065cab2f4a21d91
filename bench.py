#!/usr/bin/env python3
"""MoE-block forward benchmark on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload mixtral]

One step = one full block forward through libmxmoe (routing, plan, activation
quantization, gate/up Group-GEMM with fused SiLU-gate, h quantization, down
Group-GEMM, combine) on synthetic inputs already resident in HBM.  The timed
steps carry no per-phase events (those run in separate eager forwards after
the timed region); --graph times replays of the forward captured once in a
HIP graph instead.  Prints one
JSON line: effective TFLOP/s (2*m*N*K over real routed rows, summed over all
linears) and microseconds per layer, the roofline of the dominant kernel (the
gate/up Group-GEMM launch, timed with HIP events on the library's stream), and
the CPU oracle timed on a bounded token sample.

The default workload is the Qwen2-57B-A14B-shaped prefill block, the largest
single-GPU configuration: 16384 tokens, hidden 3584, 64 routed experts of FFN
2560, top-8, one shared expert of FFN 20480, Zipf(1.0) routing skew; hot
experts (ranks 1-10) and the shared expert w8a8, the others w4a4.

The 256 MiB Infinity Cache is defeated by rotation: the timed steps cycle
through ceil(512 MiB / touched bytes) + 1 independent copies of the packed
weights and of x, so no step finds the previous step's operands in the cache.
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np

HBM_PEAK = 8.0e12            # B/s
# dense MFMA peaks of MI355X by operand type (int8 in OP/s)
MFMA_PEAK = {"i8": 5.0e15, "fp8": 5.0e15, "fp6": 10.1e15, "fp4": 10.1e15, "bf16": 2.5e15, "fp16": 2.5e15}
ROTATE_BYTES = 512 << 20     # Infinity Cache (256 MiB) defeat: rotate copies covering twice its size


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def act_bytes(s):
    """Bytes per activation element a linear of scheme s reads: 0.5 for MXFP4
    codes, 1 for int8 / FP8 codes, 2 for 16-bit rows."""
    if getattr(s, "fmt", 0) == 1:
        return 0.5
    return 1.0 if s.a_bits < 16 else 2.0


def mfma_dtype(s, act):
    """Operand type of the MFMA a scheme runs on (the key of MFMA_PEAK)."""
    fmt = getattr(s, "fmt", 0)
    if fmt == 1:
        return "fp4"
    if fmt == 2:
        return "fp8"
    if fmt == 3:
        return "fp6"
    return "i8" if s.a_bits < 16 else act


def group_stats(blk, counts):
    """Per (phase, expert) algorithmic flops / bytes and the MFMA dtype."""
    cfg = blk.cfg
    out = []
    for e, lins in enumerate(blk.linears):
        m = int(counts[e]) if e < cfg.E else cfg.T
        if m == 0:
            continue
        for phase, idx in ((0, (0, 1)), (1, (2,))):
            fl = by = 0.0
            for j in idx:
                q = lins[j]
                fl += 2.0 * m * q.n * q.k
                by += q.nbytes_packed + m * q.k * act_bytes(q.scheme)
            n_out = lins[idx[0]].n
            by += m * n_out * 2.0          # h rows, or slot rows in the activation dtype
            s = lins[idx[0]].scheme
            out.append({"expert": e, "phase": phase, "m": m, "flops": fl, "bytes": by,
                        "dtype": mfma_dtype(s, cfg.act), "scheme": s.name})
    return out


def roofline(groups, phase, t_s, traffic=None):
    """Roofline of one Group-GEMM launch: algorithmic flops and bytes of the
    phase's groups over the launch time; traffic: measured HBM bytes per launch
    (rocprofv3 counters, copy-calibrated) or None."""
    g = [x for x in groups if x["phase"] == phase]
    flops = sum(x["flops"] for x in g)
    nbytes = sum(x["bytes"] for x in g)
    t_mfma = sum(x["flops"] / MFMA_PEAK[x["dtype"]] for x in g)
    t_hbm = nbytes / HBM_PEAK
    if t_mfma >= t_hbm:
        peak = flops / t_mfma / 1e12          # dtype-weighted MFMA peak
        ach = flops / t_s / 1e12
        out = {"bound": "mfma", "achieved": round(ach, 2), "peak": round(peak, 1), "unit": "TFLOP/s",
               "frac": round(ach / peak, 4)}
    else:
        ach = nbytes / t_s / 1e9
        out = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK / 1e9, "unit": "GB/s",
               "frac": round(ach / (HBM_PEAK / 1e9), 4)}
    out["traffic"] = traffic
    out["algorithmic_bytes"] = round(nbytes)
    return out


def per_group(blocks, xs, blk, ids, w, groups, reps=6):
    """Groups of one phase with the same scheme and the same bound (HBM when
    moving the group's bytes at 8 TB/s takes longer than its MFMA work at the
    dtype's peak, else MFMA), each timed alone with an expert mask (the launch
    then holds only their tiles), against the roof of its bound.  The
    repetitions rotate over the cache-defeating copies."""
    import torch
    from paper_2505_05799_amd import mxmoe as M
    cfg = blk.cfg
    G = cfg.E + cfg.n_shared
    classes = {}
    for g in groups:
        t_mem = g["bytes"] / HBM_PEAK
        t_mma = g["flops"] / MFMA_PEAK[g["dtype"]]
        key = (g["phase"], g["scheme"], "hbm" if t_mem > t_mma else "mfma")
        classes.setdefault(key, []).append(g)
    out = []
    ev = M.PhaseEvents()
    for (phase, scheme, bound), gs in sorted(classes.items()):
        mask = [0] * G
        for g in gs:
            mask[g["expert"]] = 1
        for i in range(2):
            blocks[i % len(blocks)].forward(xs[i % len(xs)], ids, w, expert_mask=mask, skip_combine=True)
        ts = []
        for i in range(reps):
            blocks[i % len(blocks)].forward(xs[i % len(xs)], ids, w, expert_mask=mask, skip_combine=True, events=ev)
            torch.cuda.synchronize()
            ts.append(ev.elapsed_ms()[1 if phase == 0 else 3])
        t = float(np.median(ts)) / 1e3
        if bound == "hbm":
            frac = sum(g["bytes"] for g in gs) / t / HBM_PEAK
        else:
            frac = sum(g["flops"] / MFMA_PEAK[g["dtype"]] for g in gs) / t
        rows = [g["m"] for g in gs]
        out.append({"phase": "gate_up" if phase == 0 else "down", "scheme": scheme, "bound": bound,
                    "experts": len(gs), "rows": [min(rows), max(rows)], "ms_alone": round(t * 1e3, 4),
                    "frac": round(frac, 3)})
    return out


def measured_traffic(workload, phase):
    """HBM bytes per launch from the committed counter summary of this workload
    and phase, or None if there is none or the kernel sources changed since."""
    from paper_2505_05799_amd import profiling as P
    name = ("group_gemm_gate_up_" if phase == 0 else "group_gemm_down_") + workload + "_traffic.txt"
    rec = P.read_summary(os.path.join(ROOT, "profiles", name))
    return None if rec is None or rec.get("workload") != workload else rec["traffic_bytes"]


def copy_calibration():
    """A plain device copy of known size, for scaling the memory counters."""
    import torch
    from paper_2505_05799_amd import profiling as P
    a = torch.empty(P.COPY_BYTES, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    log(f"[bench] copied {P.COPY_BYTES >> 20} MiB 3 times")


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(blk, tokens, seed=0):
    """The CPU oracle as it stands, on a uniform random sample of `tokens`
    tokens of the workload (all their routed experts and the shared experts)."""
    from oracle import mxmoe_oracle as O
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [os.cpu_count() or 1])
    except Exception:
        cores = os.cpu_count() or 1
    cfg = blk.cfg
    n = min(tokens, cfg.T)
    sel = np.sort(np.random.default_rng([seed, 11]).choice(cfg.T, size=n, replace=False))
    ids = blk.topk_ids[sel]
    counts = np.bincount(ids.ravel(), minlength=cfg.E)
    flops = cfg.scaled(n).flops(counts)
    t0 = time.perf_counter()
    O.moe_forward(blk.x[sel], ids, blk.topk_w[sel], blk.linears, cfg.E, cfg.act)
    dt = time.perf_counter() - t0
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{n} of {cfg.T} tokens drawn uniformly at random (seed {seed}): their "
                      f"{int((counts > 0).sum())} routed experts and {cfg.n_shared} shared expert(s), fp64 "
                      f"numpy incl. dequantization of every linear touched",
            "seconds": round(dt, 2), "cpu_model": cpu_model()}


def touched_bytes(blk, counts):
    """Packed weight bytes of the experts that receive tokens, plus x."""
    cfg = blk.cfg
    b = 0
    for e, lins in enumerate(blk.linears):
        if e < cfg.E and counts[e] == 0:
            continue
        b += sum(q.nbytes_packed for q in lins)
    return b + blk.x.nbytes


def rotation_copies(mb, blk, x, n):
    """n - 1 further MoEBlocks over device copies of the packed weights, and
    copies of x, for cache-defeating rotation."""
    import copy
    from paper_2505_05799_amd import mxmoe as M
    blocks, xs = [mb], [x]
    for _ in range(n - 1):
        packed = []
        for ps in mb.packed:
            row = []
            for p in ps:
                c = copy.copy(p)
                c.buf = p.buf.clone()
                row.append(c)
            packed.append(row)
        blocks.append(M.MoEBlock(blk, packed=packed))
        xs.append(x.clone())
    return blocks, xs


def compare_per_expert(args):
    """One Group-GEMM launch per phase against the same micro-kernels launched
    once per expert (the per-expert invocation the paper's motivation study
    measures, Sec. 3.2 and its throughput figure): 60 experts, gate+up of shape
    [N, K] = [2816, 2048] per expert, top-4, 512 tokens, uniform schemes.  The
    per-expert figure sums the HIP-event durations of the single-expert
    launches (each runs after its own plan, which is not counted), so it
    leaves out launch gaps: a lower bound on sequential execution."""
    import torch
    from paper_2505_05799_amd import mxmoe as M
    from paper_2505_05799_amd import workloads as W
    out = []
    for sch in (W.W16, W.W4G128, W.W8A8, W.MXFP4, W.FP8):
        cfg = W.BlockConfig(f"per_expert_{sch.name}", T=512, H=2048, F=1408, E=60, k=4, n_shared=0, F_shared=0,
                            act="bf16", zipf_s=args.zipf, alloc=lambda e, r, s=sch: (s, s, s),
                            description="60 experts [2816, 2048] gate+up, top-4, 512 tokens")
        blk = W.make_block(cfg, seed=args.seed)
        mb = M.MoEBlock(blk)
        x = M.act_tensor(blk.x, cfg.act)
        ids = torch.from_numpy(blk.topk_ids.copy()).cuda()
        w = torch.from_numpy(blk.topk_w.copy()).cuda()
        counts = np.bincount(blk.topk_ids.ravel(), minlength=cfg.E)
        live = [e for e in range(cfg.E) if counts[e] > 0]
        fl_gu = sum(2.0 * 2 * int(counts[e]) * cfg.F * cfg.H for e in live)
        for _ in range(args.warmup):
            mb.forward(x, ids, w, skip_combine=True)
        reps = max(args.steps, 3)
        ev = M.PhaseEvents()
        fused = []
        for _ in range(reps):
            mb.forward(x, ids, w, skip_combine=True, events=ev)
            torch.cuda.synchronize()
            fused.append(ev.elapsed_ms())
        seq = []
        for _ in range(reps):
            tot = np.zeros(M.N_PHASES)
            for e in live:
                mask = [0] * cfg.E
                mask[e] = 1
                mb.forward(x, ids, w, skip_combine=True, events=ev, expert_mask=mask)
                torch.cuda.synchronize()
                tot += np.array(ev.elapsed_ms())
            seq.append(tot)
        f = np.mean(fused, axis=0)
        q = np.mean(seq, axis=0)
        rec = {"scheme": sch.name, "tokens": 512, "experts_live": len(live),
               "gate_up_ms_fused": round(float(f[1]), 4), "gate_up_ms_per_expert_sum": round(float(q[1]), 4),
               "gate_up_tflops_fused": round(fl_gu / (f[1] / 1e3) / 1e12, 1),
               "gate_up_tflops_per_expert": round(fl_gu / (q[1] / 1e3) / 1e12, 1),
               "down_ms_fused": round(float(f[3]), 4), "down_ms_per_expert_sum": round(float(q[3]), 4),
               "speedup_gate_up": round(float(q[1] / f[1]), 2)}
        print(json.dumps(rec), flush=True)
        out.append(rec)
        del mb
        torch.cuda.empty_cache()
    return out


def pct(v, q):
    return round(float(np.percentile(v, q)), 4)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="qwen2")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-tokens", type=int, default=6144)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-rotate", action="store_true", help="time one copy of the operands (no cache defeat)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 256 MiB device copy (memory-counter calibration)")
    ap.add_argument("--compare-per-expert", action="store_true",
                    help="one Group-GEMM launch vs per-expert launches of the same micro-kernels "
                         "(60 experts [2816, 2048], top-4, 512 tokens); one JSON line per scheme")
    ap.add_argument("--zipf", type=float, default=1.5, help="router skew of --compare-per-expert")
    ap.add_argument("--no-groups", action="store_true", help="skip the per-group roofline breakdown")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of the forward captured in a HIP graph instead of eager forwards")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}); "
              "the multi-GPU expert-parallel layout is a design, not a measured path.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2505_05799_amd import mxmoe as M
    from paper_2505_05799_amd import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.compare_per_expert:
        M.load_library()
        compare_per_expert(args)
        return
    M.load_library()
    cfg = W.CONFIGS[args.workload]
    t0 = time.perf_counter()
    log(f"[bench] generating {cfg.name}: {cfg.description}")
    blk = W.make_block(cfg, seed=args.seed)
    log(f"[bench] inputs ready in {time.perf_counter() - t0:.1f}s; packing")
    mb = M.MoEBlock(blk)
    x = M.act_tensor(blk.x, cfg.act)
    ids = torch.from_numpy(blk.topk_ids.copy()).cuda()
    w = torch.from_numpy(blk.topk_w.copy()).cuda()
    y = torch.empty_like(x)
    counts = np.bincount(blk.topk_ids.ravel(), minlength=cfg.E)
    flops = cfg.flops(counts)
    touched = touched_bytes(blk, counts)
    ncopy = 1 if args.no_rotate else -(-ROTATE_BYTES // touched) + 1
    blocks, xs = rotation_copies(mb, blk, x, ncopy)
    torch.cuda.synchronize()
    log(f"[bench] packed {sum(p.nbytes for ps in mb.packed for p in ps) / 1e6:.1f} MB "
        f"({touched / 1e6:.1f} MB touched per forward, {ncopy} rotating copies); "
        f"{flops / 1e9:.1f} GFLOP per forward; warmup {args.warmup}")

    def step(i, ev=None):
        c = i % ncopy
        blocks[c].forward(xs[c], ids, w, y=y, events=ev)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    graphs = None
    if args.graph:
        # every copy's forward captured once; a replay issues the same kernels
        # without host launch overhead between them
        cs = torch.cuda.Stream()
        cs.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cs):
            for c in range(ncopy):
                step(c)
        torch.cuda.current_stream().wait_stream(cs)
        torch.cuda.synchronize()
        graphs = []
        for c in range(ncopy):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                step(c)
            graphs.append(g)
        for i in range(args.warmup):
            graphs[i % ncopy].replay()
        torch.cuda.synchronize()
    # Timed region: exactly `steps` forwards.  Eager steps carry the library's
    # per-phase HIP events (recorded on the stream the kernels run on), which
    # give the per-step durations and the dominant launch's duration.
    evs = [M.PhaseEvents() for _ in range(args.steps)] if graphs is None else None
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)] if graphs is not None else None
    log(f"[bench] timing {args.steps} steps ({'eager' if graphs is None else 'graph replays'})")
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for i in range(args.steps):
        if graphs is None:
            step(i, evs[i])
        else:
            starts[i].record()
            graphs[i % ncopy].replay()
    if starts is not None:
        starts[args.steps].record()
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    ms = (t2 - t1) * 1e3 / args.steps
    if graphs is None:
        phases = np.array([e.elapsed_ms() for e in evs])          # [steps, 5]
        per_step = np.array([e.span_ms() for e in evs])
    else:
        # phase durations of graph replays: eager forwards with events after the timed region
        evs = [M.PhaseEvents() for _ in range(args.steps)]
        for i in range(args.steps):
            step(i, evs[i])
        torch.cuda.synchronize()
        phases = np.array([e.elapsed_ms() for e in evs])
        per_step = np.array([starts[i].elapsed_time(starts[i + 1]) for i in range(args.steps)])
    ph_mean = phases.mean(axis=0)
    groups = group_stats(blk, counts)
    phase_gu, phase_dn = 1, 3
    dom = phase_gu if ph_mean[phase_gu] >= ph_mean[phase_dn] else phase_dn
    dname = "gate|up" if dom == phase_gu else "down"
    roof = roofline(groups, 0 if dom == phase_gu else 1, ph_mean[dom] / 1e3,
                    measured_traffic(args.workload, 0 if dom == phase_gu else 1))
    kact = "bf16" if cfg.act == "bf16" else "fp16"
    roof["kernel"] = f"group_gemm_kernel<{kact}, {dname}>"
    roof["launch_ms"] = round(float(ph_mean[dom]), 4)
    other = roofline(groups, 1 if dom == phase_gu else 0, ph_mean[phase_dn if dom == phase_gu else phase_gu] / 1e3,
                     measured_traffic(args.workload, 1 if dom == phase_gu else 0))
    other["kernel"] = f"group_gemm_kernel<{kact}, {'down' if dom == phase_gu else 'gate|up'}>"
    dtypes = sorted({g["dtype"] for g in groups})

    rec = {
        "metric": "MoE-block us/layer + effective TFLOP/s; % of HBM/MFMA roofline per group",
        "value": round(flops / (ms / 1e3) / 1e12, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "us_per_layer": round(ms * 1e3, 1),
        "step_ms": {"median": pct(per_step, 50), "p10": pct(per_step, 10), "p90": pct(per_step, 90)},
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "+".join(dtypes),
        "data": "synthetic",
        "config": {"workload": cfg.description, "name": cfg.name, "tokens": cfg.T, "hidden": cfg.H, "ffn": cfg.F,
                   "experts": cfg.E, "top_k": cfg.k, "shared_experts": cfg.n_shared,
                   "ffn_shared": cfg.F_shared, "avg_weight_bits": round(W.avg_weight_bits(cfg), 3),
                   "gflop": round(flops / 1e9, 2)},
        "roofline": roof,
        "roofline_other": other,
        "phases_ms": {n: round(float(v), 4) for n, v in zip(M.PHASE_NAMES, ph_mean)},
        "timing": ("eager forwards with per-phase HIP events" if graphs is None
                   else "replays of the forward captured in a HIP graph"),
        "cache_defeat": (f"rotating {ncopy} copies of the packed weights and x "
                         f"({touched / 1e6:.1f} MB touched per forward)" if ncopy > 1 else "none"),
    }
    if not args.no_groups:
        log("[bench] per-group rooflines (each class of groups timed alone)")
        rec["groups"] = per_group(blocks, xs, blk, ids, w, groups)
    if not args.no_cpu_baseline:
        log(f"[bench] CPU oracle on {args.cpu_tokens} random tokens")
        rec["cpu_baseline"] = cpu_baseline(blk, args.cpu_tokens, args.seed)
    else:
        rec["cpu_baseline"] = None
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
