"""HBM traffic of a Group-GEMM launch from rocprofv3 counter runs.

Two counter passes over the same command (FETCH_SIZE, then WRITE_SIZE; one
counter group per run) give KiB per dispatch; each is scaled by what the same
counter reads for a plain copy of known size (torch's device-to-device copy of
256 MiB, which runs the runtime's copyBuffer kernel), because the counters do
not see every memory channel at face value.  The summary records a hash of the
kernel's sources; a reader treats the figure as stale once they change.

    python -m paper_2505_05799_amd.profiling \\
        --fetch F.csv --write W.csv --copy-fetch CF.csv --copy-write CW.csv \\
        --kernel "group_gemm_kernel<1, 0>" --out profiles/NAME.txt --command "..."

With --sq, the csv files are SQ counter passes (each a run of its own, with
GRBM_GUI_ACTIVE in every pass) and the summary gives, per kernel, the MFMA
pipe utilisation, the instruction mix per MFMA instruction and where the
wavefronts' resident cycles went:

    python -m paper_2505_05799_amd.profiling --sq --csv A.csv --csv B.csv \
        --kernel "group_gemm_kernel<1, 0>" --kernel "group_gemm_kernel<1, 1>" \
        --workload qwen2 --out profiles/NAME.txt --command "..."
"""

import argparse
import csv
import hashlib
import json
import os

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
COPY_KERNEL = "__amd_rocclr_copyBuffer"
COPY_BYTES = 256 << 20          # bytes read and bytes written per copy dispatch
# sources whose change invalidates a traffic figure of the Group-GEMM
GEMM_SOURCES = ("group_gemm_impl.h", "mxmoe_internal.h", "group_gemm.hip", "gg_bf16_p0.hip", "gg_bf16_p1.hip",
                "gg_f16_p0.hip", "gg_f16_p1.hip")
MARK = "# traffic-json: "


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def counter_kib(path: str, kernel: str, counter: str):
    """Mean counter value (KiB) per dispatch of the kernels whose name contains
    `kernel`, and the dispatch count."""
    vals = {}
    with open(path, newline="") as fh:
        for row in csv.DictReader(fh):
            if row["Counter_Name"] != counter or kernel not in row["Kernel_Name"]:
                continue
            d = row["Dispatch_Id"]
            vals[d] = vals.get(d, 0.0) + float(row["Counter_Value"])
    if not vals:
        raise SystemExit(f"no {counter} rows for kernel '{kernel}' in {path}")
    return sum(vals.values()) / len(vals), len(vals)


def summarize(fetch, write, copy_fetch, copy_write, kernel):
    f_kib, nf = counter_kib(fetch, kernel, "FETCH_SIZE")
    w_kib, nw = counter_kib(write, kernel, "WRITE_SIZE")
    cf_kib, _ = counter_kib(copy_fetch, COPY_KERNEL, "FETCH_SIZE")
    cw_kib, _ = counter_kib(copy_write, COPY_KERNEL, "WRITE_SIZE")
    f_scale = COPY_BYTES / 1024.0 / cf_kib
    w_scale = COPY_BYTES / 1024.0 / cw_kib
    read_b = f_kib * 1024.0 * f_scale
    write_b = w_kib * 1024.0 * w_scale
    return {"kernel": kernel, "dispatches": [nf, nw], "fetch_kib": round(f_kib, 1), "write_kib": round(w_kib, 1),
            "copy_fetch_kib": round(cf_kib, 1), "copy_write_kib": round(cw_kib, 1),
            "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4),
            "read_bytes": round(read_b), "write_bytes": round(write_b), "traffic_bytes": round(read_b + write_b),
            "sources": kernel_source_hash()}


def read_summary(path: str):
    """The traffic record of a summary file, or None if absent or stale."""
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        for line in fh:
            if line.startswith(MARK):
                rec = json.loads(line[len(MARK):])
                return rec if rec.get("sources") == kernel_source_hash() else None
    return None


# SQ counters: the shader engines' counters are summed over the chip; the
# GRBM_GUI_ACTIVE value in these csv files reads about 8 x (duration x shader
# clock), i.e. it is summed over the 8 XCDs, so one XCD's busy cycles are a
# eighth of it.  The MFMA pipe utilisation is the busy cycles of all 1024
# SIMDs over 1024 x one XCD's GUI-active cycles.
N_XCD = 8
N_SIMD = 1024


def sq_counters(paths, kernel):
    """Per-dispatch means of every counter in the csv files for the kernels
    whose name contains `kernel`, plus the mean duration (ns)."""
    tot, cnt, dur = {}, {}, {}
    for path in paths:
        per = {}
        with open(path, newline="") as fh:
            for row in csv.DictReader(fh):
                if kernel not in row["Kernel_Name"]:
                    continue
                key = (path, row["Dispatch_Id"])
                per.setdefault(key, {})
                name = row["Counter_Name"]
                per[key][name] = per[key].get(name, 0.0) + float(row["Counter_Value"])
                dur[key] = int(row["End_Timestamp"]) - int(row["Start_Timestamp"])
        for key, vals in per.items():
            for name, v in vals.items():
                tot[name] = tot.get(name, 0.0) + v
                cnt[name] = cnt.get(name, 0) + 1
    if not tot:
        raise SystemExit(f"no counter rows for kernel '{kernel}' in {paths}")
    mean = {k: tot[k] / cnt[k] for k in tot}
    mean["duration_ns"] = sum(dur.values()) / len(dur)
    mean["dispatches"] = max(cnt.values())
    return mean


def sq_derived(c):
    """Derived figures of one kernel's SQ counter means (absent inputs skip a figure)."""
    out = {}
    g = c.get("GRBM_GUI_ACTIVE")
    if g:
        out["clock_ghz"] = round(g / N_XCD / c["duration_ns"], 3)
        if "SQ_VALU_MFMA_BUSY_CYCLES" in c:
            out["mfma_busy"] = round(c["SQ_VALU_MFMA_BUSY_CYCLES"] / (g / N_XCD * N_SIMD), 4)
    m = c.get("SQ_INSTS_MFMA")
    if m:
        if "SQ_INSTS_VALU" in c:  # SQ_INSTS_VALU counts the MFMA instructions too
            out["valu_per_mfma"] = round((c["SQ_INSTS_VALU"] - m) / m, 3)
        for k, name in (("SQ_INSTS_LDS", "lds_per_mfma"), ("SQ_INSTS_VMEM_RD", "vmem_rd_per_mfma"),
                        ("SQ_INSTS_SALU", "salu_per_mfma")):
            if k in c:
                out[name] = round(c[k] / m, 3)
    w = c.get("SQ_WAVE_CYCLES")
    if w:
        for k, name in (("SQ_WAIT_ANY", "wait_any"), ("SQ_WAIT_INST_ANY", "wait_inst_any"),
                        ("SQ_WAIT_INST_LDS", "wait_inst_lds"), ("SQ_ACTIVE_INST_ANY", "active_any"),
                        ("SQ_ACTIVE_INST_VALU", "active_valu"), ("SQ_ACTIVE_INST_LDS", "active_lds"),
                        ("SQ_ACTIVE_INST_VMEM", "active_vmem")):
            if k in c:
                out[name + "_of_wave_cycles"] = round(c[k] / w, 4)
    return out


def sq_main(a):
    lines = [f"# SQ counters per launch, workload {a.workload}",
             "# rocprofv3 counter passes (one run each), from the repository root, TMPDIR=/tmp:"]
    lines += [f"#   {c}" for c in a.command]
    lines += ["# mfma_busy: SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x GRBM_GUI_ACTIVE / 8 XCDs);",
              "#   clock_ghz: GRBM_GUI_ACTIVE / 8 / duration (the shader clock the launch ran at);",
              "#   x_per_mfma: instructions of a class per MFMA instruction (VALU without the MFMAs);",
              "#   *_of_wave_cycles: SQ_WAIT_* / SQ_ACTIVE_INST_* over SQ_WAVE_CYCLES (resident wavefront cycles)"]
    recs = {}
    for k in a.kernel:
        c = sq_counters(a.csv, k)
        d = sq_derived(c)
        recs[k] = {"derived": d, "counters": {n: round(v, 1) for n, v in sorted(c.items())}}
        lines.append(f"# {k}: " + ", ".join(f"{n} {v}" for n, v in d.items()))
        lines.append(f"#   raw means per dispatch: " + ", ".join(f"{n} {v:.4g}" for n, v in sorted(c.items())))
    lines.append(f"# kernel sources hash {kernel_source_hash()}")
    lines.append(MARK.replace("traffic", "sq") + json.dumps({"workload": a.workload, "kernels": recs,
                                                             "sources": kernel_source_hash()}))
    with open(a.out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--sq", action="store_true", help="summarize SQ counter passes (--csv) instead of traffic")
    ap.add_argument("--csv", action="append", default=[])
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-fetch")
    ap.add_argument("--copy-write")
    ap.add_argument("--kernel", action="append", required=True)
    ap.add_argument("--workload", required=True)
    ap.add_argument("--out", required=True)
    ap.add_argument("--command", action="append", default=[], help="command lines that produced the csv files")
    a = ap.parse_args()
    if a.sq:
        if not a.csv:
            ap.error("--sq needs at least one --csv")
        return sq_main(a)
    if not (a.fetch and a.write and a.copy_fetch and a.copy_write) or len(a.kernel) != 1:
        ap.error("a traffic summary needs --fetch, --write, --copy-fetch, --copy-write and one --kernel")
    a.kernel = a.kernel[0]
    rec = summarize(a.fetch, a.write, a.copy_fetch, a.copy_write, a.kernel)
    rec["workload"] = a.workload
    lines = [f"# HBM traffic per launch of {a.kernel}, workload {a.workload}",
             "# rocprofv3 counter passes (one counter group per run), from the repository root, TMPDIR=/tmp:"]
    lines += [f"#   {c}" for c in a.command]
    lines += [f"# copy calibration: {COPY_KERNEL} of {COPY_BYTES >> 20} MiB reads {rec['copy_fetch_kib']} KiB "
              f"(FETCH_SIZE) and writes {rec['copy_write_kib']} KiB (WRITE_SIZE) per dispatch; "
              f"scales {rec['fetch_scale']} / {rec['write_scale']}",
              f"# kernel: {rec['fetch_kib']} KiB FETCH_SIZE, {rec['write_kib']} KiB WRITE_SIZE per dispatch "
              f"(mean of {rec['dispatches'][0]} / {rec['dispatches'][1]} dispatches)",
              f"# scaled HBM bytes per launch: read {rec['read_bytes'] / 1e9:.3f} GB, "
              f"written {rec['write_bytes'] / 1e9:.3f} GB, total {rec['traffic_bytes'] / 1e9:.3f} GB",
              f"# kernel sources hash {rec['sources']}",
              MARK + json.dumps(rec)]
    with open(a.out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


if __name__ == "__main__":
    main()
