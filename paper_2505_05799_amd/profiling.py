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


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--fetch", required=True)
    ap.add_argument("--write", required=True)
    ap.add_argument("--copy-fetch", required=True)
    ap.add_argument("--copy-write", required=True)
    ap.add_argument("--kernel", required=True)
    ap.add_argument("--workload", required=True)
    ap.add_argument("--out", required=True)
    ap.add_argument("--command", action="append", default=[], help="command lines that produced the csv files")
    a = ap.parse_args()
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
