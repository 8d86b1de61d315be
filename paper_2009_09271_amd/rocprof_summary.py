"""Short text summaries of rocprofv3 CSV output, for the files under profiles/.

    python -m paper_2009_09271_amd.rocprof_summary stats <kernel_stats.csv> --out F --command CMD
    python -m paper_2009_09271_amd.rocprof_summary pmc <fetch counter_collection.csv>
        <write counter_collection.csv> --kernel NAME --calib NAME --calib-bytes B --alg-bytes A
        --out F --command CMD [--command2 CMD2]

`stats` tabulates every kernel's launch count and average / min / max duration.  `pmc` turns
FETCH_SIZE and WRITE_SIZE (KiB per dispatch, one rocprofv3 run each) into HBM bytes per launch of
one kernel, scaled by what the same counters read for a plain copy kernel of known size
(`--calib`, moving `--calib-bytes` in each direction per launch).  It records a hash of the kernel
sources so that a stale measurement can be recognised.
"""

from __future__ import annotations

import argparse
import csv
import hashlib
import os
import statistics
import sys

_HERE = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCES = [os.path.join(_HERE, "csrc", "ef_kernels.h"), os.path.join(_HERE, "csrc", "ef_device.h")]


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def short_name(name: str) -> str:
    n = name.replace("void ", "").replace("efs::", "")
    for cut in ("(Tables", "(int", "(efs", "(unsigned"):
        if cut in n:
            n = n.split(cut)[0]
    n = n.strip()
    if len(n) > 72:  # library kernels of other components (PyTorch fills and RNG): keep them short
        n = n[:69] + "..."
    return n


def stats(path, out, command):
    rows = list(csv.DictReader(open(path)))
    lines = ["# rocprofv3 kernel statistics", "", "Command (from the repository root):", "", "```",
             command, "```", "", f"Kernel sources hash: `{kernel_source_hash()}`", "",
             "| kernel | launches | avg us | min us | max us | share of GPU time |",
             "|---|---:|---:|---:|---:|---:|"]
    for r in rows:
        lines.append(f"| `{short_name(r['Name'])}` | {int(r['Calls'])} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                     f"{float(r['Percentage']):.1f} % |")
    text = "\n".join(lines) + "\n"
    with open(out, "w") as f:
        f.write(text)
    print(text)


def _counter_avg(path, counter):
    """Average counter value per dispatch, per kernel short name."""
    per = {}
    for r in csv.DictReader(open(path)):
        if r.get("Counter_Name") != counter:
            continue
        per.setdefault(short_name(r["Kernel_Name"]), []).append(float(r["Counter_Value"]))
    return {k: (statistics.fmean(v), len(v)) for k, v in per.items()}


def pmc(fetch_csv, write_csv, kernel, calib, calib_bytes, alg_bytes, out, command, command2):
    fe = _counter_avg(fetch_csv, "FETCH_SIZE")
    wr = _counter_avg(write_csv, "WRITE_SIZE")
    for need in (kernel, calib):
        if need not in fe or need not in wr:
            sys.exit(f"kernel {need!r} missing from the counter files (have {sorted(fe)})")
    kib = 1024.0
    f_scale = calib_bytes / (fe[calib][0] * kib)
    w_scale = calib_bytes / (wr[calib][0] * kib)
    fetch_b = fe[kernel][0] * kib * f_scale
    write_b = wr[kernel][0] * kib * w_scale
    traffic = fetch_b + write_b
    lines = ["# HBM traffic from rocprofv3 counters", "",
             "FETCH_SIZE run (from the repository root):", "", "```", command, "```", "",
             "WRITE_SIZE run:", "", "```", command2, "```", "",
             f"Kernel sources hash: `{kernel_source_hash()}`", "",
             "| kernel | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB |", "|---|---:|---:|---:|"]
    for k in sorted(set(fe) | set(wr)):
        fv = f"{fe[k][0]:.0f}" if k in fe else "-"
        wv = f"{wr[k][0]:.0f}" if k in wr else "-"
        n = fe[k][1] if k in fe else wr[k][1]
        lines.append(f"| `{k}` | {n} | {fv} | {wv} |")
    lines += ["", f"Calibration: `{calib}` moves {calib_bytes} bytes each way per launch; the counters read "
              f"{fe[calib][0] * kib:.0f} fetched and {wr[calib][0] * kib:.0f} written bytes, scale factors "
              f"{f_scale:.4f} (fetch) and {w_scale:.4f} (write).", "",
              f"`{kernel}`: {fetch_b:.0f} bytes fetched + {write_b:.0f} bytes written = {traffic:.0f} bytes per "
              f"launch (scaled); algorithmic bytes per launch {alg_bytes}; ratio {traffic / alg_bytes:.4f}.", "",
              f"traffic_bytes_per_launch: {traffic:.0f}", f"kernel: {kernel}"]
    text = "\n".join(lines) + "\n"
    with open(out, "w") as f:
        f.write(text)
    print(text)


def read_traffic(path, kernel):
    """Scaled HBM bytes per launch of the kernel whose name starts with `kernel` from a `pmc`
    summary, or None when the summary is missing, is for another kernel, or was taken on
    different kernel sources."""
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if line.startswith("Kernel sources hash:"):
            vals["hash"] = line.split("`")[1]
        elif ":" in line and line.split(":")[0] in ("traffic_bytes_per_launch", "kernel"):
            k, v = line.split(":", 1)
            vals[k] = v.strip()
    if vals.get("hash") != kernel_source_hash() or not vals.get("kernel", "").startswith(kernel):
        return None
    try:
        return float(vals["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("stats")
    a.add_argument("csv")
    a.add_argument("--out", required=True)
    a.add_argument("--command", required=True)
    b = sub.add_parser("pmc")
    b.add_argument("fetch_csv")
    b.add_argument("write_csv")
    b.add_argument("--kernel", required=True)
    b.add_argument("--calib", required=True)
    b.add_argument("--calib-bytes", type=float, required=True)
    b.add_argument("--alg-bytes", type=float, required=True)
    b.add_argument("--out", required=True)
    b.add_argument("--command", required=True)
    b.add_argument("--command2", required=True)
    args = ap.parse_args()
    if args.cmd == "stats":
        stats(args.csv, args.out, args.command)
    else:
        pmc(args.fetch_csv, args.write_csv, args.kernel, args.calib, args.calib_bytes, args.alg_bytes, args.out,
            args.command, args.command2)


if __name__ == "__main__":
    main()
