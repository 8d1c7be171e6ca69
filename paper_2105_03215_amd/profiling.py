"""Summaries of rocprofv3 output for the committed profiles.

stats    kernel-trace statistics (``--kernel-trace --stats --output-format
         csv``) -> a short text table headed by the command that made it.
traffic  HBM bytes of the conv kernels per step from two counter runs
         (``--pmc FETCH_SIZE`` and ``--pmc WRITE_SIZE``, KiB per dispatch),
         each scaled by what the same counter reads for a plain device copy of
         known size (``bench.py --copy-calibration MIB`` under the same
         counter) -> JSON read by bench.py.

Usage:
  python -m paper_2105_03215_amd.profiling stats --csv X_kernel_stats.csv \
      --cmd "<command>" --out profiles/NAME.txt
  python -m paper_2105_03215_amd.profiling traffic --fetch F.csv --write W.csv \
      --copy-fetch CF.csv --copy-write CW.csv --copy-mib 512 --workload resnet50_v1_bs32 \
      --out profiles/traffic.json
"""

import argparse
import csv
import hashlib
import json
import os
import statistics

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CONV_KERNELS = ("conv_mfma_kernel", "conv_dma_kernel", "splitk_reduce_kernel")
RUN_MARKER = "nchw_to_nhwc_kernel"  # one dispatch per run of the CNN subgraphs


def _short(name):
    return name.replace("byoc::(anonymous namespace)::", "").replace("void ", "")


def stats(csv_path, cmd, out, top=25):
    rows = list(csv.DictReader(open(csv_path)))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    lines = ["# rocprofv3 kernel statistics", "# command: " + cmd,
             "# %-70s %6s %12s %10s %6s" % ("kernel", "calls", "total_us", "avg_us", "pct")]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"]))[:top]:
        lines.append("  %-70s %6s %12.1f %10.2f %6.2f" % (
            _short(r["Name"])[:70], r["Calls"], float(r["TotalDurationNs"]) / 1e3,
            float(r["AverageNs"]) / 1e3, 100.0 * float(r["TotalDurationNs"]) / total))
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    return out


def _counter(path, counter):
    per = {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        per[int(r["Dispatch_Id"])] = (r["Kernel_Name"], float(r["Counter_Value"]))
    return [per[k] for k in sorted(per)]


def _copy_kib(path, counter):
    vals = [v for n, v in _counter(path, counter) if "copyBuffer" in n or "copy" in n.lower()]
    if not vals:
        raise RuntimeError("no copy kernel in %s" % path)
    big = max(vals)
    return statistics.median([v for v in vals if v > 0.5 * big])


def conv_kernel_digest():
    """Digest of the conv kernel sources and of the planner that picks them."""
    h = hashlib.sha256()
    for name in ("conv_mfma.hip", "conv_dma.hip", "engine.cpp"):
        with open(os.path.join(ROOT, "paper_2105_03215_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic(fetch, write, copy_fetch, copy_write, copy_mib, workload, out):
    copy_bytes = copy_mib * 2 ** 20
    f_scale = copy_bytes / (_copy_kib(copy_fetch, "FETCH_SIZE") * 1024.0)
    w_scale = copy_bytes / (_copy_kib(copy_write, "WRITE_SIZE") * 1024.0)
    res = {}
    for name, path, counter, scale in (("fetch", fetch, "FETCH_SIZE", f_scale),
                                       ("write", write, "WRITE_SIZE", w_scale)):
        disp = _counter(path, counter)
        runs = sum(1 for n, _ in disp if RUN_MARKER in n)
        conv = sum(v for n, v in disp if any(k in n for k in CONV_KERNELS))
        res[name] = conv * 1024.0 * scale / max(runs, 1)
        res[name + "_runs"] = runs
    doc = {"workload": workload, "conv_kernel_digest": conv_kernel_digest(),
           "conv_bytes_per_step": round(res["fetch"] + res["write"]),
           "conv_fetch_bytes_per_step": round(res["fetch"]),
           "conv_write_bytes_per_step": round(res["write"]),
           "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4),
           "copy_calibration_mib": copy_mib, "runs_counted": res["fetch_runs"],
           "counters": "FETCH_SIZE and WRITE_SIZE (KiB per dispatch), separate rocprofv3 runs"}
    with open(out, "w") as f:
        json.dump(doc, f, indent=1)
    return doc


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd_name", required=True)
    a = sub.add_parser("stats")
    a.add_argument("--csv", required=True)
    a.add_argument("--cmd", required=True)
    a.add_argument("--out", required=True)
    b = sub.add_parser("traffic")
    for k in ("fetch", "write", "copy-fetch", "copy-write", "workload", "out"):
        b.add_argument("--" + k, required=True)
    b.add_argument("--copy-mib", type=int, required=True)
    args = ap.parse_args()
    if args.cmd_name == "stats":
        print(stats(args.csv, args.cmd, args.out))
    else:
        print(json.dumps(traffic(args.fetch, args.write, args.copy_fetch, args.copy_write,
                                 args.copy_mib, args.workload, args.out)))


if __name__ == "__main__":
    main()
