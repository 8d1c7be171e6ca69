"""Summaries of rocprofv3 output for the committed profiles.

stats    kernel trace (``--kernel-trace --stats --output-format csv``, the
         per-dispatch ``*_kernel_trace.csv``) -> a short text table headed by
         the command that made it: per kernel, calls and time per run over the
         last N runs of the subgraph (the runs after the engine's autotune),
         and the per-run time of the conv/dense MFMA kernel class.
traffic  HBM bytes of the conv kernels per run from two counter runs
         (``--pmc FETCH_SIZE`` and ``--pmc WRITE_SIZE``, KiB per dispatch),
         each scaled by what the same counter reads for a plain device copy of
         known size (``bench.py --copy-calibration MIB`` under the same
         counter), over the last N runs -> JSON read by bench.py.

A run of the ResNet subgraph starts with its fused stem kernel (of its int8
form: the boundary quantize kernel), the marker used to split the dispatch
stream into runs.

Usage:
  python -m paper_2105_03215_amd.profiling stats --trace X_kernel_trace.csv \
      --cmd "<command>" --last-runs 60 --flops-per-run F --out profiles/NAME.txt
  python -m paper_2105_03215_amd.profiling traffic --fetch F.csv --write W.csv \
      --copy-fetch CF.csv --copy-write CW.csv --copy-mib 512 --last-runs 2 \
      --workload resnet50_v1_bs32 --out profiles/traffic.json
"""

import argparse
import csv
import hashlib
import json
import os
import statistics

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CONV_KERNELS = ("conv_mfma_kernel", "conv_dma_kernel", "conv_halo_kernel", "stem_conv_maxpool_kernel",
                "splitk_reduce_kernel", "dense_rows_kernel")
RUN_MARKER = "stem_conv_maxpool_kernel"  # one dispatch per run of the ResNet subgraphs


def _short(name):
    return name.replace("byoc::(anonymous namespace)::", "").replace("void ", "")


def _is_conv(name, kernels=CONV_KERNELS):
    return any(k in name for k in kernels)


def _last_runs(rows, name_key, last_runs, marker=RUN_MARKER):
    """The rows from the start of the last `last_runs` runs on."""
    starts = [i for i, r in enumerate(rows) if marker in r[name_key]]
    if len(starts) < last_runs:
        raise RuntimeError("only %d runs (marker %s) in the trace" % (len(starts), marker))
    return rows[starts[-last_runs]:], last_runs


def stats(trace_path, cmd, out, last_runs, flops_per_run=0.0, top=25, marker=RUN_MARKER,
          kernels=CONV_KERNELS, class_name="conv/dense MFMA class", unit="FLOP"):
    rows = sorted(csv.DictReader(open(trace_path)), key=lambda r: int(r["Start_Timestamp"]))
    rows, runs = _last_runs(rows, "Kernel_Name", last_runs, marker)
    per = {}
    for r in rows:
        d = per.setdefault(r["Kernel_Name"], [0, 0])
        d[0] += 1
        d[1] += int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    total = sum(v[1] for v in per.values())
    conv_ns = sum(v[1] for k, v in per.items() if _is_conv(k, kernels))
    conv_calls = sum(v[0] for k, v in per.items() if _is_conv(k, kernels))
    lines = ["# rocprofv3 kernel statistics (last %d runs of the subgraph, after autotune)" % runs,
             "# command: " + cmd,
             "# %-70s %9s %10s %12s %6s" % ("kernel", "calls/run", "avg_us", "us/run", "pct")]
    for k, (calls, ns) in sorted(per.items(), key=lambda kv: -kv[1][1])[:top]:
        lines.append("  %-70s %9.2f %10.2f %12.2f %6.2f" % (
            _short(k)[:70], calls / runs, ns / calls / 1e3, ns / runs / 1e3, 100.0 * ns / total))
    lines.append("# all kernels: %.1f us per run" % (total / runs / 1e3))
    lines.append("# %s (%s): %.1f launches, %.1f us per run, avg %.2f us per launch" % (
        class_name, ", ".join(kernels), conv_calls / runs, conv_ns / runs / 1e3, conv_ns / max(conv_calls, 1) / 1e3))
    if flops_per_run:
        lines.append("# %s: %.1f G%s per run -> %.1f T%s/s of pure kernel time" % (
            class_name, flops_per_run / 1e9, unit, flops_per_run / (conv_ns / runs * 1e-9) / 1e12, unit))
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    return out


def _counter(path, counter):
    per = {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        per[int(r["Dispatch_Id"])] = {"name": r["Kernel_Name"], "value": float(r["Counter_Value"])}
    return [per[k] for k in sorted(per)]


def _copy_kib(path, counter):
    vals = [d["value"] for d in _counter(path, counter) if "copy" in d["name"].lower()]
    if not vals:
        raise RuntimeError("no copy kernel in %s" % path)
    big = max(vals)
    return statistics.median([v for v in vals if v > 0.5 * big])


CONV_SOURCES = ("conv_mfma.hip", "conv_dma.hip", "conv_halo.hip", "lds_dma.h", "stem.hip", "dense_rows.hip",
                "engine.cpp")
I8_KERNELS = ("conv_i8_kernel",)
I8_SOURCES = ("conv_i8.hip", "quant.hip", "lds_dma.h", "engine.cpp")


def conv_kernel_digest(sources=CONV_SOURCES):
    """Digest of the conv kernel sources and of the planner that picks them."""
    h = hashlib.sha256()
    for name in sources:
        with open(os.path.join(ROOT, "paper_2105_03215_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic(fetch, write, copy_fetch, copy_write, copy_mib, workload, out, last_runs, marker=RUN_MARKER,
            kernels=CONV_KERNELS, sources=CONV_SOURCES):
    copy_bytes = copy_mib * 2 ** 20
    f_scale = copy_bytes / (_copy_kib(copy_fetch, "FETCH_SIZE") * 1024.0)
    w_scale = copy_bytes / (_copy_kib(copy_write, "WRITE_SIZE") * 1024.0)
    res = {}
    for name, path, counter, scale in (("fetch", fetch, "FETCH_SIZE", f_scale),
                                       ("write", write, "WRITE_SIZE", w_scale)):
        disp, runs = _last_runs(_counter(path, counter), "name", last_runs, marker)
        conv = sum(d["value"] for d in disp if _is_conv(d["name"], kernels))
        res[name] = conv * 1024.0 * scale / runs
        res[name + "_runs"] = runs
    doc = {"workload": workload, "conv_kernel_digest": conv_kernel_digest(sources),
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
    a.add_argument("--trace", required=True)
    a.add_argument("--cmd", required=True)
    a.add_argument("--out", required=True)
    a.add_argument("--last-runs", type=int, required=True)
    a.add_argument("--flops-per-run", type=float, default=0.0)
    a.add_argument("--marker", default=RUN_MARKER, help="kernel launched once per run of the subgraph")
    a.add_argument("--kernels", default=",".join(CONV_KERNELS), help="kernels of the summed class")
    a.add_argument("--class-name", default="conv/dense MFMA class")
    a.add_argument("--unit", default="FLOP", help="FLOP, or OP for integer work")
    b = sub.add_parser("traffic")
    for k in ("fetch", "write", "copy-fetch", "copy-write", "workload", "out"):
        b.add_argument("--" + k, required=True)
    b.add_argument("--copy-mib", type=int, required=True)
    b.add_argument("--last-runs", type=int, required=True)
    b.add_argument("--int8", action="store_true",
                   help="the int8 conv class (runs split at the boundary quantize kernel)")
    args = ap.parse_args()
    if args.cmd_name == "stats":
        print(stats(args.trace, args.cmd, args.out, args.last_runs, args.flops_per_run, marker=args.marker,
                    kernels=tuple(args.kernels.split(",")), class_name=args.class_name, unit=args.unit))
    else:
        kw = dict(marker="::quantize", kernels=I8_KERNELS, sources=I8_SOURCES) if args.int8 else {}
        print(json.dumps(traffic(args.fetch, args.write, args.copy_fetch, args.copy_write,
                                 args.copy_mib, args.workload, args.out, args.last_runs, **kw)))


if __name__ == "__main__":
    main()
