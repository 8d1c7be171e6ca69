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

A run of the ResNet subgraph starts with its fused stem kernel, the marker
used to split the dispatch stream into runs; the int8 form's runs are cut at
its int8 stem.

classes  per kernel class of one workload: pure kernel time (kernel trace),
         HBM bytes read / written (FETCH_SIZE / WRITE_SIZE runs, scaled by a
         copy of known size), GB/s against 8 TB/s, and for the MFMA classes
         the MFMA busy fraction and the bf16 MFMA FLOPs issued -> JSON.
run      runs one workload's engine alone (autotuned, HIP-graph replay) for a
         kernel trace of it: the small configurations (single conv, ResNet-18
         block, batch-1 networks, BERT FFN) are cut into runs by their launch
         count (--launches-per-run) instead of a marker kernel.

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
                "splitk_reduce_kernel", "dense_rows_kernel", "bottleneck_kernel", "ir_block_kernel")
RUN_MARKER = "stem_conv_maxpool_kernel"  # one dispatch per run of the ResNet subgraphs
# kernels compiled for bf16 and for int8 codes: the int8 form has `true` as
# its last template argument
DUAL_KERNELS = ("bottleneck_kernel", "conv_halo_kernel", "stem_conv_maxpool_kernel")


def _short(name):
    return name.replace("byoc::(anonymous namespace)::", "").replace("void ", "")


def _is_int8(name):
    if "conv_i8_kernel" in name:
        return True
    if not any(k in name for k in DUAL_KERNELS):
        return False
    head = name.rsplit("(", 1)[0].rstrip("> ")
    return head.rsplit(",", 1)[-1].strip() == "true"


def _is_conv(name, kernels=CONV_KERNELS):
    """Is the kernel in the class of `kernels`?  A kernel of DUAL_KERNELS
    belongs to the int8 class (the one listing conv_i8_kernel) in its int8
    form and to the other class in its bf16 form."""
    if not any(k in name for k in kernels):
        return False
    return _is_int8(name) == ("conv_i8_kernel" in kernels)


def _last_runs(rows, name_key, last_runs, marker=RUN_MARKER, skip_last=0):
    """The rows of the last `last_runs` runs before the final `skip_last`
    runs (a run starts at its marker kernel, or is `marker` dispatches long
    when the marker is a number)."""
    if isinstance(marker, int):
        end = len(rows) - skip_last * marker
        if end - last_runs * marker < 0:
            raise RuntimeError("only %d dispatches in the trace" % len(rows))
        return rows[end - last_runs * marker:end], last_runs
    hit = marker if callable(marker) else (lambda n: marker in n)
    starts = [i for i, r in enumerate(rows) if hit(r[name_key])]
    if len(starts) < last_runs + skip_last:
        raise RuntimeError("only %d runs (marker %s) in the trace" % (len(starts), getattr(marker, "__name__", marker)))
    end = starts[len(starts) - skip_last] if skip_last else len(rows)
    return rows[starts[len(starts) - skip_last - last_runs]:end], last_runs


def stats(trace_path, cmd, out, last_runs, flops_per_run=0.0, top=25, marker=RUN_MARKER,
          kernels=CONV_KERNELS, class_name="conv/dense MFMA class", unit="FLOP", skip_last=0):
    rows = sorted(csv.DictReader(open(trace_path)), key=lambda r: int(r["Start_Timestamp"]))
    rows, runs = _last_runs(rows, "Kernel_Name", last_runs, marker, skip_last)
    per = {}
    for r in rows:
        d = per.setdefault(r["Kernel_Name"], [0, 0])
        d[0] += 1
        d[1] += int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    total = sum(v[1] for v in per.values())
    conv_ns = sum(v[1] for k, v in per.items() if _is_conv(k, kernels))
    conv_calls = sum(v[0] for k, v in per.items() if _is_conv(k, kernels))
    lines = ["# rocprofv3 kernel statistics (%d runs of the subgraph after autotune%s)" % (
                 runs, ", before the last %d" % skip_last if skip_last else ", the last ones"),
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


CONV_SOURCES = ("conv_mfma.hip", "conv_dma.hip", "conv_halo.hip", "bottleneck.hip", "ir_block.hip", "lds_dma.h",
                "stem.hip", "dense_rows.hip", "engine.cpp")
I8_KERNELS = ("conv_i8_kernel", "bottleneck_kernel", "conv_halo_kernel", "stem_conv_maxpool_kernel")
I8_SOURCES = ("conv_i8.hip", "conv_halo.hip", "bottleneck.hip", "stem.hip", "quant.hip", "quant_epilogue.h", "lds_dma.h",
              "engine.cpp")


def I8_MARKER(name):  # a run of an int8 ResNet starts at its int8 stem
    return "stem_conv_maxpool_kernel" in name and _is_int8(name)


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


KERNEL_CLASSES = {
    "conv/dense bf16 MFMA": CONV_KERNELS,
    "conv int8 MFMA": I8_KERNELS,
    "depthwise": ("depthwise3x3_kernel", "depthwise_kernel", "depthwise_i8_kernel"),
    "pooling": ("maxpool_nhwc_kernel", "avgpool_nhwc_kernel", "avgpool_win_nhwc_kernel", "maxpool_i8_kernel",
                "avgpool_i8_kernel"),
    "add": ("add_bf16_kernel", "add_i8_kernel"),
    "boundary transform": ("nchw_to_nhwc_kernel", "nhwc_to_nchw_kernel", "rows_to_padded_kernel",
                           "padded_to_rows_kernel", "cast_kernel", "quantize_kernel", "dequantize_kernel",
                           "quantize_im2col_kernel"),
    "fp32 conv": ("conv_f32_kernel", "conv_f32_regs_kernel"),
}


def _class_of(name):
    for cls, ks in KERNEL_CLASSES.items():
        if _is_conv(name, ks):
            return cls
    return None


def _rows_by_dispatch(path):
    """{dispatch id: {"name": kernel, counter: value, ...}} of a counter CSV."""
    per = {}
    for r in csv.DictReader(open(path)):
        d = per.setdefault(int(r["Dispatch_Id"]), {"name": r["Kernel_Name"]})
        d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return [per[k] for k in sorted(per)]


CLOCK_GHZ = 2.4   # peak engine clock
SIMDS = 1024      # 256 CUs x 4


def class_counters(trace, fetch, write, mfma, copy_fetch, copy_write, copy_mib, last_runs, marker, workload, cmd,
                   out, alg_bytes=None, alg_flops=None, trace_runs=20, trace_skip_last=0):
    """Per kernel class and run: pure kernel time (kernel trace: the
    `trace_runs` runs before the final `trace_skip_last`), HBM bytes read
    and written (FETCH_SIZE, WRITE_SIZE of the last `last_runs` runs, scaled
    by a copy of known size), achieved GB/s against 8 TB/s, and for the
    MFMA classes the bf16 MFMA FLOPs issued (SQ_INSTS_VALU_MFMA_MOPS_BF16 x
    512) and the MFMA busy fraction: SQ_VALU_MFMA_BUSY_CYCLES (summed over
    the SIMDs) over the class's kernel time x 1024 SIMDs x 2.4 GHz."""
    rows = sorted(csv.DictReader(open(trace)), key=lambda r: int(r["Start_Timestamp"]))
    rows, runs = _last_runs(rows, "Kernel_Name", trace_runs, marker, trace_skip_last)
    res = {}
    for r in rows:
        cls = _class_of(r["Kernel_Name"])
        if cls is None:
            continue
        d = res.setdefault(cls, {"launches": 0, "ns": 0})
        d["launches"] += 1
        d["ns"] += int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    f_scale = copy_mib * 2 ** 20 / (_copy_kib(copy_fetch, "FETCH_SIZE") * 1024.0)
    w_scale = copy_mib * 2 ** 20 / (_copy_kib(copy_write, "WRITE_SIZE") * 1024.0)
    for path, counter, scale, key in ((fetch, "FETCH_SIZE", f_scale, "fetch_bytes"),
                                      (write, "WRITE_SIZE", w_scale, "write_bytes")):
        disp, nr = _last_runs(_rows_by_dispatch(path), "name", last_runs, marker)
        for d in disp:
            cls = _class_of(d["name"])
            if cls in res:
                res[cls][key] = res[cls].get(key, 0.0) + d.get(counter, 0.0) * 1024.0 * scale / nr
    if mfma:
        disp, nr = _last_runs(_rows_by_dispatch(mfma), "name", last_runs, marker)
        for d in disp:
            cls = _class_of(d["name"])
            if cls in res:
                c = res[cls]
                c["mfma_busy"] = c.get("mfma_busy", 0.0) + d.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / nr
                c["mfma_bf16_flops"] = c.get("mfma_bf16_flops", 0.0) + d.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) * 512 / nr
    doc = {"workload": workload, "command": cmd, "trace_runs": runs, "counter_runs": last_runs,
           "copy_calibration_mib": copy_mib, "clock_ghz_assumed": CLOCK_GHZ,
           "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4), "classes": {}}
    for cls, c in res.items():
        us = c["ns"] / runs / 1e3
        e = {"launches_per_run": c["launches"] / runs, "us_per_run": round(us, 2)}
        if "fetch_bytes" in c or "write_bytes" in c:
            b = c.get("fetch_bytes", 0.0) + c.get("write_bytes", 0.0)
            e.update({"hbm_read_bytes": round(c.get("fetch_bytes", 0.0)), "hbm_write_bytes": round(c.get("write_bytes", 0.0)),
                      "hbm_gbs": round(b / (us * 1e-6) / 1e9, 1), "hbm_frac_of_8tbs": round(b / (us * 1e-6) / 8e12, 4)})
        if alg_bytes and cls in alg_bytes:
            e["algorithmic_bytes"] = alg_bytes[cls]
            e["algorithmic_gbs"] = round(alg_bytes[cls] / (us * 1e-6) / 1e9, 1)
        if c.get("mfma_bf16_flops", 0.0) > 0:
            e["mfma_busy_frac"] = round(c["mfma_busy"] / (us * 1e3 * CLOCK_GHZ * SIMDS), 4)
            e["mfma_bf16_flops_issued"] = round(c["mfma_bf16_flops"])
            e["mfma_bf16_tflops_issued"] = round(c["mfma_bf16_flops"] / (us * 1e-6) / 1e12, 1)
            e["mfma_bf16_frac_of_peak"] = round(c["mfma_bf16_flops"] / (us * 1e-6) / 2516.6e12, 4)
        if alg_flops and cls in alg_flops:
            e["algorithmic_flops"] = alg_flops[cls]
        doc["classes"][cls] = e
    with open(out, "w") as f:
        json.dump(doc, f, indent=1)
    return doc


def run_workload(name, batch, runs, warmup, autotune=True):
    """One workload's engine alone: autotune (unless off), `warmup` runs,
    then `runs` HIP-graph replays, nothing after them (so the trace ends
    with them)."""
    import torch

    from . import capi, runtime, workloads

    wl = workloads.build(name, **({("batch" if name == "bert_ffn" else "n"): batch} if batch else {}))
    sg = capi.Subgraph(wl.graph, wl.consts, device=0)
    try:
        dev = "cuda:0"
        s = torch.cuda.Stream(device=dev)
        ins = runtime.inputs_for(sg, wl.inputs, dev)
        outs = runtime.outputs_for(sg, dev)
        torch.cuda.synchronize()
        sg.set_options(autotune=autotune, graph_replay=True)
        for _ in range(warmup):
            sg.run(ins, outs, s)
        s.synchronize()
        for _ in range(runs):
            sg.run(ins, outs, s)
        s.synchronize()
        launches = sg.launches()
    finally:
        sg.close()
    return {"workload": name, "batch": batch, "runs": runs, "launches_per_run": len(launches),
            "flops_per_run": sum(l["flops"] for l in launches), "launches": [l["name"] for l in launches]}


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd_name", required=True)
    r = sub.add_parser("run", help="run one workload's engine alone (for a kernel trace)")
    r.add_argument("--workload", required=True)
    r.add_argument("--batch", type=int, default=0, help="batch size (networks); 0: the workload's default")
    r.add_argument("--runs", type=int, default=50)
    r.add_argument("--warmup", type=int, default=10)
    r.add_argument("--no-autotune", action="store_true", help="keep the built-in (or forced) kernel choice")
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
    a.add_argument("--skip-last", type=int, default=0, help="runs at the end of the trace to leave out")
    a.add_argument("--int8", action="store_true", help="the int8 MFMA class, runs cut at the int8 stem")
    a.add_argument("--launches-per-run", type=int, default=0,
                   help="cut runs by their dispatch count instead of the marker kernel")
    b = sub.add_parser("traffic")
    for k in ("fetch", "write", "copy-fetch", "copy-write", "workload", "out"):
        b.add_argument("--" + k, required=True)
    b.add_argument("--copy-mib", type=int, required=True)
    b.add_argument("--last-runs", type=int, required=True)
    b.add_argument("--int8", action="store_true",
                   help="the int8 conv class (runs split at the boundary quantize kernel)")
    c = sub.add_parser("classes", help="per-class time, HBM bytes and MFMA utilisation of one workload")
    for k in ("trace", "fetch", "write", "copy-fetch", "copy-write", "workload", "cmd", "out"):
        c.add_argument("--" + k, required=True)
    c.add_argument("--mfma", default=None, help="counter CSV of SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE, "
                                                "SQ_INSTS_VALU_MFMA_MOPS_BF16")
    c.add_argument("--copy-mib", type=int, required=True)
    c.add_argument("--last-runs", type=int, required=True)
    c.add_argument("--marker", default=RUN_MARKER)
    c.add_argument("--launches-per-run", type=int, default=0,
                   help="cut runs by their dispatch count instead of the marker kernel")
    c.add_argument("--trace-runs", type=int, default=20)
    c.add_argument("--trace-skip-last", type=int, default=0,
                   help="runs at the end of the trace to leave out (the bench's per-launch-event profile runs)")
    c.add_argument("--launches-json", default=None,
                   help="bench --dump-launches table: algorithmic bytes and flops per class")
    args = ap.parse_args()
    if args.cmd_name == "run":
        print(json.dumps(run_workload(args.workload, args.batch, args.runs, args.warmup, not args.no_autotune)),
              flush=True)
        return
    if args.cmd_name in ("stats", "classes") and args.launches_per_run > 0:
        args.marker = args.launches_per_run
    if args.cmd_name == "classes":
        alg_b = alg_f = None
        if args.launches_json:
            kinds = {"conv_mfma": "conv/dense bf16 MFMA", "reduce": "conv/dense bf16 MFMA", "conv_i8": "conv int8 MFMA",
                     "depthwise": "depthwise", "maxpool": "pooling", "avgpool": "pooling", "add": "add",
                     "transform": "boundary transform", "conv_f32": "fp32 conv"}
            alg_b, alg_f = {}, {}
            for l in json.load(open(args.launches_json)):
                k = kinds.get(l["kind"])
                if k:
                    alg_b[k] = alg_b.get(k, 0) + l["bytes"]
                    alg_f[k] = alg_f.get(k, 0) + l["flops"]
        print(json.dumps(class_counters(args.trace, args.fetch, args.write, args.mfma, args.copy_fetch,
                                        args.copy_write, args.copy_mib, args.last_runs, args.marker, args.workload,
                                        args.cmd, args.out, alg_b, alg_f, args.trace_runs, args.trace_skip_last),
                         indent=1))
        return
    if args.cmd_name == "stats":
        marker, kernels = (I8_MARKER, I8_KERNELS) if args.int8 else (args.marker, tuple(args.kernels.split(",")))
        print(stats(args.trace, args.cmd, args.out, args.last_runs, args.flops_per_run, marker=marker,
                    kernels=kernels, class_name=args.class_name, unit=args.unit, skip_last=args.skip_last))
    else:
        kw = dict(marker=I8_MARKER, kernels=I8_KERNELS, sources=I8_SOURCES) if args.int8 else {}
        print(json.dumps(traffic(args.fetch, args.write, args.copy_fetch, args.copy_write,
                                 args.copy_mib, args.workload, args.out, args.last_runs, **kw)))


if __name__ == "__main__":
    main()
