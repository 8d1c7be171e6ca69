"""Throughput of offloaded subgraphs on one MI355X.

One step = one run of the whole offloaded subgraph over one batch of
synthetic input already resident in HBM.  The headline is ResNet-50 v1 at
batch 32 (input layout transform, 53 conv composites, max-pool, global
average pool, classifier); the line also carries the other workloads the
method is measured on, each timed the same way (engine autotune on, the
launch sequence on a side stream both as direct launches and as HIP-graph
replay, the faster mode reported):

  configs      the single fp32 conv composite (us per call), the ResNet-18
               basic block (us per block), ResNet-50 at batch 1, MobileNetV2
               at batch 1 and 16 (depthwise / pooling HBM GB/s), the
               BERT-base-shaped FFN stack (tokens/s, fraction of MFMA peak);
  timing       warm (back-to-back) and cold (a 512 MiB buffer written before
               every run, evicting L2 and the 256 MB MALL) per-step times of
               the headline, median / p10 / p90;
  roofline     the dominant kernel class (the bf16 MFMA conv/dense kernels)
               from per-launch HIP events on the run stream;
  partitioned  the network as an operator-level model through the
               partitioner and the partitioned-model runtime;
  quantized    the network partially quantized to int8;
  other_workloads  VGG19, DarkNet-53, Inception V3 at batch 32;
  cpu_baseline the oracle timed on this host on the headline workload; the
               same leg also evaluates the oracle on every timed workload
               (sampled for the large ones) and reports each one's parity
               error next to its tolerance.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "images/sec (bs1, bs32) ResNet-50 offloaded subgraph; conv TFLOP/s as % MFMA peak"
PEAK_BF16_TFLOPS = 2516.6  # dense bf16 MFMA: 256 CU x 2.4 GHz x 4096 FLOP/clk
PEAK_F32_TFLOPS = 157.3    # fp32 (vector / MFMA)
PEAK_INT8_TOPS = 5033.2    # dense int8 MFMA: 256 CU x 2.4 GHz x 8192 OP/clk
PEAK_HBM_GBS = 8000.0
BF16_TOL, F32_TOL = 1e-2, 1e-4
EVICT_MIB = 512            # > the 256 MB MALL plus every L2


def _pct(xs):
    import numpy as np
    a = np.asarray(xs, dtype=np.float64)
    return {"median": round(float(np.median(a)), 5), "p10": round(float(np.percentile(a, 10)), 5),
            "p90": round(float(np.percentile(a, 90)), 5), "n": int(a.size)}


def _timed_runs(sg, ins, outs, stream, steps):
    """Mean ms per run over `steps` back-to-back runs, one HIP event pair on
    the run stream around all of them (the contract's K timed steps)."""
    import torch
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    with torch.cuda.stream(stream):
        start.record(stream)
        for _ in range(steps):
            sg.run(ins, outs, stream)
        end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return start.elapsed_time(end) / steps, wall


def _per_step(sg, ins, outs, stream, steps, evict=None):
    """ms of each run from its own event pair on the run stream; with
    `evict`, that buffer is overwritten on the run stream before every run,
    outside the pair (cold caches)."""
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for a, b in evs:
            if evict is not None:
                evict.fill_(1.0)
            a.record(stream)
            sg.run(ins, outs, stream)
            b.record(stream)
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in evs]


def _grouped(sg, ins, outs, stream, groups, per_group):
    """ms per run for latency-bound engines: `groups` event pairs around
    `per_group` back-to-back runs each."""
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(groups)]
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for a, b in evs:
            a.record(stream)
            for _ in range(per_group):
                sg.run(ins, outs, stream)
            b.record(stream)
    torch.cuda.synchronize()
    return [a.elapsed_time(b) / per_group for a, b in evs]


def _profile(sg, ins, outs, stream, steps):
    """Per-launch durations (ms per run) from HIP events recorded by the
    library on the run stream around every launch."""
    import torch
    sg.profile_begin(steps)
    for _ in range(steps):
        sg.run(ins, outs, stream)
    ms, runs = sg.profile_end()
    torch.cuda.synchronize()
    return [m / max(runs, 1) for m in ms], runs


def _roofline(launches, per_launch_ms, step_ms, traffic=None):
    """Roofline of the conv/dense MFMA class.  Its time per step is the
    timed step (HIP events around the timed steps) less the other
    kernels' per-launch event times: per-launch events add a gap of their
    own to every launch, the step time only the launches' own gaps."""
    conv_kinds = ("conv_mfma", "reduce")
    conv_ev_ms = sum(t for l, t in zip(launches, per_launch_ms) if l["kind"] in conv_kinds)
    other_ms = sum(t for l, t in zip(launches, per_launch_ms) if l["kind"] not in conv_kinds)
    conv_ms = max(step_ms - other_ms, 1e-9)
    conv_flops = sum(l["flops"] for l in launches if l["kind"] == "conv_mfma")
    n_conv = sum(1 for l in launches if l["kind"] == "conv_mfma")
    achieved = conv_flops / (conv_ms * 1e-3) / 1e12
    # per-layer floor: each conv launch at its own roofline, max(flops / MFMA
    # peak, algorithmic bytes / HBM peak); the 1x1 layers are HBM-bound, so
    # the whole class cannot reach the MFMA peak
    floor_ms = sum(max(l["flops"] / (PEAK_BF16_TFLOPS * 1e12), l["bytes"] / (PEAK_HBM_GBS * 1e9)) * 1e3
                   for l in launches if l["kind"] == "conv_mfma")
    return {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic,
            "kernel": ("conv/dense bf16 MFMA class (stem_conv_maxpool, conv_dma, conv_halo, conv_mfma, bottleneck, ir_block, dense_rows, "
                       "splitk_reduce kernels), %d launches per step" % n_conv),
            "flops_per_step": conv_flops, "kernel_ms_per_step": round(conv_ms, 4),
            "per_launch_event_ms_per_step": round(conv_ev_ms, 4),
            "per_launch_event_frac": round(conv_flops / (conv_ev_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)
            if conv_ev_ms > 0 else None,
            "layer_floor_ms_per_step": round(floor_ms, 4),
            "frac_of_layer_floor": round(floor_ms / conv_ms, 4)}


def _class_summary(launches, per_launch_ms):
    """Per kernel class: launches, ms per run, algorithmic bytes and flops,
    and the achieved rates against the HBM and bf16 MFMA peaks."""
    out = {}
    for l, t in zip(launches, per_launch_ms):
        d = out.setdefault(l["kind"], {"launches": 0, "ms": 0.0, "flops": 0, "bytes": 0})
        d["launches"] += 1
        d["ms"] += t
        d["flops"] += l["flops"]
        d["bytes"] += l["bytes"]
    for d in out.values():
        d["ms"] = round(d["ms"], 4)
        d["gbs"] = round(d["bytes"] / (d["ms"] * 1e-3) / 1e9, 1) if d["ms"] > 0 else None
        d["hbm_frac"] = round(d["gbs"] / PEAK_HBM_GBS, 4) if d["gbs"] else None
        d["tflops"] = round(d["flops"] / (d["ms"] * 1e-3) / 1e12, 2) if d["ms"] > 0 else None
    return out


def _conv_kernel_digest():
    """Digest of the conv kernel sources and their planner: stored traffic
    counts apply only to the kernels they were measured on."""
    from paper_2105_03215_amd import profiling
    return profiling.conv_kernel_digest()


def _copy_calibration(mib):
    """A plain device-to-device copy of known size (for scaling the HBM
    byte counters): three copies of `mib` MiB."""
    import torch
    n = mib * 2 ** 20 // 4
    a = torch.empty(n, dtype=torch.float32, device="cuda:0").fill_(1.0)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()


class Measured:
    """One workload as the benchmark runs it: engine, autotune, the faster
    launch mode on the run stream, timing, per-launch profile and the host copy of the
    outputs of the timed configuration (for the parity report)."""

    def __init__(self, key, wl, sg, ms, launches, per_launch, outputs):
        self.key, self.wl, self.ms = key, wl, ms
        self.launches, self.per_launch, self.outputs = launches, per_launch, outputs


def _measure(args, key, wl, dev, stream, timing="steps", graph=None, consts=None):
    """Create the engine, tune it, time it, profile it, keep its outputs.
    timing: "steps" (one event pair around args.steps runs), "grouped"
    (20 pairs around 100 runs each: latency-bound engines)."""
    import torch

    from paper_2105_03215_amd import capi, runtime

    sg = capi.Subgraph(graph or wl.graph, consts or wl.consts, device=0)
    try:
        ins = runtime.inputs_for(sg, wl.inputs, dev)
        outs = runtime.outputs_for(sg, dev)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        if not args.no_autotune:
            sg.set_options(autotune=True)
        tune_s = time.perf_counter() - t0
        res = {"tune_s": round(tune_s, 3)}
        if timing == "grouped":
            # latency-bound engines: direct launches and graph replay both
            # timed (a graph launch costs more host time than a few direct
            # launches); the faster one is the engine's figure
            modes = [("direct launches", False)] + ([] if args.eager else [("HIP graph replay", True)])
            best = None
            for label, replay in modes:
                sg.set_options(graph_replay=replay)
                for _ in range(args.warmup):
                    sg.run(ins, outs, stream)
                torch.cuda.synchronize()
                st = _pct(_grouped(sg, ins, outs, stream, 20, 100))
                res["ms_" + ("graph" if replay else "direct")] = st
                if best is None or st["median"] < best[1]["median"]:
                    best = (label, st, replay)
            sg.set_options(graph_replay=best[2])
            res["ms"], res["launch_mode"] = best[1], best[0]
            ms = res["ms"]["median"]
        else:
            # throughput engines: the K steps timed in both modes, as the
            # headline is
            best = None
            for label, replay in [("direct launches", False)] + ([] if args.eager else [("HIP graph replay", True)]):
                sg.set_options(graph_replay=replay)
                for _ in range(args.warmup):
                    sg.run(ins, outs, stream)
                torch.cuda.synchronize()
                t_ms, _ = _timed_runs(sg, ins, outs, stream, args.steps)
                res["ms_" + ("graph" if replay else "direct")] = round(t_ms, 4)
                if best is None or t_ms < best[0]:
                    best = (t_ms, label, replay)
            sg.set_options(graph_replay=best[2])
            ms, res["launch_mode"] = best[0], best[1]
        host = [runtime.to_host_f64(o) for o in outs]
        sg.set_options(graph_replay=False)
        launches = sg.launches()
        per_launch, _ = _profile(sg, ins, outs, stream, min(args.steps, 20))
    finally:
        sg.close()
    m = Measured(key, wl, None, ms, launches, per_launch, host)
    m.extra = res
    return m


def _config_lines(args, dev, stream):
    """configs[0], [1], [3], [4] of the benchmark set and ResNet-50 batch 1:
    the latency-bound ones as us per call (median of 20 groups of 100 runs),
    the others as throughput; each with its kernel classes."""
    from paper_2105_03215_amd import workloads

    out, measured = {}, []

    m = _measure(args, "conv_f32", workloads.build("conv_f32"), dev, stream, timing="grouped")
    measured.append(m)
    fl = sum(l["flops"] for l in m.launches)
    out["conv_f32"] = {
        "config": "single conv2d 3x3 + bias + ReLU, fp32, 1x16x32x32 -> 32 channels",
        "us_per_call": round(m.ms * 1e3, 2), "us_per_call_p10_p90": [round(m.extra["ms"]["p10"] * 1e3, 2),
                                                                      round(m.extra["ms"]["p90"] * 1e3, 2)],
        "gflops": round(fl / (m.ms * 1e-3) / 1e9, 2), "dtype": "f32",
        "roofline": {"bound": "launch latency", "note": "%.1f MFLOP: %.3f us at the fp32 peak of %.1f TFLOP/s"
                     % (fl / 1e6, fl / (PEAK_F32_TFLOPS * 1e12) * 1e6, PEAK_F32_TFLOPS)},
        "launch_mode": m.extra["launch_mode"], "us_direct": round(m.extra["ms_direct"]["median"] * 1e3, 2),
        "us_graph": round(m.extra["ms_graph"]["median"] * 1e3, 2) if "ms_graph" in m.extra else None,
        "launches": len(m.launches)}

    m = _measure(args, "resnet18_block", workloads.build("resnet18_block"), dev, stream, timing="grouped")
    measured.append(m)
    fl = sum(l["flops"] for l in m.launches)
    tf = fl / (m.ms * 1e-3) / 1e12
    out["resnet18_block"] = {
        "config": "ResNet-18 basic block, bf16, 1x64x56x56 (conv3x3+bias+ReLU, conv3x3+bias+residual+ReLU)",
        "us_per_block": round(m.ms * 1e3, 2), "us_p10_p90": [round(m.extra["ms"]["p10"] * 1e3, 2),
                                                             round(m.extra["ms"]["p90"] * 1e3, 2)],
        "tflops": round(tf, 2), "mfma_frac": round(tf / PEAK_BF16_TFLOPS, 4), "launches": len(m.launches),
        "launch_mode": m.extra["launch_mode"], "us_direct": round(m.extra["ms_direct"]["median"] * 1e3, 2),
        "us_graph": round(m.extra["ms_graph"]["median"] * 1e3, 2) if "ms_graph" in m.extra else None,
        "kernel_classes": _class_summary(m.launches, m.per_launch)}

    if not args.no_bs1 and not (args.variant == "resnet50_v1" and args.batch == 1):
        m = _measure(args, "resnet50_v1_bs1", workloads.build("resnet50_v1", n=1), dev, stream, timing="grouped")
        measured.append(m)
        fl = sum(l["flops"] for l in m.launches if l["kind"] == "conv_mfma")
        out["resnet50_v1_bs1"] = {
            "images_per_s": round(1.0 / (m.ms * 1e-3), 1), "ms_per_step": round(m.ms, 4),
            "ms_p10_p90": [m.extra["ms"]["p10"], m.extra["ms"]["p90"]],
            "conv_tflops": round(fl / (m.ms * 1e-3) / 1e12, 2), "launches": len(m.launches),
            "launch_mode": m.extra["launch_mode"],
            "ms_direct": m.extra["ms_direct"]["median"], "ms_graph": m.extra.get("ms_graph", {}).get("median")}

    for n in (1, 16):
        m = _measure(args, "mobilenet_v2_bs%d" % n, workloads.build("mobilenet_v2", n=n), dev, stream,
                     timing="grouped" if n == 1 else "steps")
        measured.append(m)
        cls = _class_summary(m.launches, m.per_launch)
        fl = sum(l["flops"] for l in m.launches if l["kind"] == "conv_mfma")
        out["mobilenet_v2_bs%d" % n] = {
            "images_per_s": round(n / (m.ms * 1e-3), 1), "ms_per_step": round(m.ms, 4),
            "conv_tflops": round(fl / (m.ms * 1e-3) / 1e12, 2), "launches": len(m.launches),
            "launch_mode": m.extra["launch_mode"],
            "depthwise": ({k: cls["depthwise"][k] for k in ("launches", "ms", "bytes", "gbs", "hbm_frac")}
                          if "depthwise" in cls else
                          {"launches": 0, "note": "every depthwise conv runs inside its fused inverted-residual "
                                                  "block (ir_block kernels, in the conv/dense MFMA class)"}),
            "kernel_classes": cls}

    m = _measure(args, "bert_ffn", workloads.build("bert_ffn"), dev, stream)
    measured.append(m)
    fl = sum(l["flops"] for l in m.launches)
    tf = fl / (m.ms * 1e-3) / 1e12
    out["bert_ffn"] = {
        "config": "BERT-base FFN x12, 1024 tokens (batch 8 x seq 128), hidden 768 -> 3072 (GELU) -> 768 + residual",
        "tokens_per_s": round(1024 / (m.ms * 1e-3), 1), "ms_per_step": round(m.ms, 4),
        "tflops": round(tf, 2), "mfma_frac": round(tf / PEAK_BF16_TFLOPS, 4), "launches": len(m.launches),
        "kernel_classes": _class_summary(m.launches, m.per_launch)}
    return out, measured


def _cpu_info():
    """CPU model, NumPy's BLAS and the threads its pool runs."""
    info = {}
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    info["cpu_model"] = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        import numpy as np
        blas = np.__config__.CONFIG["Build Dependencies"]["blas"]
        info["numpy_blas"] = "%s %s" % (blas.get("name"), blas.get("version"))
    except Exception:  # noqa: BLE001 - build metadata is optional
        pass
    try:
        from threadpoolctl import threadpool_info
        info["blas_pools"] = [{"api": p.get("internal_api"), "threads": p.get("num_threads"),
                               "version": p.get("version")} for p in threadpool_info()]
    except Exception:  # noqa: BLE001
        pass
    return info


def _sampled(wl, rows):
    import numpy as np
    g = dict(wl.graph)
    g["inputs"] = [dict(d, shape=[len(rows)] + list(d["shape"][1:])) for d in wl.graph["inputs"]]
    return g, [np.ascontiguousarray(a[rows]) for a in wl.inputs]


def _cpu_baseline_leg(headline, measured, cpu_images):
    """The oracle (NumPy float64) on this host: timed on the headline
    workload (the cpu_baseline), and evaluated on every timed workload to
    report the parity error of the outputs the GPU produced in its timed
    configuration.  The only place the benchmark runs the oracle."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle

    def err_of(got, ref):
        return float(np.max(np.abs(np.asarray(got) - ref) / (np.abs(ref) + 1.0)))

    cores = len(os.sched_getaffinity(0))
    parity = {}
    with threadpool_limits(limits=cores):
        n = headline.wl.inputs[0].shape[0]
        rows = list(range(min(cpu_images, n)))
        g, x = _sampled(headline.wl, rows)
        t0 = time.perf_counter()
        ref = oracle.run_graph(g, headline.wl.consts, x, mode="bf16io")[0]
        dt = time.perf_counter() - t0
        parity[headline.key] = {"err": err_of(headline.outputs[0][rows], ref), "tol": BF16_TOL,
                                "sample": "%d of %d images" % (len(rows), n), "mode": "bf16io",
                                "oracle_s": round(dt, 2)}
        cpu = {"value": round(len(rows) / dt, 4), "unit": "images/s", "cores": cores, "kind": "oracle",
               "threads": cores,
               "sample": "%d of the %d images of %s, one oracle call (NumPy float64, bf16io), %.1f s"
                         % (len(rows), n, headline.key, dt)}
        cpu.update(_cpu_info())
        for m in measured:
            wl = m.wl
            f32 = m.key == "conv_f32"
            mode, tol = ("exact", F32_TOL) if f32 else ("bf16io", BF16_TOL)
            n = wl.inputs[0].shape[0]
            rows = list(range(n)) if (n <= 16 or m.key == "bert_ffn") else [0, n - 1]
            g, x = _sampled(wl, rows)
            t0 = time.perf_counter()
            ref = oracle.run_graph(g, wl.consts, x, mode=mode)[0]
            entry = {"err": err_of(m.outputs[0][rows], ref), "tol": tol, "mode": mode,
                     "sample": "%s of %d %s" % ("all" if len(rows) == n else len(rows), n,
                                                "token rows" if m.key == "bert_ffn" else "images")}
            if m.key in ("bert_ffn", "darknet53_bs32"):
                ex = oracle.run_graph(g, wl.consts, x, mode="exact")[0]
                entry["oracle_bf16io_vs_exact"] = err_of(ex, ref)
                entry["note"] = ("bf16 storage along a long residual stream: flips of single roundings spread "
                                 "between layers; the oracle's own bf16io-vs-exact spread is of the same size")
            entry["oracle_s"] = round(time.perf_counter() - t0, 2)
            entry["ok"] = entry["err"] <= tol
            parity[m.key] = entry
    parity[headline.key]["ok"] = parity[headline.key]["err"] <= BF16_TOL
    for v in parity.values():
        v["err"] = float("%.4e" % v["err"])
    return cpu, parity


def _partitioned(args, wl, dev, stream):
    """The same network as an operator-level model with a softmax head on the
    host: partitioned (Sec. 3.1), then run by the partitioned-model runtime
    (Sec. 3.4) - the head on the host, the offloaded function through its
    cached engine."""
    import torch

    from paper_2105_03215_amd import host_runtime, partition

    g = partition.lower_subgraph(wl.graph, wl.consts)
    g.outputs = [g.call("nn.softmax", [g.outputs[0]], axis=-1)]
    t0 = time.perf_counter()
    part = partition.partition(g)
    part_ms = (time.perf_counter() - t0) * 1e3
    mod = host_runtime.Module(part, "cuda:0", graph_replay=not args.eager)
    try:
        if not args.no_autotune:
            for e in mod.engines:
                e.set_options(autotune=True)
        xs = [torch.from_numpy(x).to(dev) for x in wl.inputs]
        for _ in range(args.warmup):
            mod.run(xs, stream)
        torch.cuda.synchronize()
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            start.record(stream)
            for _ in range(args.steps):
                mod.run(xs, stream)
            end.record(stream)
        torch.cuda.synchronize()
        ms = start.elapsed_time(end) / args.steps
    finally:
        mod.close()
    st = part.stats()
    return {"images_per_s": round(args.batch / (ms * 1e-3), 1), "ms_per_step": round(ms, 4),
            "launch_mode": "direct launches" if args.eager else "HIP graph replay per function",
            "partition_ms": round(part_ms, 2),
            "functions": st["functions"], "host_steps": sum(1 for k, _ in part.steps if k == "host"),
            "node_offload": round(st["node_offload"], 4), "mac_offload": round(st["mac_offload"], 4)}


def _quantized(args, wl, dev, stream, calib_images=2, variant=None):
    """The same network partially quantized (Sec. 3.2, Fig. 4a): scales and
    zero points calibrated through the executor on a few images, int8 codes
    inside the function, quantize / dequantize at its boundary.  Same
    measurement as the headline; the conv class is priced against the dense
    int8 MFMA peak."""
    import copy

    import numpy as np

    from paper_2105_03215_amd import quantize, runtime

    variant = variant or args.variant
    t0 = time.perf_counter()
    cal = copy.deepcopy(wl.graph)
    cal["inputs"] = [dict(d, shape=[calib_images] + d["shape"][1:]) for d in cal["inputs"]]
    batch = [runtime.to_device(np.ascontiguousarray(a[:calib_images]), d["dtype"], dev)
             for a, d in zip(wl.inputs, cal["inputs"])]
    ranges = quantize.calibrate(cal, wl.consts, [batch])
    qg = quantize.quantize_graph(wl.graph, ranges)
    calib_s = time.perf_counter() - t0
    n = wl.inputs[0].shape[0]
    m = _measure(args, "%s_bs%d_int8" % (variant, n), wl, dev, stream, graph=qg)
    launches, per_launch, ms = m.launches, m.per_launch, m.ms
    if args.dump_launches and variant == args.variant:
        root, ext = os.path.splitext(args.dump_launches)
        with open(root + "_int8" + ext, "w") as f:
            json.dump([dict(l, ms=round(t, 5)) for l, t in zip(launches, per_launch)], f, indent=1)
    other_ms = sum(t for l, t in zip(launches, per_launch) if l["kind"] != "conv_i8")
    conv_ms = max(ms - other_ms, 1e-9)
    ops = sum(l["flops"] for l in launches if l["kind"] == "conv_i8")
    tops = ops / (conv_ms * 1e-3) / 1e12
    traffic = None
    tpath = os.path.join(ROOT, "profiles", "traffic_int8.json")
    if os.path.exists(tpath):
        from paper_2105_03215_amd import profiling
        with open(tpath) as f:
            tj = json.load(f)
        if (tj.get("workload") == "%s_bs%d_int8" % (variant, n)
                and tj.get("conv_kernel_digest") == profiling.conv_kernel_digest(profiling.I8_SOURCES)):
            traffic = tj.get("conv_bytes_per_step")
    return {"workload": "%s_bs%d_int8" % (variant, n), "images_per_s": round(n / (ms * 1e-3), 1),
            "ms_per_step": round(ms, 4), "launch_mode": m.extra["launch_mode"],
            "dtype": "int8 codes, int32 accumulation",
            "calibration": "%d images through the executor, %.2f s" % (calib_images, calib_s),
            "parity": "int8 codes are exact integer sums and float32 rescalings, independent of the tiling: "
                      "checked bit for bit against the int8 oracle on all 32 images in the GPU tests",
            "roofline": {"bound": "mfma", "achieved": round(tops, 2), "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                         "frac": round(tops / PEAK_INT8_TOPS, 4), "traffic": traffic,
                         "kernel": "conv/dense int8 MFMA class (the int8 stem, fused bottleneck blocks, conv_i8, "
                                   "the windowed 3x3 kernel), %d launches per step"
                                   % sum(1 for l in launches if l["kind"] == "conv_i8"),
                         "ops_per_step": ops, "kernel_ms_per_step": round(conv_ms, 4)},
            "kernel_classes": _class_summary(launches, per_launch), "launches": len(launches)}


def _other_workload(args, name, batch, dev, stream):
    """Throughput and conv-class roofline of another fully offloaded network
    (same measurement as the headline: autotune, inputs in HBM, the faster
    of direct launches and graph replay)."""
    from paper_2105_03215_amd import capi, workloads

    wl = workloads.build(name, n=batch)
    m = _measure(args, "%s_bs%d" % (name, batch), wl, dev, stream)
    roof = _roofline(m.launches, m.per_launch, m.ms)
    out = {"workload": m.key, "images_per_s": round(batch / (m.ms * 1e-3), 1),
           "ms_per_step": round(m.ms, 4), "launch_mode": m.extra["launch_mode"],
           "gflop_per_image": round(2 * wl.macs / batch / 1e9, 3),
           "conv_tflops": roof["achieved"], "conv_frac": roof["frac"], "launches": len(m.launches)}
    if not args.no_quantized:  # the same network partially quantized, as the headline's int8 leg
        try:
            q = _quantized(args, wl, dev, stream, variant=name)
            out["int8"] = {"images_per_s": q["images_per_s"], "ms_per_step": q["ms_per_step"],
                           "launch_mode": q["launch_mode"],
                           "conv_tops": q["roofline"]["achieved"], "conv_frac": q["roofline"]["frac"]}
        except capi.ByocError as e:  # operators without an int8 form
            out["int8"] = {"skipped": str(e)}
    return out, m


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--batch", type=int, default=32)
    ap.add_argument("--variant", default="resnet50_v1",
                    help="network of the headline run: resnet50_v1 (the benchmark), resnet50_v1b, vgg19, "
                         "darknet53, inception_v3, mobilenet_v2")
    ap.add_argument("--cpu-images", type=int, default=32)
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle leg (the CPU baseline and the parity report)")
    ap.add_argument("--no-bs1", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the conv_f32, ResNet-18 block, ResNet-50 bs1, MobileNetV2 and BERT FFN lines")
    ap.add_argument("--no-other", action="store_true", help="skip the VGG19, DarkNet-53 and Inception V3 bs32 lines")
    ap.add_argument("--no-quantized", action="store_true",
                    help="skip the int8 (partially quantized) run of the network")
    ap.add_argument("--no-partitioned", action="store_true",
                    help="skip the operator-level model run through the partitioner and its runtime")
    ap.add_argument("--no-autotune", action="store_true",
                    help="keep the built-in conv kernel choice (no on-device tuning at setup)")
    ap.add_argument("--no-cold", action="store_true", help="skip the cold-cache per-step timing")
    ap.add_argument("--eager", action="store_true",
                    help="headline value from direct launches even where HIP-graph replay is faster")
    ap.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "traffic.json"))
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a device copy of MIB MiB three times (counter calibration)")
    ap.add_argument("--dump-launches", default=None,
                    help="write a per-launch table (time, flops, bytes, roofline) to this JSON file")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: this executor has no multi-GPU path "
              "(batch sharding across GPUs needs no collective and is not built); "
              "use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2105_03215_amd import capi, runtime, workloads

    if args.copy_calibration:
        _copy_calibration(args.copy_calibration)
        print(json.dumps({"copy_calibration_mib": args.copy_calibration, "copies": 3}))
        return

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = workloads.build(args.variant, n=args.batch)
    t0 = time.perf_counter()
    sg = capi.Subgraph(wl.graph, wl.consts, device=0)
    create_s = time.perf_counter() - t0
    stream = torch.cuda.Stream(device=dev)
    ins = runtime.inputs_for(sg, wl.inputs, dev)
    outs = runtime.outputs_for(sg, dev)
    torch.cuda.synchronize()
    tune_s = None
    if not args.no_autotune:
        t0 = time.perf_counter()
        sg.set_options(autotune=True)
        tune_s = time.perf_counter() - t0
    for _ in range(args.warmup):
        sg.run(ins, outs, stream)
    torch.cuda.synchronize()
    ms_eager, wall_eager = _timed_runs(sg, ins, outs, stream, args.steps)
    sg.set_options(graph_replay=True)
    for _ in range(args.warmup):
        sg.run(ins, outs, stream)
    torch.cuda.synchronize()
    ms_graph, wall_graph = _timed_runs(sg, ins, outs, stream, args.steps)
    # the engine's figure is the faster of its two run modes, both timed
    # the same way above (as for the latency-bound configurations)
    if args.eager or ms_eager < ms_graph:
        sg.set_options(graph_replay=False)
        ms, wall, mode = ms_eager, wall_eager, "direct launches"
    else:
        ms, wall, mode = ms_graph, wall_graph, "HIP graph replay"
    value = args.batch / (ms * 1e-3)
    host_out = [runtime.to_host_f64(o) for o in outs]
    # warm / cold per-step distributions of the same configuration
    warm = _pct(_per_step(sg, ins, outs, stream, max(args.steps, 50)))
    timing = {"warm_ms": warm, "warm_images_per_s_at_median": round(args.batch / (warm["median"] * 1e-3), 1)}
    if not args.no_cold:
        evict = torch.empty(EVICT_MIB * 2 ** 20 // 4, dtype=torch.float32, device=dev)
        cold = _pct(_per_step(sg, ins, outs, stream, max(args.steps, 50), evict=evict))
        del evict
        timing.update({"cold_ms": cold, "cold_images_per_s_at_median": round(args.batch / (cold["median"] * 1e-3), 1),
                       "cold_eviction": "%d MiB written on the run stream before each run, outside its event pair"
                                        % EVICT_MIB})
    sg.set_options(graph_replay=False)
    launches = sg.launches()
    per_launch, runs = _profile(sg, ins, outs, stream, args.steps)
    traffic = None
    if os.path.exists(args.traffic_json):
        with open(args.traffic_json) as f:
            tj = json.load(f)
        if (tj.get("workload") == "%s_bs%d" % (args.variant, args.batch)
                and tj.get("conv_kernel_digest") == _conv_kernel_digest()):
            traffic = tj.get("conv_bytes_per_step")
    roof = _roofline(launches, per_launch, ms, traffic)
    roof["profiled_ms_per_step"] = round(sum(per_launch), 4)
    if args.dump_launches:
        table = []
        for l, t in zip(launches, per_launch):
            floor_ms = max(l["flops"] / (PEAK_BF16_TFLOPS * 1e12), l["bytes"] / (PEAK_HBM_GBS * 1e9)) * 1e3
            table.append(dict(l, ms=round(t, 5), roofline_ms=round(floor_ms, 5),
                              frac=round(floor_ms / t, 4) if t > 0 else None))
        with open(args.dump_launches, "w") as f:
            json.dump(table, f, indent=1)
    stats = sg.stats()
    sg.close()
    headline = Measured("%s_bs%d" % (args.variant, args.batch), wl, None, ms, launches, per_launch, host_out)

    measured = []
    configs = None
    if not args.no_configs:
        configs, measured = _config_lines(args, dev, stream)
    parted = None
    if not args.no_partitioned:
        parted = _partitioned(args, wl, dev, stream)
    quant = None
    if not args.no_quantized:
        try:
            quant = _quantized(args, wl, dev, stream)
        except capi.ByocError as e:  # e.g. operators without an int8 form
            quant = {"workload": "%s_bs%d_int8" % (args.variant, args.batch), "skipped": str(e)}
    other = None
    if not args.no_other:
        other = []
        for name in ("vgg19", "darknet53", "inception_v3"):
            line, m = _other_workload(args, name, 32, dev, stream)
            other.append(line)
            measured.append(m)

    cpu, parity = None, None
    if not args.no_cpu_baseline:
        cpu, parity = _cpu_baseline_leg(headline, measured, args.cpu_images)

    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "images/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded uniform[0,1) images, random He-init weights with folded BN)",
        "config": {"workload": "%s_bs%d" % (args.variant, args.batch), "batch": args.batch,
                   "input": list(wl.inputs[0].shape), "gflop_per_image": round(2 * wl.macs / args.batch / 1e9, 3),
                   "launches_per_step": len(launches), "parallelism": "none (1 GPU)",
                   "launch_mode": mode},
        "eager_images_per_s": round(args.batch / (ms_eager * 1e-3), 1),
        "graph_images_per_s": round(args.batch / (ms_graph * 1e-3), 1),
        "timing": timing,
        "roofline": roof,
        "cpu_baseline": cpu,
        "parity": parity,
        "bs1": (configs or {}).get("resnet50_v1_bs1"),
        "configs": configs,
        "partitioned": parted,
        "quantized": quant,
        "other_workloads": other,
        "kernel_classes": _class_summary(launches, per_launch),
        "create_s": round(create_s, 3),
        "autotune_s": None if tune_s is None else round(tune_s, 3),
        "weight_bytes": stats["weight_bytes"], "arena_bytes": stats["arena_bytes"],
        "wall_s_timed": round(wall, 4),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
