"""Throughput of the offloaded ResNet-50 v1 subgraph on one MI355X.

One step = one run of the whole offloaded subgraph (input layout transform,
53 conv composites, max-pool, global average pool, classifier) over a batch
of 32 synthetic 3x224x224 images already resident in HBM.  Prints one JSON
line with images/s, the roofline of the dominant kernel class (the bf16 MFMA
implicit-GEMM conv/dense kernels) measured with per-launch HIP events on the
run stream, the batch-1 figures, the same network as an operator-level
model partitioned for the executor and run by the partitioned-model runtime
with a host softmax head, and the CPU oracle timed on a bounded sample of the
same workload.

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
PEAK_INT8_TOPS = 5033.2  # dense int8 MFMA: 256 CU x 2.4 GHz x 8192 OP/clk
PEAK_HBM_GBS = 8000.0


def _timed_runs(sg, ins, outs, stream, steps):
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
    timed step (HIP events around the graph-replayed steps) less the other
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
            "kernel": ("conv/dense bf16 MFMA class (stem_conv_maxpool, conv_dma, conv_halo, conv_mfma, dense_rows, "
                       "splitk_reduce kernels), %d launches per step" % n_conv),
            "flops_per_step": conv_flops, "kernel_ms_per_step": round(conv_ms, 4),
            "per_launch_event_ms_per_step": round(conv_ev_ms, 4),
            "per_launch_event_frac": round(conv_flops / (conv_ev_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "layer_floor_ms_per_step": round(floor_ms, 4),
            "frac_of_layer_floor": round(floor_ms / conv_ms, 4)}


def _class_summary(launches, per_launch_ms):
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


def _cpu_baseline(wl, images):
    """The oracle (bf16io mode, float64 NumPy) on the first `images` images
    of the workload, on this host's cores."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle
    cores = len(os.sched_getaffinity(0))
    graph = dict(wl.graph)
    graph["inputs"] = [dict(d, shape=[images] + d["shape"][1:]) for d in wl.graph["inputs"]]
    x = [np.ascontiguousarray(a[:images]) for a in wl.inputs]
    with threadpool_limits(limits=cores):
        t0 = time.perf_counter()
        oracle.run_graph(graph, wl.consts, x, mode="bf16io")
        dt = time.perf_counter() - t0
    return {"value": round(images / dt, 4), "unit": "images/s", "cores": cores, "kind": "oracle",
            "sample": "%d of the 32 images, one oracle call (NumPy float64, bf16io), %.1f s"
                      % (images, dt)}


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
    import torch

    from paper_2105_03215_amd import capi, quantize, runtime

    variant = variant or args.variant
    t0 = time.perf_counter()
    cal = copy.deepcopy(wl.graph)
    cal["inputs"] = [dict(d, shape=[calib_images] + d["shape"][1:]) for d in cal["inputs"]]
    batch = [runtime.to_device(np.ascontiguousarray(a[:calib_images]), d["dtype"], dev)
             for a, d in zip(wl.inputs, cal["inputs"])]
    ranges = quantize.calibrate(cal, wl.consts, [batch])
    qg = quantize.quantize_graph(wl.graph, ranges)
    calib_s = time.perf_counter() - t0
    sg = capi.Subgraph(qg, wl.consts, device=0)
    try:
        ins = runtime.inputs_for(sg, wl.inputs, dev)
        outs = runtime.outputs_for(sg, dev)
        if not args.no_autotune:
            sg.set_options(autotune=True)
        sg.set_options(graph_replay=not args.eager)
        for _ in range(args.warmup):
            sg.run(ins, outs, stream)
        torch.cuda.synchronize()
        ms, _ = _timed_runs(sg, ins, outs, stream, args.steps)
        sg.set_options(graph_replay=False)
        launches = sg.launches()
        per_launch, _ = _profile(sg, ins, outs, stream, args.steps)
    finally:
        sg.close()
    if args.dump_launches and variant == args.variant:
        root, ext = os.path.splitext(args.dump_launches)
        with open(root + "_int8" + ext, "w") as f:
            json.dump([dict(l, ms=round(t, 5)) for l, t in zip(launches, per_launch)], f, indent=1)
    n = wl.inputs[0].shape[0]
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
            "ms_per_step": round(ms, 4), "dtype": "int8 codes, int32 accumulation",
            "calibration": "%d images through the executor, %.2f s" % (calib_images, calib_s),
            "roofline": {"bound": "mfma", "achieved": round(tops, 2), "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                         "frac": round(tops / PEAK_INT8_TOPS, 4), "traffic": traffic,
                         "kernel": "conv/dense int8 MFMA class (conv_i8), %d launches per step"
                                   % sum(1 for l in launches if l["kind"] == "conv_i8"),
                         "ops_per_step": ops, "kernel_ms_per_step": round(conv_ms, 4)},
            "kernel_classes": _class_summary(launches, per_launch), "launches": len(launches)}


def _other_workload(args, name, batch, dev, stream):
    """Throughput and conv-class roofline of another fully offloaded network
    (same measurement as the headline: graph replay, autotune, inputs in
    HBM)."""
    import torch

    from paper_2105_03215_amd import capi, runtime, workloads

    wl = workloads.build(name, n=batch)
    sg = capi.Subgraph(wl.graph, wl.consts, device=0)
    try:
        ins = runtime.inputs_for(sg, wl.inputs, dev)
        outs = runtime.outputs_for(sg, dev)
        if not args.no_autotune:
            sg.set_options(autotune=True)
        sg.set_options(graph_replay=not args.eager)
        for _ in range(args.warmup):
            sg.run(ins, outs, stream)
        torch.cuda.synchronize()
        ms, _ = _timed_runs(sg, ins, outs, stream, args.steps)
        sg.set_options(graph_replay=False)
        launches = sg.launches()
        per_launch, _ = _profile(sg, ins, outs, stream, args.steps)
    finally:
        sg.close()
    roof = _roofline(launches, per_launch, ms)
    out = {"workload": "%s_bs%d" % (name, batch), "images_per_s": round(batch / (ms * 1e-3), 1),
           "ms_per_step": round(ms, 4), "gflop_per_image": round(2 * wl.macs / batch / 1e9, 3),
           "conv_tflops": roof["achieved"], "conv_frac": roof["frac"], "launches": len(launches)}
    if not args.no_quantized:  # the same network partially quantized, as the headline's int8 leg
        try:
            q = _quantized(args, wl, dev, stream, variant=name)
            out["int8"] = {"images_per_s": q["images_per_s"], "ms_per_step": q["ms_per_step"],
                           "conv_tops": q["roofline"]["achieved"], "conv_frac": q["roofline"]["frac"]}
        except capi.ByocError as e:  # operators without an int8 form
            out["int8"] = {"skipped": str(e)}
    return out


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
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-bs1", action="store_true")
    ap.add_argument("--no-other", action="store_true", help="skip the VGG19, DarkNet-53 and Inception V3 bs32 lines")
    ap.add_argument("--no-quantized", action="store_true",
                    help="skip the int8 (partially quantized) run of the network")
    ap.add_argument("--no-partitioned", action="store_true",
                    help="skip the operator-level model run through the partitioner and its runtime")
    ap.add_argument("--no-autotune", action="store_true",
                    help="keep the built-in conv kernel choice (no on-device tuning at setup)")
    ap.add_argument("--eager", action="store_true",
                    help="headline value from direct launches instead of HIP-graph replay")
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
    sg.set_options(graph_replay=False)
    if args.eager:
        ms, wall, mode = ms_eager, wall_eager, "direct launches"
    else:
        ms, wall, mode = ms_graph, wall_graph, "HIP graph replay"
    value = args.batch / (ms * 1e-3)
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

    bs1 = None
    if not args.no_bs1 and args.batch != 1:
        wl1 = workloads.build(args.variant, n=1)
        sg1 = capi.Subgraph(wl1.graph, wl1.consts, device=0)
        if not args.no_autotune:
            sg1.set_options(autotune=True)
        ins1 = runtime.inputs_for(sg1, wl1.inputs, dev)
        outs1 = runtime.outputs_for(sg1, dev)
        for _ in range(args.warmup):
            sg1.run(ins1, outs1, stream)
        ms1e, _ = _timed_runs(sg1, ins1, outs1, stream, max(args.steps, 200))
        sg1.set_options(graph_replay=True)
        for _ in range(args.warmup):
            sg1.run(ins1, outs1, stream)
        ms1g, _ = _timed_runs(sg1, ins1, outs1, stream, max(args.steps, 200))
        ms1 = ms1e if args.eager else ms1g
        bs1 = {"images_per_s": round(1.0 / (ms1 * 1e-3), 1), "ms_per_step": round(ms1, 4),
               "launch_mode": mode, "eager_images_per_s": round(1.0 / (ms1e * 1e-3), 1),
               "launches": len(sg1.launches())}
        sg1.close()

    parted = None
    if not args.no_partitioned:
        parted = _partitioned(args, wl, dev, stream)
    quant = None
    if not args.no_quantized:
        try:
            quant = _quantized(args, wl, dev, stream)
        except capi.ByocError as e:  # e.g. depthwise convs have no int8 form
            quant = {"workload": "%s_bs%d_int8" % (args.variant, args.batch), "skipped": str(e)}
    other = None
    if not args.no_other:
        other = [_other_workload(args, "vgg19", 32, dev, stream),
                 _other_workload(args, "darknet53", 32, dev, stream),
                 _other_workload(args, "inception_v3", 32, dev, stream)]

    cpu = None
    if not args.no_cpu_baseline:
        cpu = _cpu_baseline(wl, args.cpu_images)

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
        "roofline": roof,
        "cpu_baseline": cpu,
        "bs1": bs1,
        "partitioned": parted,
        "quantized": quant,
        "other_workloads": other,
        "kernel_classes": _class_summary(launches, per_launch),
        "create_s": round(create_s, 3),
        "autotune_s": None if tune_s is None else round(tune_s, 3),
        "weight_bytes": stats["weight_bytes"], "arena_bytes": stats["arena_bytes"],
        "wall_s_timed": round(wall, 4),
    }
    sg.close()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
