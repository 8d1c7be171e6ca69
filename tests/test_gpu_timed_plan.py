"""Parity of exactly what the benchmark times.

bench.py times every workload with the engine's autotune on (each conv /
dense launch takes the fastest of its result-identical kernel variants,
chosen by timing on the device) on a non-default stream, in HIP-graph replay
and in direct launches, and reports the faster mode.  Here each of those
configurations is built the same way, at the benchmark's size, run several
times in both modes (the output buffer poisoned between runs), and compared:

* bit for bit with the engine's built-in plan (autotune changes speed only);
* with the oracle (bf16io mode) on every image / token row of the batch,
  within max |gpu - oracle| / (|oracle| + 1) <= 1e-2 (fp32: 1e-4 against the
  exact oracle).

The BERT-shaped FFN stack (twelve residual layers in bf16 storage) and
DarkNet-53 (23 residual adds after the activation) do not meet 1e-2 end to
end for any implementation that accumulates in fp32: one rounding that
lands on the other side of a bf16 tie perturbs the next layer's inputs
enough to flip further roundings, and the flips spread along the residual
stream.  Those cases are recorded as expected failures with the measured
error and the oracle's own bf16io-vs-exact spread (parity_util.
gate_end_to_end); their composites are held to one bf16 ulp teacher-forced
in test_gpu_configs.py.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2105_03215_amd import capi, runtime, workloads
from parity_util import BF16_TOL, F32_TOL, announce, gate_end_to_end, rel_err

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _bitwise_equal(a, b):
    if a.dtype == torch.bfloat16:
        return torch.equal(a.view(torch.int16), b.view(torch.int16))
    return torch.equal(a, b)


def timed_plan_outputs(wl, replays=3):
    """Outputs of the benchmark's launch configuration (autotune, a side
    stream) after `replays` graph replays and as many direct-launch runs,
    checked bit for bit against the built-in plan's after every run."""
    sg = capi.Subgraph(wl.graph, wl.consts, device=0)
    s = torch.cuda.Stream(device=DEV)
    try:
        ins = runtime.inputs_for(sg, wl.inputs, DEV)
        ref = runtime.outputs_for(sg, DEV)
        torch.cuda.synchronize()
        sg.run(ins, ref, s)
        s.synchronize()
        sg.set_options(autotune=True)
        out = runtime.outputs_for(sg, DEV)
        for replay in (True, False):
            sg.set_options(graph_replay=replay)
            for rep in range(replays):
                for o in out:
                    o.fill_(float("nan"))
                torch.cuda.synchronize()
                sg.run(ins, out, s)
                s.synchronize()
                for a, b in zip(ref, out):
                    assert _bitwise_equal(a, b), "%s run %d differs from the built-in plan" % (
                        "graph" if replay else "direct", rep)
        names = [l["name"] for l in sg.launches()]
        return [runtime.to_host_f64(o) for o in out], names
    finally:
        sg.close()


def _check(name, n=None, mode="bf16io", tol=BF16_TOL, **kw):
    wl = workloads.build(name, n=n, **kw) if n is not None else workloads.build(name, **kw)
    announce("timed plan %s n=%s %s" % (name, n, kw))
    got, names = timed_plan_outputs(wl)
    ref = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode=mode)
    errs = [rel_err(g, o) for g, o in zip(got, ref)]
    print("timed plan %s n=%s: err %s (tol %.0e), %d launches" % (name, n, ["%.3e" % e for e in errs], tol,
                                                                    len(names)), flush=True)
    for g in got:
        assert np.all(np.isfinite(g))
    assert max(errs) <= tol
    return got, ref


def test_conv_f32_timed_plan():
    _check("conv_f32", mode="exact", tol=F32_TOL)


def test_resnet18_block_timed_plan():
    _check("resnet18_block")


def test_resnet50_bs1_timed_plan():
    _check("resnet50_v1", n=1)


@pytest.mark.timeout(600)
def test_resnet50_bs32_timed_plan_all_images():
    got, ref = _check("resnet50_v1", n=32)
    per_image = [rel_err(got[0][i], ref[0][i]) for i in range(32)]
    print("resnet50 bs32 per-image err max %.3e min %.3e" % (max(per_image), min(per_image)))


def test_mobilenet_v2_bs1_timed_plan():
    _check("mobilenet_v2", n=1)


@pytest.mark.timeout(600)
def test_mobilenet_v2_bs16_timed_plan_all_images():
    _check("mobilenet_v2", n=16)


@pytest.mark.timeout(900)
def test_vgg19_bs32_timed_plan_all_images():
    _check("vgg19", n=32)


@pytest.mark.timeout(900)
def test_darknet53_bs32_timed_plan_all_images():
    wl = workloads.build("darknet53", n=32)
    announce("timed plan darknet53 n=32")
    got, _ = timed_plan_outputs(wl)
    assert np.all(np.isfinite(got[0]))
    io = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="bf16io")[0]
    ex = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="exact")[0]
    gate_end_to_end(rel_err(got[0], io), rel_err(io, ex), "timed plan darknet53 bs32, all 32 images")


@pytest.mark.timeout(900)
def test_inception_v3_bs32_timed_plan_all_images():
    _check("inception_v3", n=32)


@pytest.mark.timeout(600)
def test_bert_ffn_timed_plan_all_rows():
    wl = workloads.build("bert_ffn")
    announce("timed plan bert_ffn 1024 tokens")
    got, _ = timed_plan_outputs(wl)
    assert np.all(np.isfinite(got[0]))
    io = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="bf16io")[0]
    ex = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="exact")[0]
    gate_end_to_end(rel_err(got[0], io), rel_err(io, ex), "timed plan bert_ffn, all 1024 tokens")


@pytest.mark.timeout(900)
def test_resnet50_bs32_int8_timed_plan_all_images():
    """The partially quantized network as the benchmark times it: every
    image's codes equal the int8 oracle's (exact integer sums, the same
    float32 rescalings)."""
    from oracle import quant as OQ
    from parity_util import oracle_calibrated_int8
    wl = workloads.build("resnet50_v1", n=32)
    qg = oracle_calibrated_int8(wl.graph, wl.consts, [np.ascontiguousarray(a[:2]) for a in wl.inputs])
    announce("timed plan resnet50_v1 bs32 int8")
    got, names = timed_plan_outputs(workloads.Workload(qg, wl.consts, wl.inputs, wl.macs, wl.conv_macs))
    # the fused int8 stem, the seven stage-1/2 blocks fused (three convs each,
    # four with the projection), the other 30 convs and the classifier
    assert names.count("stem_conv_maxpool_i8") == 1, names
    assert sum(1 for n in names if n.startswith("bottleneck_i8_")) == 7, names
    assert sum(1 for n in names if n.startswith("conv_i8")) == 30, names
    ref = OQ.run_quantized_graph(qg, wl.consts, wl.inputs)[0]
    diff = np.abs(got[0] - ref.astype(np.float64))
    print("timed plan resnet50 bs32 int8: %d of %d outputs differ" % (int((diff > 0).sum()), diff.size))
    assert np.array_equal(got[0], ref.astype(np.float64))


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["vgg19", "darknet53"])
def test_other_networks_bs32_int8_timed_plan_sampled(name):
    """The int8 forms of VGG19 and DarkNet-53 at the benchmark's batch 32
    and full resolution, autotuned and graph-replayed as the benchmark runs
    them; the int8 oracle recomputes images 0 and 31 (each image's codes
    depend only on that image), which must match bit for bit."""
    from oracle import quant as OQ
    from parity_util import oracle_calibrated_int8
    wl = workloads.build(name, n=32)
    qg = oracle_calibrated_int8(wl.graph, wl.consts, [np.ascontiguousarray(a[:2]) for a in wl.inputs])
    announce("timed plan %s bs32 int8" % name)
    got, names = timed_plan_outputs(workloads.Workload(qg, wl.consts, wl.inputs, wl.macs, wl.conv_macs))
    assert any(n.startswith("conv_i8") for n in names)
    rows = [0, 31]
    g2 = dict(qg)
    g2["inputs"] = [dict(d, shape=[2] + list(d["shape"][1:])) for d in qg["inputs"]]
    ref = OQ.run_quantized_graph(g2, wl.consts, [np.ascontiguousarray(a[rows]) for a in wl.inputs])[0]
    diff = np.abs(got[0][rows] - ref.astype(np.float64))
    print("timed plan %s bs32 int8: %d of %d sampled outputs differ" % (name, int((diff > 0).sum()), diff.size))
    assert np.array_equal(got[0][rows], ref.astype(np.float64))
