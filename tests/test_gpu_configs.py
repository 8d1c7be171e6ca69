"""End-to-end parity of the workloads on the GPU against the oracle.

Small workloads are compared on every output element; the batched ones at
their full size in the benchmark's launch configuration, on images (or
token rows) that the oracle recomputes one by one - every image of a CNN
batch and every token row of the FFN stack is independent of the others.
"""

import numpy as np
import pytest

import oracle
from paper_2105_03215_amd import workloads
from parity_util import (BF16_TOL, F32_TOL, announce, gate_end_to_end, rel_err, term_scale_node,
                         within_one_ulp)

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _gpu(wl):
    from paper_2105_03215_amd import capi, runtime
    sg = capi.Subgraph(wl.graph, wl.consts, device=0)
    try:
        return runtime.run_once(sg, wl.inputs, DEV)
    finally:
        sg.close()


def _sample_inputs(wl, rows):
    return [np.ascontiguousarray(a[rows]) for a in wl.inputs]


def _sample_graph(wl, n):
    g = dict(wl.graph)
    g["inputs"] = [dict(d, shape=[n] + d["shape"][1:]) for d in wl.graph["inputs"]]
    return g


def test_conv_f32_config():
    announce("conv_f32 config")
    wl = workloads.conv_f32()
    g = _gpu(wl)[0]
    o = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="exact")[0]
    assert rel_err(g, o) <= F32_TOL


def test_resnet18_block():
    announce("resnet18_block 1x64x56x56")
    wl = workloads.resnet18_block()
    g = _gpu(wl)[0]
    o = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="bf16io")[0]
    assert g.shape == (1, 64, 56, 56)
    assert rel_err(g, o) <= BF16_TOL


def test_resnet18_block_teacher_forced():
    """Every composite recomputed by the oracle from the GPU's own inputs."""
    announce("resnet18_block teacher forced")
    wl = workloads.resnet18_block()
    graph = dict(wl.graph)
    graph["outputs"] = [{"name": n["name"], "dtype": "bf16", "layout": "NCHW"} for n in graph["nodes"]]
    wl2 = workloads.Workload(graph, wl.consts, wl.inputs, wl.macs, wl.conv_macs)
    gpu = _gpu(wl2)
    vals = {"x": oracle.bf16.round_bf16(wl.inputs[0])}
    for c in graph["constants"]:
        vals[c["name"]] = wl.consts[c["index"]]
    for node, g in zip(graph["nodes"], gpu):
        args = [vals[r] for r in node["inputs"]]
        ref = oracle.run_node(node, args)
        assert within_one_ulp(g, ref, term_scale_node(node, args)).all(), node["name"]
        vals[node["name"]] = g


@pytest.mark.parametrize("variant", ["resnet50_v1", "resnet50_v1b"])
def test_resnet50_bs1(variant):
    announce(variant + " bs1")
    wl = workloads.build(variant, n=1)
    g = _gpu(wl)[0]
    o = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="bf16io")[0]
    assert g.shape == (1, 1000)
    err = rel_err(g, o)
    print("%s bs1 err %.3e" % (variant, err))
    assert err <= BF16_TOL


def test_resnet50_bs32_sampled():
    announce("resnet50_v1 bs32 sampled images 0 and 31")
    wl = workloads.build("resnet50_v1", n=32)
    g = _gpu(wl)[0]
    rows = [0, 31]
    o = oracle.run_graph(_sample_graph(wl, 2), wl.consts, _sample_inputs(wl, rows), mode="bf16io")[0]
    err = rel_err(g[rows], o)
    print("resnet50 bs32 err %.3e" % err)
    assert err <= BF16_TOL
    assert np.all(np.isfinite(g))


def test_resnet50_f32_input_boundary():
    announce("resnet50_v1 bs2 f32 input (boundary cast)")
    wl = workloads.resnet50(n=2, input_dtype="f32")
    g = _gpu(wl)[0]
    o = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="bf16io")[0]
    assert rel_err(g, o) <= BF16_TOL


def test_mobilenet_v2_bs1():
    announce("mobilenet_v2 bs1")
    wl = workloads.build("mobilenet_v2", n=1)
    g = _gpu(wl)[0]
    o = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="bf16io")[0]
    err = rel_err(g, o)
    print("mobilenet_v2 bs1 err %.3e" % err)
    assert err <= BF16_TOL


def test_mobilenet_v2_bs16_sampled():
    announce("mobilenet_v2 bs16 sampled images 0 and 15")
    wl = workloads.build("mobilenet_v2", n=16)
    g = _gpu(wl)[0]
    rows = [0, 15]
    o = oracle.run_graph(_sample_graph(wl, 2), wl.consts, _sample_inputs(wl, rows), mode="bf16io")[0]
    err = rel_err(g[rows], o)
    print("mobilenet_v2 bs16 err %.3e" % err)
    assert err <= BF16_TOL


def test_vgg19_bs1_112():
    announce("vgg19 bs1 112x112")
    wl = workloads.build("vgg19", n=1, hw=112)
    g = _gpu(wl)[0]
    o = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="bf16io")[0]
    assert g.shape == (1, 1000)
    err = rel_err(g, o)
    print("vgg19 bs1 112 err %.3e" % err)
    assert err <= BF16_TOL


def test_vgg19_bs8_sampled():
    announce("vgg19 bs8 224x224 sampled image 7")
    wl = workloads.build("vgg19", n=8)
    g = _gpu(wl)[0]
    rows = [7]
    o = oracle.run_graph(_sample_graph(wl, 1), wl.consts, _sample_inputs(wl, rows), mode="bf16io")[0]
    err = rel_err(g[rows], o)
    print("vgg19 bs8 err %.3e" % err)
    assert err <= BF16_TOL
    assert np.all(np.isfinite(g))


def test_darknet53_teacher_forced():
    """All 76 composites of DarkNet-53 (bs1, 128x128), each recomputed by
    the oracle from the GPU's own inputs, within one bf16 ulp."""
    announce("darknet53 teacher forced, 76 composites")
    wl = workloads.build("darknet53", n=1, hw=128)
    graph = dict(wl.graph)
    graph["outputs"] = [{"name": n["name"], "dtype": "bf16"} for n in graph["nodes"]]
    gpu = _gpu(workloads.Workload(graph, wl.consts, wl.inputs, wl.macs, wl.conv_macs))
    vals = {"x": oracle.bf16.round_bf16(wl.inputs[0])}
    consts = {c["name"]: wl.consts[c["index"]] for c in graph["constants"]}
    for node, g in zip(graph["nodes"], gpu):
        args = [vals[r] if r in vals else consts[r] for r in node["inputs"]]
        ref = oracle.run_node(node, args)
        assert within_one_ulp(g, ref, term_scale_node(node, args)).all(), node["name"]
        vals[node["name"]] = g


def _darknet_gate(graph, consts, inputs, got, what):
    io = oracle.run_graph(graph, consts, inputs, mode="bf16io")[0]
    ex = oracle.run_graph(graph, consts, inputs, mode="exact")[0]
    gate_end_to_end(rel_err(got, io), rel_err(io, ex), what)


def test_darknet53_bs1_128():
    announce("darknet53 bs1 128x128")
    wl = workloads.build("darknet53", n=1, hw=128)
    g = _gpu(wl)[0]
    _darknet_gate(wl.graph, wl.consts, wl.inputs, g, "darknet53 bs1 128x128")


def test_darknet53_bs32_sampled():
    announce("darknet53 bs32 256x256 sampled images 0 and 31")
    wl = workloads.build("darknet53", n=32)
    g = _gpu(wl)[0]
    assert np.all(np.isfinite(g))
    rows = [0, 31]
    _darknet_gate(_sample_graph(wl, 2), wl.consts, _sample_inputs(wl, rows), g[rows], "darknet53 bs32 images 0, 31")


def test_inception_v3_bs1():
    announce("inception_v3 bs1 299x299")
    wl = workloads.build("inception_v3", n=1)
    g = _gpu(wl)[0]
    o = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="bf16io")[0]
    err = rel_err(g, o)
    print("inception_v3 bs1 err %.3e" % err)
    assert err <= BF16_TOL


def test_inception_v3_bs32_sampled():
    announce("inception_v3 bs32 299x299 sampled images 0 and 31")
    wl = workloads.build("inception_v3", n=32)
    g = _gpu(wl)[0]
    rows = [0, 31]
    o = oracle.run_graph(_sample_graph(wl, 2), wl.consts, _sample_inputs(wl, rows), mode="bf16io")[0]
    err = rel_err(g[rows], o)
    print("inception_v3 bs32 err %.3e" % err)
    assert err <= BF16_TOL
    assert np.all(np.isfinite(g))


def test_bert_ffn_layers_teacher_forced():
    """All 24 dense composites at full size (1024 tokens), each recomputed by
    the oracle on 64 sampled token rows from the GPU's own layer input."""
    announce("bert_ffn teacher forced, 24 composites")
    wl = workloads.build("bert_ffn")
    graph = dict(wl.graph)
    graph["outputs"] = [{"name": n["name"], "dtype": "bf16"} for n in graph["nodes"]]
    wl2 = workloads.Workload(graph, wl.consts, wl.inputs, wl.macs, wl.conv_macs)
    gpu = _gpu(wl2)
    rows = np.random.default_rng(0).choice(1024, 64, replace=False)
    vals = {"x": wl.inputs[0][rows]}
    consts = {c["name"]: wl.consts[c["index"]] for c in graph["constants"]}
    worst = 0.0
    for node, g in zip(graph["nodes"], gpu):
        args = [vals[r] if r in vals else consts[r] for r in node["inputs"]]
        ref = oracle.run_node(node, args)
        assert within_one_ulp(g[rows], ref, term_scale_node(node, args)).all(), node["name"]
        worst = max(worst, rel_err(g[rows], ref))
        vals[node["name"]] = g[rows]
    print("bert per-layer worst err %.3e" % worst)
    assert worst <= BF16_TOL


def test_bert_ffn_end_to_end_sampled():
    """Full stack on 64 sampled rows against the fixed 1e-2 gate (an expected
    failure with its measured error when the bf16 residual stream drifts
    past it, see gate_end_to_end)."""
    announce("bert_ffn end to end sampled rows")
    wl = workloads.build("bert_ffn")
    g = _gpu(wl)[0]
    rows = np.random.default_rng(1).choice(1024, 64, replace=False)
    graph = dict(wl.graph)
    graph["inputs"] = [dict(graph["inputs"][0], shape=[64, 768])]
    io = oracle.run_graph(graph, wl.consts, [wl.inputs[0][rows]], mode="bf16io")[0]
    ex = oracle.run_graph(graph, wl.consts, [wl.inputs[0][rows]], mode="exact")[0]
    gate_end_to_end(rel_err(g[rows], io), rel_err(io, ex), "bert_ffn 64 sampled rows")
