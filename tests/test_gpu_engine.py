"""Engine behaviour on the GPU: run-to-run bitwise determinism (including the
split-K path), guard canaries around outputs, runs on a non-default stream,
two engines on two streams, the profiling and introspection calls, and
argument errors of run()."""

import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2105_03215_amd import capi, runtime, workloads
from paper_2105_03215_amd.workloads import GraphBuilder
from parity_util import BF16_TOL, announce, rel_err

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _splitk_workload():
    g = GraphBuilder("splitk_det", 2000)
    x = g.input("x", [1, 512, 7, 7], "uniform")
    y = g.conv(x, 512, 3, act="relu", name="y")
    g.output(y)
    return g.finish()


def _kgroups_workload():
    g = GraphBuilder("kgroups_det", 2001)
    x = g.input("x", [1, 64, 56, 56], "uniform")
    y = g.conv(x, 64, 3, act="relu", name="y")
    g.output(y)
    return g.finish()


@pytest.mark.parametrize("name", ["resnet18_block", "splitk", "kgroups4"])
def test_bitwise_deterministic(name, monkeypatch):
    announce("determinism " + name)
    wl = {"resnet18_block": workloads.resnet18_block, "splitk": _splitk_workload,
          "kgroups4": _kgroups_workload}[name]()
    sg = capi.Subgraph(wl.graph, wl.consts)
    try:
        if name == "splitk":
            assert any(l["kind"] == "reduce" for l in sg.launches())
        if name == "kgroups4":  # few tiles: four reduction groups in one workgroup
            assert any("_k4_" in l["name"] for l in sg.launches()), [l["name"] for l in sg.launches()]
        if name != "resnet18_block":
            o = oracle.run_graph(wl.graph, wl.consts, wl.inputs)[0]
        ins = runtime.inputs_for(sg, wl.inputs, DEV)
        a = runtime.outputs_for(sg, DEV)
        b = runtime.outputs_for(sg, DEV)
        sg.run(ins, a)
        sg.run(ins, b)
        torch.cuda.synchronize()
        for x, y in zip(a, b):
            assert torch.equal(x.view(torch.int16), y.view(torch.int16))
        if name != "resnet18_block":
            assert rel_err(runtime.to_host_f64(a[0]), o) <= BF16_TOL
    finally:
        sg.close()


def _canary_run(wl):
    sg = capi.Subgraph(wl.graph, wl.consts)
    try:
        ins = runtime.inputs_for(sg, wl.inputs, DEV)
        bufs, outs = [], []
        pad = 4096
        for j in range(sg.n_out):
            d = sg.io_desc(1, j)
            n = int(np.prod(d["shape"]))
            dt = runtime.torch_dtype(d["dtype"])
            buf = torch.full((n + 2 * pad,), -7.0, dtype=dt, device=DEV)
            bufs.append(buf)
            outs.append(buf[pad:pad + n].view(d["shape"]))
        sg.run(ins, outs)
        torch.cuda.synchronize()
        for buf, o in zip(bufs, outs):
            n = o.numel()
            assert torch.all(buf[:pad] == -7.0) and torch.all(buf[pad + n:] == -7.0)
        return [runtime.to_host_f64(o) for o in outs]
    finally:
        sg.close()


def test_output_canaries_4d_and_2d():
    announce("canaries")
    wl = workloads.resnet18_block(n=1, c=64, hw=14)
    g = _canary_run(wl)[0]
    o = oracle.run_graph(wl.graph, wl.consts, wl.inputs)[0]
    assert rel_err(g, o) <= BF16_TOL
    wl = workloads.bert_ffn(batch=1, seq=40, layers=2)
    g = _canary_run(wl)[0]
    o = oracle.run_graph(wl.graph, wl.consts, wl.inputs)[0]
    assert rel_err(g, o) <= BF16_TOL


def test_nondefault_streams_two_engines():
    announce("two engines on two streams")
    w1 = workloads.resnet18_block(n=2, c=64, hw=28)
    w2 = workloads.mobilenet_v2(n=1, hw=96)
    s1 = torch.cuda.Stream(device=DEV)
    s2 = torch.cuda.Stream(device=DEV)
    e1 = capi.Subgraph(w1.graph, w1.consts)
    e2 = capi.Subgraph(w2.graph, w2.consts)
    try:
        i1, o1 = runtime.inputs_for(e1, w1.inputs, DEV), runtime.outputs_for(e1, DEV)
        i2, o2 = runtime.inputs_for(e2, w2.inputs, DEV), runtime.outputs_for(e2, DEV)
        torch.cuda.synchronize()
        for _ in range(3):
            e1.run(i1, o1, s1)
            e2.run(i2, o2, s2)
        s1.synchronize()
        s2.synchronize()
        g1 = runtime.to_host_f64(o1[0])
        g2 = runtime.to_host_f64(o2[0])
    finally:
        e1.close()
        e2.close()
    assert rel_err(g1, oracle.run_graph(w1.graph, w1.consts, w1.inputs)[0]) <= BF16_TOL
    assert rel_err(g2, oracle.run_graph(w2.graph, w2.consts, w2.inputs)[0]) <= BF16_TOL


def test_profiling_and_introspection():
    announce("profiling api")
    wl = workloads.resnet18_block()
    sg = capi.Subgraph(wl.graph, wl.consts)
    try:
        st = sg.stats()
        assert st["macs"] == wl.macs and st["weight_bytes"] > 0 and st["arena_bytes"] > 0
        assert sg.io_desc(0, 0) == {"dtype": "bf16", "layout": "NCHW", "shape": [1, 64, 56, 56]}
        launches = sg.launches()
        kinds = [l["kind"] for l in launches]
        assert kinds[0] == "transform" and kinds[-1] == "transform"
        assert sum(l["flops"] for l in launches) == 2 * wl.macs
        ins = runtime.inputs_for(sg, wl.inputs, DEV)
        outs = runtime.outputs_for(sg, DEV)
        sg.profile_begin(3)
        for _ in range(4):
            sg.run(ins, outs)
        ms, runs = sg.profile_end()
        assert runs == 3 and len(ms) == len(launches) and all(t > 0 for t in ms)
        with pytest.raises(capi.ByocError):
            sg.profile_end()
    finally:
        sg.close()


def test_run_argument_errors():
    announce("run argument errors")
    wl = workloads.conv_f32(n=1, c=4, hw=6, k=3)
    sg = capi.Subgraph(wl.graph, wl.consts)
    try:
        ins = runtime.inputs_for(sg, wl.inputs, DEV)
        outs = runtime.outputs_for(sg, DEV)
        with pytest.raises(capi.ByocError) as ei:
            sg.run(ins + ins, outs)
        assert ei.value.status_name == "INVALID_ARG" and "expected 1 inputs" in str(ei.value)
        with pytest.raises(capi.ByocError):
            sg.run([0], outs)
        lib = capi.load_library()
        assert lib.byoc_subgraph_destroy(None) == 0
        assert lib.byoc_subgraph_run(None, None, 0, None, 0, None) == 1
    finally:
        sg.close()


def test_graph_replay_matches_eager():
    """HIP-graph replay: every replay, with eager torch work and host
    synchronisations between replays, equals the direct-launch result bit for
    bit; new output pointers are recorded anew; the null stream falls back to
    direct launches."""
    announce("graph replay")
    wl = workloads.resnet18_block(n=2, c=64, hw=28)
    sg = capi.Subgraph(wl.graph, wl.consts)
    s = torch.cuda.Stream(device=DEV)
    try:
        ins = runtime.inputs_for(sg, wl.inputs, DEV)
        ref = runtime.outputs_for(sg, DEV)
        sg.run(ins, ref, s)
        s.synchronize()
        sg.set_options(graph_replay=True)
        outs = runtime.outputs_for(sg, DEV)
        for rep in range(4):
            outs[0].fill_(-1.0)
            torch.cuda.synchronize()
            sg.run(ins, outs, s)
            s.synchronize()
            assert torch.equal(outs[0].view(torch.int16), ref[0].view(torch.int16)), rep
        other = runtime.outputs_for(sg, DEV)
        sg.run(ins, other, s)
        sg.run(ins, outs, s)
        s.synchronize()
        assert torch.equal(other[0].view(torch.int16), ref[0].view(torch.int16))
        assert torch.equal(outs[0].view(torch.int16), ref[0].view(torch.int16))
        null_out = runtime.outputs_for(sg, DEV)
        sg.run(ins, null_out, 0)
        torch.cuda.synchronize()
        assert torch.equal(null_out[0].view(torch.int16), ref[0].view(torch.int16))
        with pytest.raises(capi.ByocError):
            capi._check(sg.lib.byoc_subgraph_set_options(sg.handle, 6))
        sg.set_options(graph_replay=False)
    finally:
        sg.close()


@pytest.mark.parametrize("name", ["resnet18_block", "resnet50_bs2", "bert_ffn"])
def test_autotune_keeps_results_bitwise(name):
    """Autotune swaps conv kernel variants only among result-identical ones:
    outputs stay bit-for-bit those of the built-in choice, also under graph
    replay, and turning it off restores the built-in launch plan."""
    announce("autotune " + name)
    if name == "resnet18_block":
        wl = workloads.resnet18_block(n=2, c=64, hw=28)
    elif name == "resnet50_bs2":
        wl = workloads.build("resnet50_v1", n=2)
    else:
        wl = workloads.bert_ffn(batch=1, seq=40, layers=1)
    sg = capi.Subgraph(wl.graph, wl.consts)
    s = torch.cuda.Stream(device=DEV)
    try:
        ins = runtime.inputs_for(sg, wl.inputs, DEV)
        ref = runtime.outputs_for(sg, DEV)
        sg.run(ins, ref, s)
        s.synchronize()
        names0 = [l["name"] for l in sg.launches()]
        sg.set_options(autotune=True)
        for replay in (False, True):
            sg.set_options(graph_replay=replay)
            out = runtime.outputs_for(sg, DEV)
            sg.run(ins, out, s)
            sg.run(ins, out, s)
            s.synchronize()
            for a, b in zip(ref, out):
                assert torch.equal(a.view(torch.int16), b.view(torch.int16)), (name, replay)
        sg.set_options(graph_replay=False, autotune=False)
        assert [l["name"] for l in sg.launches()] == names0
    finally:
        sg.close()


@pytest.mark.parametrize("name,n", [("resnet50_v1", 32), ("resnet50_v1", 1), ("inception_v3", 2),
                                    ("darknet53", 2), ("mobilenet_v2", 4)])
def test_two_streams_match_one_stream(name, n, monkeypatch):
    """With two-stream execution (BYOC_STREAMS=2) launches that do not
    depend on their predecessor run on the engine's side stream (fork and
    join through events, also when captured as a graph).  Outputs equal those
    of the single-stream plan bit for bit, on direct launches and on graph
    replays, with the output buffer poisoned between runs (a missing
    dependency shows as a difference)."""
    announce("two streams vs one: %s n=%d" % (name, n))
    wl = workloads.build(name, n=n)
    monkeypatch.delenv("BYOC_STREAMS", raising=False)
    one = capi.Subgraph(wl.graph, wl.consts)
    monkeypatch.setenv("BYOC_STREAMS", "2")
    two = capi.Subgraph(wl.graph, wl.consts)
    monkeypatch.delenv("BYOC_STREAMS")
    s = torch.cuda.Stream(device=DEV)
    try:
        ins = runtime.inputs_for(one, wl.inputs, DEV)
        ref = runtime.outputs_for(one, DEV)
        one.run(ins, ref, s)
        s.synchronize()
        for replay in (False, True, True, True):
            two.set_options(graph_replay=replay)
            out = runtime.outputs_for(two, DEV)
            for o in out:
                o.fill_(float("nan"))
            torch.cuda.synchronize()
            for _ in range(2):
                two.run(ins, out, s)
            s.synchronize()
            for a, b in zip(ref, out):
                assert torch.equal(a.view(torch.int16), b.view(torch.int16)), (name, n, replay)
    finally:
        one.close()
        two.close()
