"""The allocation-free entry point byoc_subgraph_run_static against
byoc_subgraph_run: the same engine, the same inputs, outputs bit for bit
equal, for two calls in a row where the second runs a smaller input (an
engine of the same network at a smaller batch) on the scratch the first one
left behind, then the first engine again.  ResNet-50 at batch 1 is built
with split-K launches, whose fp32 partial sums live in the scratch too.  An
engine whose intermediates exceed the scratch is rejected before anything is
enqueued."""

import pytest
import torch

from paper_2105_03215_amd import capi, runtime, workloads
from parity_util import announce

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
SCRATCH_BYTES = 64 << 20


def _engine(name, n):
    wl = workloads.build(name, n=n)
    sg = capi.Subgraph(wl.graph, wl.consts, device=0)
    return wl, sg


def _static_vs_run(sg, wl, stream):
    ins = runtime.inputs_for(sg, wl.inputs, DEV)
    ref = runtime.outputs_for(sg, DEV)
    out = runtime.outputs_for(sg, DEV)
    for o in out:
        o.fill_(-3.0)
    torch.cuda.synchronize()
    sg.run(ins, ref, stream)
    sg.run_static(ins, out, stream)
    stream.synchronize()
    for a, b in zip(ref, out):
        assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                           b.view(torch.int16) if b.dtype == torch.bfloat16 else b)


def test_run_static_matches_run_two_calls_second_smaller(monkeypatch):
    announce("run_static: resnet50_v1 bs4 then bs1 (split-K), then bs4 again")
    s = torch.cuda.Stream(device=DEV)
    wl2, sg2 = _engine("resnet50_v1", 4)
    monkeypatch.setenv("BYOC_CONV_SPLIT", "4")  # few-tile layers as split-K launches
    wl1, sg1 = _engine("resnet50_v1", 1)
    monkeypatch.delenv("BYOC_CONV_SPLIT")
    try:
        a2 = sg2.stats()["arena_bytes"]
        a1 = sg1.stats()["arena_bytes"]
        assert 0 < a1 < a2 <= SCRATCH_BYTES
        assert any(l["kind"] == "reduce" for l in sg1.launches())  # split-K partials in the scratch
        _static_vs_run(sg2, wl2, s)
        _static_vs_run(sg1, wl1, s)   # smaller input on the larger call's leftovers
        _static_vs_run(sg2, wl2, s)
    finally:
        sg1.close()
        sg2.close()


def test_run_static_dense_stack():
    announce("run_static: bert_ffn 2 layers, 40 tokens")
    s = torch.cuda.Stream(device=DEV)
    wl = workloads.bert_ffn(batch=1, seq=40, layers=2)
    sg = capi.Subgraph(wl.graph, wl.consts, device=0)
    try:
        _static_vs_run(sg, wl, s)
        _static_vs_run(sg, wl, s)
    finally:
        sg.close()


def test_run_static_rejects_engine_beyond_scratch():
    announce("run_static: resnet50_v1 bs32 rejected (arena > scratch)")
    wl, sg = _engine("resnet50_v1", 32)
    try:
        assert sg.stats()["arena_bytes"] > SCRATCH_BYTES
        ins = runtime.inputs_for(sg, wl.inputs, DEV)
        out = runtime.outputs_for(sg, DEV)
        out[0].fill_(-3.0)
        torch.cuda.synchronize()
        with pytest.raises(capi.ByocError) as ei:
            sg.run_static(ins, out)
        assert ei.value.status_name == "INVALID_ARG" and "static scratch" in str(ei.value)
        torch.cuda.synchronize()
        assert torch.all(out[0] == -3.0)   # nothing was enqueued
    finally:
        sg.close()
