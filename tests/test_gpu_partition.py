"""Partitioned models on the GPU (Sec. 3.4): host steps in PyTorch, the
offloaded functions through the HIP library's cached engines, against the
partitioned program on the oracle (bf16 storage semantics, host results
stored as bf16 like the runtime does)."""

import numpy as np
import pytest
import torch

from paper_2105_03215_amd import host_runtime, partition as P, runtime, workloads
from ir_ref import run_partitioned
from parity_util import BF16_TOL, announce, rel_err
from test_partition import _inception_like_graph, _mixed_graph

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _bf16_graph(g):
    """The same graph with bf16 activations (inputs declared bf16)."""
    for i in g.inputs:
        g.nodes[i].dtype = "bf16"
    for n in g.nodes:
        if n.op not in ("input", "const"):
            n.dtype = "bf16"
    return g


def _check(g, inputs, max_ops=None, runs=2, graph_replay=False):
    part = P.partition(g, max_ops=max_ops)
    ref = run_partitioned(part, inputs, mode="bf16io")
    mod = host_runtime.Module(part, DEV, graph_replay=graph_replay)
    try:
        xs = [torch.from_numpy(np.asarray(x, np.float32)).to(DEV) for x in inputs]
        first = None
        for _ in range(runs):
            outs = mod.run(xs)
            torch.cuda.synchronize()
            got = [runtime.to_host_f64(o) for o in outs]
            if first is None:
                first = got
            else:  # cached engines, same data entries: identical results
                for a, b in zip(first, got):
                    assert np.array_equal(a, b)
        for gv, rv in zip(first, ref):
            assert rel_err(gv, rv) <= BF16_TOL, rel_err(gv, rv)
    finally:
        mod.close()
    return part


@pytest.mark.parametrize("max_ops,replay", [(None, False), (4, False), (4, True)])
def test_mixed_graph_partitioned(max_ops, replay):
    """Host steps between several functions; with graph replay the
    functions' engines replay their launch sequences on the module's fixed
    data entries (three runs, identical results)."""
    announce("partitioned mixed graph max_ops=%s replay=%s" % (max_ops, replay))
    g = _bf16_graph(_mixed_graph())
    x = workloads.to_bf16_values(np.random.default_rng(11).random((2, 3, 17, 15)).astype(np.float32))
    part = _check(g, [x], max_ops=max_ops, runs=3 if replay else 2, graph_replay=replay)
    assert len(part.functions) >= 2
    assert any(k == "host" for k, _ in part.steps)


def test_resnet50_with_host_head():
    """ResNet-50 lowered to operators, a softmax head on the host: one
    offloaded function with every conv, then the host step."""
    announce("partitioned resnet50 + softmax")
    wl = workloads.build("resnet50_v1", n=2, hw=64)
    g = P.lower_subgraph(wl.graph, wl.consts)
    g.outputs = [g.call("nn.softmax", [g.outputs[0]], axis=-1)]
    part = _check(g, wl.inputs)
    assert len(part.functions) == 1 and part.steps[-1][0] == "host"


def test_concat_graph_with_host_concatenation():
    """Concatenations in place and copied, an average pool and leaky ReLU
    offloaded; a concatenation the executor rejects (6 channels) runs on
    the host between the functions' outputs."""
    announce("partitioned inception-like graph with a host concatenation")
    g = _inception_like_graph(odd=True)
    x = workloads.to_bf16_values(np.random.default_rng(13).random((2, 16, 9, 9)).astype(np.float32))
    part = _check(g, [x])
    assert [g.nodes[r].op for k, r in part.steps if k == "host"] == ["concatenate"]
