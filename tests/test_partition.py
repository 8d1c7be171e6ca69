"""The partitioner (Sec. 3.1): pattern grouping, annotation, greedy region
merge, cost-based split, host fallback and serialization, on the CPU.

Pins: the region arithmetic of the paper's illustrative example (a region of
4N + 1 operators, split at 3N), the structural invariants (every operator in
exactly one place, an acyclic program, MAC-free regions on the host), the
round trip of the executor's own workloads (lowered to operators and
regrouped into the same composites), and semantics: the partitioned program
(offloaded functions through the oracle's executor of the serialized form,
host steps by reference) equals the operator-by-operator execution of the
unpartitioned graph.
"""

import numpy as np
import pytest

from oracle.bf16 import round_bf16
from paper_2105_03215_amd import capi, partition as P, workloads
from ir_ref import run_ir, run_partitioned


def _rng(seed):
    return np.random.default_rng(seed)


def _conv(g, x, k, r, rng, stride=1, bias=True, act="relu", residual=None, groups=1, residual_first=False):
    c = g.nodes[x].shape[1]
    w = g.const(rng.normal(0, (2.0 / (c // groups * r * r)) ** 0.5, size=(k, c // groups, r, r)))
    y = g.call("nn.conv2d", [x, w], strides=[stride, stride], padding=[r // 2] * 4, groups=groups)
    if bias:
        y = g.call("nn.bias_add", [y, g.const(rng.normal(0, 0.1, size=k))])
    if residual is not None:
        y = g.call("add", [residual, y] if residual_first else [y, residual])
    if act == "relu":
        y = g.call("nn.relu", [y])
    elif act == "relu6":
        y = g.call("clip", [y], a_min=0.0, a_max=6.0)
    return y


def fig3_graph(n_blocks, seed=0):
    """Region 1: n_blocks residual conv blocks (conv2d, bias_add, add, relu:
    4 operators each) and one plain conv2d, 4N + 1 operators; then an
    operator no target supports (sigmoid); then Region 2: a conv2d_bias_relu
    pattern (3 operators) and a max pool."""
    rng = _rng(seed)
    g = P.Graph()
    x = g.input("x", [1, 8, 8, 8])
    for _ in range(n_blocks):
        x = _conv(g, x, 8, 3, rng, residual=x)
    x = _conv(g, x, 8, 1, rng, bias=False, act=None)
    x = g.call("sigmoid", [x])
    x = _conv(g, x, 8, 3, rng)
    x = g.call("nn.max_pool2d", [x], pool_size=[3, 3], strides=[2, 2], padding=[1, 1, 1, 1])
    g.output(x)
    return g


def _placement_counts(part):
    g = part.graph
    seen = {}
    for f in part.functions:
        for u in f.units:
            for m in u.members:
                seen[m] = seen.get(m, 0) + 1
    for kind, ref in part.steps:
        if kind == "host":
            seen[ref] = seen.get(ref, 0) + 1
    ops = [n.id for n in g.nodes if n.op not in ("input", "const")]
    return seen, ops


def _check_invariants(part):
    seen, ops = _placement_counts(part)
    assert sorted(seen) == sorted(ops), "every operator placed"
    assert all(v == 1 for v in seen.values()), "no operator placed twice"
    # the program order is a topological order: every input is defined first
    g = part.graph
    defined = set(g.inputs) | {n.id for n in g.nodes if n.op == "const"}
    for kind, ref in part.steps:
        if kind == "host":
            assert all(i in defined for i in g.nodes[ref].inputs)
            defined.add(ref)
        else:
            f = part.functions[ref]
            assert all(i in defined for i in f.inputs)
            defined.update(m for u in f.units for m in u.members)
    assert all(o in defined for o in g.outputs)


@pytest.mark.parametrize("n", [1, 4, 6])
def test_fig3_region_arithmetic(n):
    g = fig3_graph(n)
    part = P.partition(g)
    sizes = [f.n_ops for f in part.functions]
    assert sizes == [4 * n + 1, 4], sizes
    assert [g.nodes[r].op for k, r in part.steps if k == "host"] == ["sigmoid"]
    _check_invariants(part)
    # cost-based split at 3N operators: region 1 -> 3N + (N + 1) when 3N
    # holds whole composites (N a multiple of 4), else the largest prefix
    split = P.partition(g, max_ops=3 * n)
    sizes = [f.n_ops for f in split.functions]
    assert all(s <= max(3 * n, 4) for s in sizes)  # a composite (4 operators) is never cut
    # pieces without MACs (a lone max pool) fall back to the host
    host = [g.nodes[r].op for k, r in split.steps if k == "host"]
    assert sum(sizes) + len(host) - 1 == 4 * n + 1 + 4
    assert set(host) <= {"sigmoid", "nn.max_pool2d"}
    if n % 4 == 0:
        assert sizes[:2] == [3 * n, n + 1]
    _check_invariants(split)


def test_fig3_composites_named_by_pattern():
    part = P.partition(fig3_graph(2))
    names = [n["composite"] for n in part.functions[0].graph["nodes"]]
    assert names == ["conv2d_bias_add_relu", "conv2d_bias_add_relu", "conv2d"]
    names = [n["composite"] for n in part.functions[1].graph["nodes"]]
    assert names == ["conv2d_bias_relu", "max_pool2d"]


def test_host_fallback_mac_free_region():
    """A region with no MACs stays on the host (CalcMAC(region) > 0)."""
    rng = _rng(1)
    g = P.Graph()
    x = g.input("x", [1, 4, 9, 9])
    y = g.call("sigmoid", [x])
    y = g.call("nn.max_pool2d", [y], pool_size=[3, 3], strides=[2, 2], padding=[1, 1, 1, 1])
    y = g.call("sigmoid", [y])
    y = _conv(g, y, 8, 3, rng)
    g.output(y)
    part = P.partition(g)
    assert [f.n_ops for f in part.functions] == [3]
    assert [g.nodes[r].op for k, r in part.steps if k == "host"] == ["sigmoid", "nn.max_pool2d", "sigmoid"]
    # with a criterion that keeps everything, the pool is offloaded alone
    keep_all = P.partition(g, keep=lambda gr, us: True)
    assert sorted(f.n_ops for f in keep_all.functions) == [1, 3]
    _check_invariants(part)
    _check_invariants(keep_all)


def test_shared_intermediate_is_not_fused():
    """An operator whose result is also used outside the sequence cannot be
    fused: the conv stays a composite of its own, the bias_add and relu that
    follow have no executor kernel alone and run on the host."""
    rng = _rng(2)
    g = P.Graph()
    x = g.input("x", [1, 4, 6, 6])
    w = g.const(rng.normal(0, 0.3, size=(4, 4, 3, 3)))
    c = g.call("nn.conv2d", [x, w], strides=[1, 1], padding=[1, 1, 1, 1])
    b = g.call("nn.bias_add", [c, g.const(rng.normal(0, 0.1, size=4))])
    r = g.call("nn.relu", [b])
    s = g.call("add", [c, r])
    g.output(s)
    comps, owner = P.merge_composites(g)
    assert comps[c].name == "conv2d"
    assert b not in owner and r not in owner
    part = P.partition(g)
    _check_invariants(part)


def test_residual_in_either_operand_order():
    rng = _rng(3)
    g = P.Graph()
    x = g.input("x", [2, 8, 5, 5])
    a = _conv(g, x, 8, 3, rng, residual=x, residual_first=True)
    b = _conv(g, a, 8, 1, rng, residual=a, act="relu6")
    g.output(b)
    part = P.partition(g)
    names = [n["composite"] for n in part.functions[0].graph["nodes"]]
    assert names == ["conv2d_bias_add_relu", "conv2d_bias_add_relu6"]


def _mixed_graph(seed=5):
    """A small f32 network touching every pattern, an unsupported operator in
    the middle and a host head."""
    rng = _rng(seed)
    g = P.Graph()
    x = g.input("x", [2, 3, 17, 15])
    y = _conv(g, x, 16, 3, rng, stride=2)
    y = g.call("nn.max_pool2d", [y], pool_size=[3, 3], strides=[2, 2], padding=[1, 1, 1, 1])
    a = _conv(g, y, 16, 1, rng, act="relu6")
    a = _conv(g, a, 16, 3, rng, groups=16, act="relu6")
    y = _conv(g, a, 16, 1, rng, act=None, residual=y)
    y = g.call("add", [y, _conv(g, y, 16, 3, rng)])
    y = g.call("nn.relu", [y])
    y = g.call("sigmoid", [y])
    y = _conv(g, y, 24, 3, rng, stride=2)
    y = g.call("nn.batch_flatten", [g.call("nn.global_avg_pool2d", [y])])
    w = g.const(rng.normal(0, 0.2, size=(10, 24)))
    y = g.call("nn.dense", [y, w])
    y = g.call("nn.bias_add", [y, g.const(rng.normal(0, 0.1, size=10))])
    y = g.call("nn.gelu", [y])
    y = g.call("nn.softmax", [y], axis=-1)
    g.output(y)
    return g


@pytest.mark.parametrize("max_ops", [None, 4, 9])
def test_partitioned_program_equals_graph(max_ops):
    g = _mixed_graph()
    x = _rng(9).random((2, 3, 17, 15))
    ref = run_ir(g, [x])[0]
    part = P.partition(g, max_ops=max_ops)
    _check_invariants(part)
    got = run_partitioned(part, [x], mode="exact")[0]
    assert np.max(np.abs(got - ref)) <= 1e-10 * max(1.0, np.max(np.abs(ref)))
    st = part.stats()
    assert st["mac_offload"] == 1.0
    assert st["offloaded_operators"] + sum(1 for k, _ in part.steps if k == "host") == st["operators"]


def test_functions_validate_in_the_executor():
    """Every serialized function passes the C library's validation (host
    only, no device needed)."""
    for max_ops in (None, 5):
        part = P.partition(_mixed_graph(), max_ops=max_ops)
        for f in part.functions:
            capi.validate(f.graph, f.consts)


@pytest.mark.parametrize("name,kw", [("resnet50_v1", {"n": 1, "hw": 64}), ("mobilenet_v2", {"n": 1, "hw": 64}),
                                     ("resnet18_block", {"n": 1, "c": 64, "hw": 14}),
                                     ("bert_ffn", {"batch": 1, "seq": 8, "layers": 3}),
                                     ("vgg19", {"n": 1, "hw": 32}), ("darknet53", {"n": 1, "hw": 64}),
                                     ("inception_v3", {"n": 1, "hw": 75})])
def test_workload_round_trip(name, kw):
    """The executor's workloads lowered to operators and partitioned with a
    host softmax head come back as one function with the same composites, in
    the same order, with every operator and MAC offloaded but the head."""
    wl = workloads.build(name, **kw)
    g = P.lower_subgraph(wl.graph, wl.consts)
    out = g.outputs[0]
    if len(g.nodes[out].shape) == 2:
        g.outputs = [g.call("nn.softmax", [out], axis=-1)]
    part = P.partition(g)
    assert len(part.functions) == 1
    f = part.functions[0]
    assert [n["composite"] for n in f.graph["nodes"]] == [n["composite"] for n in wl.graph["nodes"]]
    assert f.macs == wl.macs
    st = part.stats()
    assert st["mac_offload"] == 1.0
    _check_invariants(part)
    capi.validate(f.graph, f.consts)


def _inception_like_graph(seed=11, odd=False):
    """Branches joined by concatenation (one branch an average pool), leaky
    ReLU convs, a concatenation of a 6-channel tensor (not offloadable: the
    executor joins multiples of 8 channels) when ``odd``."""
    rng = _rng(seed)
    g = P.Graph()
    x = g.input("x", [2, 16, 9, 9], dtype="bf16")
    a = _conv(g, x, 16, 1, rng)
    b = _conv(g, _conv(g, x, 8, 1, rng), 24, 3, rng)
    p = g.call("nn.avg_pool2d", [x], pool_size=[3, 3], strides=[1, 1], padding=[1, 1, 1, 1],
               count_include_pad=False)
    p = _conv(g, p, 8, 1, rng)
    cat = g.call("concatenate", [a, b, p], axis=1)
    w = g.const(rng.normal(0, 0.2, size=(16, 48, 3, 3)))
    y = g.call("nn.conv2d", [cat, w], strides=[2, 2], padding=[1, 1, 1, 1])
    y = g.call("nn.bias_add", [y, g.const(rng.normal(0, 0.1, size=16))])
    y = g.call("nn.leaky_relu", [y], alpha=0.2)
    if odd:
        s6 = _conv(g, y, 6, 1, rng)
        y = g.call("concatenate", [y, s6], axis=1)
    g.output(y)
    # a bf16 function computes with bf16 weights: make the constants
    # bf16 values so that the operator-level reference uses the same ones
    for n in g.nodes:
        if n.op == "const":
            n.value = round_bf16(n.value).astype(np.float32)
    return g


@pytest.mark.parametrize("odd", [False, True])
def test_concat_avgpool_leaky_partition_semantics(odd):
    g = _inception_like_graph(odd=odd)
    x = round_bf16(_rng(12).random((2, 16, 9, 9)))
    ref = run_ir(g, [x])[0]
    part = P.partition(g)
    _check_invariants(part)
    names = [n["composite"] for f in part.functions for n in f.graph["nodes"]]
    assert "concatenate" in names and "avg_pool2d" in names and "conv2d_bias_leaky" in names
    host = [g.nodes[r].op for k, r in part.steps if k == "host"]
    assert host == (["concatenate"] if odd else [])
    got = run_partitioned(part, [x], mode="exact")[0]
    assert np.max(np.abs(got - ref)) <= 1e-10 * max(1.0, np.max(np.abs(ref)))
    for f in part.functions:
        capi.validate(f.graph, f.consts)
    leaky = [n for f in part.functions for n in f.graph["nodes"] if n["composite"] == "conv2d_bias_leaky"]
    assert leaky[0]["attrs"]["alpha"] == 0.2
