"""Pins of the oracle's subgraph executor.

The executor is checked against composite chains written out by hand from
the pure-Python brute force (and, for bf16 storage, the separately pinned
rounding), the whole single-composite fp32 workload is pinned by brute force,
and the precision modes are checked for what they must and must not round.
"""

import json

import numpy as np
import pytest

import oracle
from oracle import brute, graph
from oracle.bf16 import round_bf16
from paper_2105_03215_amd import workloads


def test_parse_composite_names():
    p = graph.parse_composite
    assert p("conv2d_bias_relu") == ("conv2d", True, False, "relu")
    assert p("conv2d_bias_add_relu") == ("conv2d", True, True, "relu")
    assert p("conv2d_bias") == ("conv2d", True, False, None)
    assert p("conv2d") == ("conv2d", False, False, None)
    assert p("conv2d_bias_relu6") == ("conv2d", True, False, "relu6")
    assert p("dense_bias_gelu") == ("dense", True, False, "gelu")
    assert p("dense_bias_add") == ("dense", True, True, None)
    assert p("add_relu") == ("add", False, True, "relu")
    assert p("max_pool2d") == ("max_pool2d", False, False, None)
    assert p("global_avg_pool2d") == ("global_avg_pool2d", False, False, None)
    for bad in ("conv3d", "conv2d_relu_bias", "dense_foo", "add_bias"):
        with pytest.raises(ValueError):
            p(bad)


def test_single_fp32_workload_by_brute_force():
    wl = workloads.conv_f32()
    out = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="exact")[0]
    x, w, b = wl.inputs[0], wl.consts[0], wl.consts[1]
    ref = np.array(brute.conv2d(x.tolist(), w.tolist(), (1, 1), (1, 1, 1, 1)))
    ref = np.maximum(ref + np.asarray(b, dtype=np.float64).reshape(1, -1, 1, 1), 0.0)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    assert out.shape == (1, 32, 32, 32)


def _chain_graph():
    rng = np.random.default_rng(7)
    x = rng.random((2, 4, 9, 9)).astype(np.float32)
    w0 = (rng.standard_normal((8, 4, 3, 3)) * 0.3).astype(np.float32)
    b0 = (rng.standard_normal(8) * 0.1).astype(np.float32)
    w1 = (rng.standard_normal((8, 8, 1, 1)) * 0.3).astype(np.float32)
    b1 = (rng.standard_normal(8) * 0.1).astype(np.float32)
    wd = (rng.standard_normal((3, 8)) * 0.3).astype(np.float32)
    bd = (rng.standard_normal(3) * 0.1).astype(np.float32)
    g = {
        "format": "byoc-subgraph", "version": 1,
        "inputs": [{"name": "x", "shape": [2, 4, 9, 9], "dtype": "f32", "layout": "NCHW"}],
        "constants": [{"name": n, "index": i, "shape": list(a.shape), "dtype": "f32"}
                      for i, (n, a) in enumerate([("w0", w0), ("b0", b0), ("w1", w1), ("b1", b1),
                                                  ("wd", wd), ("bd", bd)])],
        "nodes": [
            {"name": "c0", "composite": "conv2d_bias_relu", "inputs": ["x", "w0", "b0"],
             "attrs": {"strides": [2, 2], "padding": [1, 1, 1, 1], "groups": 1}, "out_dtype": "bf16"},
            {"name": "p0", "composite": "max_pool2d", "inputs": ["c0"],
             "attrs": {"pool_size": [3, 3], "strides": [1, 1], "padding": [1, 1, 1, 1]}, "out_dtype": "bf16"},
            {"name": "c1", "composite": "conv2d_bias_add_relu", "inputs": ["p0", "w1", "b1", "c0"],
             "attrs": {"strides": [1, 1], "padding": [0, 0, 0, 0], "groups": 1}, "out_dtype": "bf16"},
            {"name": "g", "composite": "global_avg_pool2d", "inputs": ["c1"], "out_dtype": "bf16"},
            {"name": "d", "composite": "dense_bias_gelu", "inputs": ["g", "wd", "bd"], "out_dtype": "bf16"},
        ],
        "outputs": [{"name": "d", "dtype": "bf16"}, {"name": "c1", "dtype": "bf16", "layout": "NCHW"}],
    }
    return g, [w0, b0, w1, b1, wd, bd], [x]


def test_chain_matches_hand_composition():
    g, consts, inputs = _chain_graph()
    w0, b0, w1, b1, wd, bd = [np.asarray(a, dtype=np.float64) for a in consts]
    rb = round_bf16
    x = rb(inputs[0].astype(np.float64))  # f32 input into a bf16 graph is cast
    c0 = np.array(brute.conv2d(x.tolist(), rb(w0).tolist(), (2, 2), (1, 1, 1, 1)))
    c0 = rb(np.maximum(c0 + b0.reshape(1, -1, 1, 1), 0))
    p0 = rb(np.array(brute.max_pool2d(c0.tolist(), (3, 3), (1, 1), (1, 1, 1, 1))))
    c1 = np.array(brute.conv2d(p0.tolist(), rb(w1).tolist(), (1, 1), (0, 0, 0, 0)))
    c1 = rb(np.maximum(c1 + b1.reshape(1, -1, 1, 1) + c0, 0))
    gg = rb(np.array(brute.global_avg_pool2d(c1.tolist())))
    d = np.array(brute.dense(gg.tolist(), rb(wd).tolist())) + bd
    d = rb(np.vectorize(brute.gelu)(d))
    out_d, out_c1 = oracle.run_graph(g, consts, inputs, mode="bf16io")
    np.testing.assert_allclose(out_c1, c1, rtol=0, atol=0)
    # the dense sum order differs from the brute force; allow one bf16 ulp
    np.testing.assert_allclose(out_d, d, rtol=2 ** -7, atol=1e-12)


def test_modes_round_what_they_declare():
    g, consts, inputs = _chain_graph()
    (d_io, c1_io), vals = oracle.run_graph(g, consts, inputs, mode="bf16io", keep=True)
    for name in ("c0", "p0", "c1", "g", "d"):
        assert np.array_equal(round_bf16(vals[name]), vals[name])
    (d_ex, c1_ex), vex = oracle.run_graph(g, consts, inputs, mode="exact", keep=True)
    # exact keeps unrounded intermediates; the input cast still applies
    assert not np.array_equal(round_bf16(vex["c0"]), vex["c0"])
    assert np.array_equal(vex["x"], round_bf16(inputs[0]))
    err = np.max(np.abs(d_io - d_ex) / (np.abs(d_ex) + 1))
    assert 0 < err < 1e-2
    with pytest.raises(ValueError):
        oracle.run_graph(g, consts, inputs, mode="fp16")


def test_json_string_and_dict_agree():
    g, consts, inputs = _chain_graph()
    a = oracle.run_graph(json.dumps(g), consts, inputs)
    b = oracle.run_graph(g, consts, inputs)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_run_node_teacher_forced():
    g, consts, inputs = _chain_graph()
    _, vals = oracle.run_graph(g, consts, inputs, keep=True)
    node = g["nodes"][2]
    y = oracle.run_node(node, [vals[r] for r in node["inputs"]])
    assert np.array_equal(y, vals["c1"])


def test_fp32_graph_is_not_rounded():
    wl = workloads.conv_f32(n=1, c=4, hw=6, k=3)
    out = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="bf16io")[0]
    assert not np.array_equal(round_bf16(out), out)


def test_leaky_node_takes_its_slope_from_attrs():
    """A conv2d_bias_leaky node against brute-force loops: the composite's
    pre-activation where it is >= 0, alpha times it below, with alpha read
    from the node's attrs (default 0.1)."""
    rng = np.random.default_rng(21)
    x = rng.normal(size=(1, 2, 5, 4))
    w = rng.normal(size=(3, 2, 3, 3))
    b = rng.normal(size=3)
    pre = np.array(brute.conv2d(x.tolist(), w.tolist(), (1, 1), (1, 1, 1, 1))) + b.reshape(1, 3, 1, 1)
    for attrs, a in (({"padding": [1, 1, 1, 1], "alpha": 0.3}, 0.3), ({"padding": [1, 1, 1, 1]}, 0.1)):
        node = {"name": "y", "composite": "conv2d_bias_leaky", "inputs": ["x", "w", "b"], "attrs": attrs,
                "out_dtype": "f32"}
        y = graph.run_node(node, [x, w, b], mode="exact")
        np.testing.assert_allclose(y, np.where(pre >= 0, pre, a * pre), rtol=1e-12, atol=1e-12)
        assert (pre < 0).any()
