"""Partially quantized (int8) subgraphs on the GPU against the int8 oracle.

Every int8 composite is exact integer arithmetic followed by one fixed-point
rounding, so the executor's outputs (dequantized to float32, a one-to-one
map of the codes) must equal the oracle's bit for bit.  Cases span aligned
(128-channel stages) and unaligned reductions, ragged channel counts, every
tile shape, the border correction of a nonzero input zero point under
padding, strides, residuals, ReLU / ReLU6, pools, the standalone add and the
boundary quantize / dequantize; the ResNet-50 case runs at batch 32 and
224x224 (the benchmark's configuration).  The scales and zero points of
the network cases are calibrated on the oracle's float values of the
calibration images, so the quantized function both sides receive holds
nothing the GPU computed.
"""

import copy

import numpy as np
import pytest

import oracle
from oracle import quant as OQ
from paper_2105_03215_amd import workloads
from parity_util import announce, oracle_calibrated_int8

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _run(graph, consts, inputs):
    from paper_2105_03215_amd import capi, runtime
    sg = capi.Subgraph(graph, consts, device=0)
    try:
        return runtime.run_once(sg, inputs, DEV), sg.launches()
    finally:
        sg.close()


def _q(s, z):
    return {"scale": float(s), "zero_point": int(z)}


def _conv_graph(n, c, h, w, k, r, stride, pad, zx, act, residual, bias=True, seed=0):
    rng = np.random.default_rng(seed)
    wt = rng.normal(0, (2.0 / (c * r * r)) ** 0.5, size=(k, c, r, r)).astype(np.float32)
    consts = [wt]
    cdesc = [{"name": "w", "index": 0, "shape": list(wt.shape), "dtype": "f32"}]
    ins = ["x", "w"]
    if bias:
        consts.append(rng.normal(0, 0.2, size=k).astype(np.float32))
        cdesc.append({"name": "b", "index": 1, "shape": [k], "dtype": "f32"})
        ins.append("b")
    p = (h + 2 * pad - r) // stride + 1
    q = (w + 2 * pad - r) // stride + 1
    inputs_desc = [{"name": "x", "shape": [n, c, h, w], "dtype": "f32", "quant": _q(0.011, zx)}]
    inputs = [rng.uniform(-1.2, 1.7, size=(n, c, h, w)).astype(np.float32)]
    if residual:
        inputs_desc.append({"name": "r", "shape": [n, k, p, q], "dtype": "f32", "quant": _q(0.019, -7)})
        inputs.append(rng.normal(0, 1, size=(n, k, p, q)).astype(np.float32))
        ins.append("r")
    comp = "conv2d" + ("_bias" if bias else "") + ("_add" if residual else "") + ("_" + act if act else "")
    g = {"format": "byoc-subgraph", "version": 1, "inputs": inputs_desc, "constants": cdesc,
         "nodes": [{"name": "y", "composite": comp, "inputs": ins, "out_dtype": "int8",
                    "attrs": {"strides": [stride, stride], "padding": [pad] * 4}, "quant": _q(0.023, -11)}],
         "outputs": [{"name": "y", "dtype": "f32"}]}
    return g, consts, inputs


CONV_CASES = [
    # n, c, h, w, k, r, stride, pad, zx, act, residual
    (2, 128, 14, 14, 128, 3, 1, 1, 0, "relu", False),      # aligned, interior + border, Z_x = 0
    (2, 128, 14, 13, 192, 3, 1, 1, 37, "relu", True),      # aligned, border correction, residual
    (1, 200, 9, 11, 72, 3, 2, 1, -100, None, False),       # unaligned ragged channels, stride 2
    (3, 3, 30, 30, 64, 7, 2, 3, 5, "relu", False),         # stem-like: 3 channels, 7x7
    (4, 256, 8, 8, 512, 1, 2, 0, 64, None, True),          # 1x1 stride 2 projection, residual
    (1, 64, 56, 56, 256, 1, 1, 0, -128, "relu6", False),  # many pixels: 128x128 tiles
    (2, 48, 5, 5, 40, 5, 1, 2, 90, "relu6", True),         # tiny image, every pixel on the border
    (2, 128, 14, 13, 136, 3, 1, 1, -40, "leaky", True),    # leaky ReLU on codes, residual
    (1, 64, 28, 28, 128, 1, 1, 0, 12, "leaky", False),     # leaky ReLU, 1x1
]


@pytest.mark.parametrize("case", CONV_CASES, ids=[str(i) for i in range(len(CONV_CASES))])
def test_int8_conv_bit_exact(case):
    n, c, h, w, k, r, stride, pad, zx, act, residual = case
    announce("int8 conv %s" % (case,))
    g, consts, inputs = _conv_graph(n, c, h, w, k, r, stride, pad, zx, act, residual, seed=len(str(case)))
    got, launches = _run(g, consts, inputs)
    assert any(l["kind"] == "conv_i8" for l in launches)
    ref = OQ.run_quantized_graph(g, consts, inputs)
    assert got[0].shape == ref[0].shape
    assert np.array_equal(got[0], ref[0].astype(np.float64)), np.abs(got[0] - ref[0]).max()


def test_int8_tiles_agree():
    """Every tile shape and ring depth gives the same codes (integer sums)."""
    announce("int8 conv every tile")
    import os
    g, consts, inputs = _conv_graph(2, 144, 12, 12, 136, 3, 1, 1, 21, "relu", True, seed=3)
    ref = OQ.run_quantized_graph(g, consts, inputs)[0]
    for tile in ("128x128s2w4", "128x64s4w4", "64x64s3w4", "32x64s2w4", "128x128s2w8", "128x64s3w8", "64x128s4w8"):
        os.environ["BYOC_I8_TILE"] = tile
        try:
            got, launches = _run(g, consts, inputs)
        finally:
            del os.environ["BYOC_I8_TILE"]
        name = [l["name"] for l in launches if l["kind"] == "conv_i8"][0]
        assert name == "conv_i8_" + tile.replace("s", "_s").replace("w", "_w"), name
        assert np.array_equal(got[0], ref.astype(np.float64)), tile


# 2 or 4 reduction groups (threads = 256 per group): each group sums every
# 2nd / 4th stage, the int32 sums are added in the epilogue
KG_TILES = ("64x64s3w8k2", "64x64s4w8k2", "32x64s4w8k2", "128x64s2w8k2", "128x64s3w8k2", "64x64s2w16k4",
            "32x64s3w16k4")
KG_CASES = [
    # n, c, h, w, k, r, stride, pad, zx, act, residual: 144 channels (reduction not in whole 128-code
    # stages, a ragged last stage per group), 256 channels 3x3 (aligned, 18 stages), a 1x1 with 7 stages
    (2, 144, 12, 12, 136, 3, 1, 1, 21, "relu", True),
    (2, 256, 7, 7, 200, 3, 1, 1, -7, "relu6", False),
    (3, 896, 5, 5, 72, 1, 1, 0, 3, None, True),
]


@pytest.mark.parametrize("case", KG_CASES, ids=["c%d_r%d" % (c[1], c[5]) for c in KG_CASES])
def test_int8_reduction_groups_exact(case):
    """Every reduction-group tile gives the oracle's codes exactly."""
    announce("int8 conv reduction groups %s" % (case,))
    import os
    g, consts, inputs = _conv_graph(*case, seed=60 + KG_CASES.index(case))
    ref = OQ.run_quantized_graph(g, consts, inputs)[0]
    for tile in KG_TILES:
        os.environ["BYOC_I8_TILE"] = tile
        try:
            got, launches = _run(g, consts, inputs)
        finally:
            del os.environ["BYOC_I8_TILE"]
        name = [l["name"] for l in launches if l["kind"] == "conv_i8"][0]
        assert name == "conv_i8_" + tile.replace("s", "_s").replace("w", "_w").replace("k", "_k"), name
        assert np.array_equal(got[0], ref.astype(np.float64)), tile


def test_int8_dense_pool_add():
    announce("int8 dense, pools, add")
    rng = np.random.default_rng(7)
    wd = rng.normal(0, 0.1, size=(1000, 96)).astype(np.float32)
    bd = rng.normal(0, 0.1, size=1000).astype(np.float32)
    g = {"format": "byoc-subgraph", "version": 1,
         "inputs": [{"name": "x", "shape": [5, 96, 9, 7], "dtype": "bf16", "quant": _q(0.02, -3)},
                    {"name": "z", "shape": [5, 96, 9, 7], "dtype": "f32", "quant": _q(0.03, 40)}],
         "constants": [{"name": "wd", "index": 0, "shape": [1000, 96], "dtype": "f32"},
                       {"name": "bd", "index": 1, "shape": [1000], "dtype": "f32"}],
         "nodes": [
             {"name": "a", "composite": "add_relu", "inputs": ["x", "z"], "out_dtype": "int8", "quant": _q(0.04, -128)},
             {"name": "m", "composite": "max_pool2d", "inputs": ["a"], "out_dtype": "int8",
              "attrs": {"pool_size": [3, 3], "strides": [2, 2], "padding": [1, 1, 1, 1]}},
             {"name": "p", "composite": "global_avg_pool2d", "inputs": ["m"], "out_dtype": "int8",
              "quant": _q(0.01, -120)},
             {"name": "d", "composite": "dense_bias", "inputs": ["p", "wd", "bd"], "out_dtype": "int8",
              "quant": _q(0.05, 2)}],
         "outputs": [{"name": "d", "dtype": "f32"}, {"name": "m", "dtype": "f32"}, {"name": "a", "dtype": "bf16"}]}
    x = oracle.bf16.round_bf16(rng.normal(0, 1, size=(5, 96, 9, 7))).astype(np.float32)
    z = rng.normal(0, 1, size=(5, 96, 9, 7)).astype(np.float32)
    got, _ = _run(g, [wd, bd], [x, z])
    ref = OQ.run_quantized_graph(g, [wd, bd], [x, z])
    for i in range(2):
        assert np.array_equal(got[i], ref[i].astype(np.float64)), i
    # a bf16 output is the float32 dequantized value rounded to bf16
    assert np.array_equal(got[2], oracle.bf16.round_bf16(ref[2].astype(np.float64)))


def test_int8_two_runs_and_bs1_graph():
    """The tiny mixed graph twice on one engine: identical results."""
    from paper_2105_03215_amd import capi, runtime
    import test_oracle_quant as T
    announce("int8 tiny graph twice")
    g, consts = T._tiny_int8_graph()
    x = np.random.default_rng(12).random((2, 3, 9, 9)).astype(np.float32)
    sg = capi.Subgraph(g, consts, device=0)
    try:
        a = runtime.run_once(sg, [x], DEV)[0]
        b = runtime.run_once(sg, [x], DEV)[0]
    finally:
        sg.close()
    ref = OQ.run_quantized_graph(g, consts, [x])[0]
    assert np.array_equal(a, ref.astype(np.float64)) and np.array_equal(a, b)


def _calibrated_resnet50(n, hw, calib_n=2):
    wl = workloads.build("resnet50_v1", n=n, hw=hw)
    qg = oracle_calibrated_int8(wl.graph, wl.consts, [np.ascontiguousarray(a[:calib_n]) for a in wl.inputs])
    return wl, qg


def test_int8_resnet50_small_full_compare():
    announce("int8 resnet50 n=2 hw=64")
    wl, qg = _calibrated_resnet50(2, 64)
    got, launches = _run(qg, wl.consts, wl.inputs)
    ref = OQ.run_quantized_graph(qg, wl.consts, wl.inputs)[0]
    assert np.array_equal(got[0], ref.astype(np.float64))
    assert sum(1 for l in launches if l["kind"] == "conv_i8") == 54
    # the int8 network tracks the bf16 one (a sanity bound on calibration)
    fl = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="bf16io")[0]
    assert np.corrcoef(got[0].ravel(), fl.ravel())[0, 1] > 0.9


def test_int8_resnet50_bs32_sampled():
    announce("int8 resnet50 bs32 224 sampled images 0 and 31")
    wl, qg = _calibrated_resnet50(32, 224)
    got, _ = _run(qg, wl.consts, wl.inputs)
    rows = [0, 31]
    g2 = copy.deepcopy(qg)
    g2["inputs"] = [dict(d, shape=[2] + d["shape"][1:]) for d in g2["inputs"]]
    ref = OQ.run_quantized_graph(g2, wl.consts, [np.ascontiguousarray(a[rows]) for a in wl.inputs])[0]
    assert np.array_equal(got[0][rows], ref.astype(np.float64))


DW_CASES = [
    # n, c, h, w, stride, zx, act, residual
    (2, 32, 13, 11, 1, 17, "relu6", False),
    (1, 96, 14, 14, 2, -128, "relu6", False),
    (2, 40, 7, 9, 1, 60, None, True),
    (1, 48, 10, 10, 1, -5, "leaky", True),
]


@pytest.mark.parametrize("case", DW_CASES, ids=[str(i) for i in range(len(DW_CASES))])
def test_int8_depthwise_bit_exact(case):
    n, c, h, w, stride, zx, act, residual = case
    announce("int8 depthwise %s" % (case,))
    rng = np.random.default_rng(30 + DW_CASES.index(case))
    wt = rng.normal(0, 0.4, size=(c, 1, 3, 3)).astype(np.float32)
    b = rng.normal(0, 0.2, size=c).astype(np.float32)
    p = (h + 2 - 3) // stride + 1
    q = (w + 2 - 3) // stride + 1
    ins_desc = [{"name": "x", "shape": [n, c, h, w], "dtype": "f32", "quant": _q(0.013, zx)}]
    inputs = [rng.uniform(-1.0, 2.0, size=(n, c, h, w)).astype(np.float32)]
    refs = ["x", "w", "b"]
    if residual:
        ins_desc.append({"name": "r", "shape": [n, c, p, q], "dtype": "f32", "quant": _q(0.02, 3)})
        inputs.append(rng.normal(0, 1, size=(n, c, p, q)).astype(np.float32))
        refs.append("r")
    comp = "conv2d_bias" + ("_add" if residual else "") + ("_" + act if act else "")
    g = {"format": "byoc-subgraph", "version": 1, "inputs": ins_desc,
         "constants": [{"name": "w", "index": 0, "shape": [c, 1, 3, 3], "dtype": "f32"},
                       {"name": "b", "index": 1, "shape": [c], "dtype": "f32"}],
         "nodes": [{"name": "y", "composite": comp, "inputs": refs, "out_dtype": "int8",
                    "attrs": {"strides": [stride, stride], "padding": [1, 1, 1, 1], "groups": c},
                    "quant": _q(0.03, -20)}],
         "outputs": [{"name": "y", "dtype": "f32"}]}
    got, launches = _run(g, [wt, b], inputs)
    assert any(l["name"] == "depthwise_nhwc_i8" for l in launches)
    ref = OQ.run_quantized_graph(g, [wt, b], inputs)[0]
    assert np.array_equal(got[0], ref.astype(np.float64))


def test_int8_mobilenet_v2_small_full_compare():
    announce("int8 mobilenet_v2 n=2 hw=64")
    wl = workloads.build("mobilenet_v2", n=2, hw=64)
    qg = oracle_calibrated_int8(wl.graph, wl.consts, wl.inputs)
    got, launches = _run(qg, wl.consts, wl.inputs)
    assert sum(1 for l in launches if l["name"] == "depthwise_nhwc_i8") == 17
    ref = OQ.run_quantized_graph(qg, wl.consts, wl.inputs)[0]
    assert np.array_equal(got[0], ref.astype(np.float64))


def test_int8_vgg19_small_full_compare():
    """VGG19 (2x2 max pools, the full-map fc6 conv, dense classifier) in int8."""
    announce("int8 vgg19 n=2 hw=64")
    wl = workloads.build("vgg19", n=2, hw=64)
    qg = oracle_calibrated_int8(wl.graph, wl.consts, wl.inputs)
    got, launches = _run(qg, wl.consts, wl.inputs)
    assert sum(1 for l in launches if l["kind"] == "conv_i8") == 19
    ref = OQ.run_quantized_graph(qg, wl.consts, wl.inputs)[0]
    assert np.array_equal(got[0], ref.astype(np.float64))


def test_int8_leaky_slopes_conv_and_add():
    """Leaky ReLU on codes with non-default slopes, in a conv and an add."""
    announce("int8 leaky slopes 0.3 (conv), 0.25 (add)")
    g, consts, inputs = _conv_graph(2, 64, 9, 9, 64, 3, 1, 1, 33, "leaky", False, seed=11)
    g["nodes"][0]["attrs"]["alpha"] = 0.3
    g["nodes"].append({"name": "s", "composite": "add_leaky", "inputs": ["y", "y2"], "out_dtype": "int8",
                       "attrs": {"alpha": 0.25}, "quant": _q(0.031, 14)})
    g["nodes"].insert(1, {"name": "y2", "composite": "conv2d_leaky", "inputs": ["y", "w"], "out_dtype": "int8",
                          "attrs": {"strides": [1, 1], "padding": [1, 1, 1, 1], "alpha": 0.05},
                          "quant": _q(0.027, -60)})
    g["outputs"] = [{"name": "s", "dtype": "f32"}, {"name": "y", "dtype": "f32"}]
    got, launches = _run(g, consts, inputs)
    assert any(l["name"] == "add_i8" for l in launches), [l["name"] for l in launches]
    ref = OQ.run_quantized_graph(g, consts, inputs)
    for i in range(2):
        assert np.array_equal(got[i], ref[i].astype(np.float64)), i


def test_int8_darknet53_small_full_compare():
    """DarkNet-53 (leaky ReLU after every conv, residual adds) in int8."""
    announce("int8 darknet53 n=2 hw=64")
    wl = workloads.build("darknet53", n=2, hw=64)
    qg = oracle_calibrated_int8(wl.graph, wl.consts, wl.inputs)
    got, launches = _run(qg, wl.consts, wl.inputs)
    assert sum(1 for l in launches if l["kind"] == "conv_i8") >= 52
    # every residual add follows a conv's leaky ReLU and is folded into it
    assert not any(l["name"] == "add_i8" for l in launches)
    ref = OQ.run_quantized_graph(qg, wl.consts, wl.inputs)[0]
    assert np.array_equal(got[0], ref.astype(np.float64))
    import os
    os.environ["BYOC_FUSE_POST_ADD"] = "0"
    try:
        plain, plain_launches = _run(qg, wl.consts, wl.inputs)
    finally:
        del os.environ["BYOC_FUSE_POST_ADD"]
    assert sum(1 for l in plain_launches if l["name"] == "add_i8") == 23
    assert np.array_equal(plain[0], got[0])


STEM_I8_CASES = [
    # name, (n, c, h, w), r, stride, pad, act, (pool size, stride, pad), input dtype, persistent workgroups
    ("resnet_stem_224", (2, 3, 224, 224), 7, 2, 3, "relu", (3, 2, 1), "f32", 0),
    ("resnet_stem_ragged", (2, 3, 45, 45), 7, 2, 3, "relu", (3, 2, 1), "f32", 0),
    ("stem_bf16_in_c1", (1, 1, 32, 30), 7, 2, 3, "relu", (3, 2, 1), "bf16", 0),
    ("stem_3x3_s1_pool2", (2, 4, 20, 21), 3, 1, 1, None, (2, 2, 0), "f32", 0),
    ("stem_5x5_s2_pool3_s1", (1, 3, 24, 24), 5, 2, 2, "relu6", (3, 1, 1), "f32", 0),
    ("resnet_stem_12_tiles_3_wgs", (3, 3, 64, 64), 7, 2, 3, "relu", (3, 2, 1), "f32", 3),
    ("resnet_stem_ragged_2_wgs", (2, 3, 45, 45), 7, 2, 3, "relu", (3, 2, 1), "f32", 2),
]


@pytest.mark.parametrize("case", STEM_I8_CASES, ids=[c[0] for c in STEM_I8_CASES])
def test_int8_fused_stem_exact(case, monkeypatch):
    """The int8 stem (input codes formed in the kernel, conv, max pool) as
    one launch equals the unfused quantize / conv / max-pool launches and the
    int8 oracle bit for bit; with fewer persistent workgroups than tiles too."""
    from paper_2105_03215_amd.workloads import GraphBuilder
    name, shape, r, stride, pad, act, (ps, pst, ppad), dt, grid = case
    announce("int8 stem " + name)
    g = GraphBuilder("stem_i8_" + name, 2600 + STEM_I8_CASES.index(case))
    x = g.input("x", list(shape), "uniform", dtype=dt)
    y = g.conv(x, 64, r, stride=stride, pad=pad, act=act, name="conv")
    p = g.max_pool(y, ps, pst, ppad, name="pool")
    g.output(p)
    wl = g.finish()
    qg = oracle_calibrated_int8(wl.graph, wl.consts, [np.ascontiguousarray(a[:1]) for a in wl.inputs])
    if grid:
        monkeypatch.setenv("BYOC_STEM_GRID", str(grid))
    fused, launches = _run(qg, wl.consts, wl.inputs)
    names = [l["name"] for l in launches]
    assert names == ["stem_conv_maxpool_i8", "dequantize_out"], names
    monkeypatch.setenv("BYOC_FUSE_STEM", "0")
    plain, pl = _run(qg, wl.consts, wl.inputs)
    assert "stem_conv_maxpool_i8" not in [l["name"] for l in pl]
    assert np.array_equal(fused[0], plain[0])
    ref = OQ.run_quantized_graph(qg, wl.consts, wl.inputs)[0]
    assert np.array_equal(fused[0], ref.astype(np.float64))


HALO_I8_CASES = [
    # n, c, h, w, k, r, stride, pad, zx, act, residual: 3x3 stride 1, channels a multiple of 128
    (2, 256, 14, 14, 256, 3, 1, 1, -128, "relu", False),   # ResNet stage-3 shape, border correction
    (2, 128, 14, 13, 192, 3, 1, 1, 37, "relu", True),      # one slice, residual, ragged width
    (3, 256, 7, 7, 136, 3, 1, 1, 5, "leaky", True),        # tiny images, ragged output channels
    (1, 384, 9, 11, 64, 3, 1, 1, 0, None, False),          # three slices (two patch buffers), Z_x = 0
]


@pytest.mark.parametrize("case", HALO_I8_CASES, ids=[str(i) for i in range(len(HALO_I8_CASES))])
def test_int8_halo_conv_exact(case, monkeypatch):
    """The windowed 3x3 kernel on codes (input window staged once per
    128-channel slice) equals the int8 oracle bit for bit, at every weight
    ring depth and both tile heights, with the zero rows / columns of its
    patch corrected at the border like the implicit-GEMM kernel's."""
    n, c, h, w, k, r, stride, pad, zx, act, residual = case
    announce("int8 halo conv %s" % (case,))
    g, consts, inputs = _conv_graph(n, c, h, w, k, r, stride, pad, zx, act, residual, seed=40 + len(str(case)))
    ref = OQ.run_quantized_graph(g, consts, inputs)[0]
    for ns in (2, 3, 4, 6, 8):
        monkeypatch.setenv("BYOC_I8_TILE", "h%d" % ns)
        got, launches = _run(g, consts, inputs)
        name = [l["name"] for l in launches if l["kind"] == "conv_i8"][0]
        assert name.startswith("conv_i8_halo_128x64_s%d_" % ns), name
        assert np.array_equal(got[0], ref.astype(np.float64)), ns
    for ns in (2, 3):  # the 64-pixel tile
        monkeypatch.setenv("BYOC_I8_TILE", "h%db64" % ns)
        got, launches = _run(g, consts, inputs)
        name = [l["name"] for l in launches if l["kind"] == "conv_i8"][0]
        assert name.startswith("conv_i8_halo_64x64_s%d_" % ns), name
        assert np.array_equal(got[0], ref.astype(np.float64)), ("b64", ns)
