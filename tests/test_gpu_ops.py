"""Per-composite parity of the HIP kernels against the CPU oracle.

Each case is a one-node (or two-node) subgraph with seeded inputs, at sizes
that span several workgroup tiles and leave ragged tails in pixels, channels
and the reduction; the GPU output must be within one bf16 ulp of the oracle's
bf16io result everywhere (fp32 graphs: the 1e-4 metric against the exact
oracle), which implies the 1e-2 metric of the comparison.
"""

import numpy as np
import pytest

import oracle
from paper_2105_03215_amd import workloads
from paper_2105_03215_amd.workloads import GraphBuilder
from parity_util import (BF16_TOL, F32_TOL, announce, rel_err, term_scale_graph,
                         within_one_ulp)

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _run_gpu(wl):
    from paper_2105_03215_amd import capi, runtime
    sg = capi.Subgraph(wl.graph, wl.consts, device=0)
    try:
        return runtime.run_once(sg, wl.inputs, DEV), sg.launches()
    finally:
        sg.close()


def _check_bf16(wl, case):
    announce(case)
    gpu, launches = _run_gpu(wl)
    ref = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="bf16io")
    scales = term_scale_graph(wl.graph, wl.consts, wl.inputs)
    for g, o, sc in zip(gpu, ref, scales):
        ok = within_one_ulp(g, o, sc)
        bad = np.argwhere(~ok)
        assert ok.all(), "%s: %d elements beyond one ulp, first %s gpu %r ref %r (launches %s)" % (
            case, len(bad), bad[0], g[tuple(bad[0])], o[tuple(bad[0])], [l["name"] for l in launches])
        assert rel_err(g, o) <= BF16_TOL
    return launches


CONV_CASES = [
    # name, (n, c, h, w), k, r, stride, pad, act, residual
    ("3x3_aligned_res", (1, 64, 20, 20), 64, 3, 1, 1, "relu", True),
    ("3x3_s2_c32_k48", (2, 32, 13, 11), 48, 3, 2, 1, "relu6", False),
    ("1x1_k1000_ragged", (1, 128, 7, 7), 1000, 1, 1, 0, None, False),
    ("1x1_s2", (2, 128, 15, 15), 256, 1, 2, 0, "relu", False),
    ("stem_7x7_s2_c3", (2, 3, 37, 37), 64, 7, 2, 3, "relu", False),
    ("3x3_c24_k144", (1, 24, 28, 28), 144, 3, 1, 1, "relu6", False),
    ("3x3_s2_asym_pad", (1, 16, 9, 10), 16, 3, 2, (0, 1, 1, 0), "relu", False),
    ("3x3_splitk_c512", (1, 512, 7, 7), 512, 3, 1, 1, "relu", True),
    ("1x1_splitk_c2048", (1, 2048, 7, 7), 512, 1, 1, 0, "relu", False),
    ("1x1_c16_k8", (2, 16, 10, 10), 8, 1, 1, 0, None, True),
    ("3x3_big_m", (4, 64, 56, 56), 128, 3, 2, 1, "relu", False),
    ("1x1_gelu", (1, 64, 9, 9), 72, 1, 1, 0, "gelu", False),
    ("3x3_leaky_res", (2, 64, 14, 14), 64, 3, 1, 1, "leaky", True),
    ("3x3_s2_leaky", (2, 128, 16, 16), 256, 3, 2, 1, "leaky", False),
    ("1x1_splitk_leaky", (1, 1024, 7, 7), 512, 1, 1, 0, "leaky", False),
]


def _conv_case_graph(case, seed):
    name, shape, k, r, stride, pad, act, res = case
    g = GraphBuilder("op_" + name, seed)
    x = g.input("x", list(shape), "uniform")
    rname = None
    if res:
        n, c, h, w = shape
        pads = [pad] * 4 if isinstance(pad, int) else list(pad)
        p = (h + pads[0] + pads[2] - r) // stride + 1
        q = (w + pads[1] + pads[3] - r) // stride + 1
        rname = g.input("res", [n, k, p, q], "normal")
    y = g.conv(x, k, r, stride=stride, pad=pad, act=act, residual=rname, name="y")
    g.output(y)
    return g.finish()


@pytest.mark.parametrize("case", [c for c in CONV_CASES if "splitk" in c[0]],
                         ids=[c[0] for c in CONV_CASES if "splitk" in c[0]])
def test_conv_composite_forced_splitk(case, monkeypatch):
    """Few-tile layers are planned with four reduction groups per workgroup;
    split-K over workgroups (partials reduced by a second kernel in a fixed
    order) stays available and is held to the same bar."""
    monkeypatch.setenv("BYOC_CONV_SPLIT", "4")
    launches = _check_bf16(_conv_case_graph(case, 1000 + CONV_CASES.index(case)), "conv split-K " + case[0])
    assert any(l["kind"] == "reduce" for l in launches), [l["name"] for l in launches]


@pytest.mark.parametrize("case", CONV_CASES, ids=[c[0] for c in CONV_CASES])
def test_conv_composite(case):
    name, shape, k, r, stride, pad, act, res = case
    g = GraphBuilder("op_" + name, 1000 + CONV_CASES.index(case))
    x = g.input("x", list(shape), "uniform")
    rname = None
    if res:
        n, c, h, w = shape
        pads = [pad] * 4 if isinstance(pad, int) else list(pad)
        p = (h + pads[0] + pads[2] - r) // stride + 1
        q = (w + pads[1] + pads[3] - r) // stride + 1
        rname = g.input("res", [n, k, p, q], "normal")
    y = g.conv(x, k, r, stride=stride, pad=pad, act=act, residual=rname, name="y")
    g.output(y)
    _check_bf16(g.finish(), "conv " + name)


HALO_CASES = [
    # name, (n, c, h, w), k, act, residual, forced weight-ring depth (None:
    # the built-in ring; small outputs would otherwise go to split-K)
    ("c128_7x7_multi_image_ragged_k", (6, 128, 7, 7), 136, "relu", False, 8),
    ("c256_14x14_res", (2, 256, 14, 14), 64, "relu", True, 8),
    ("c64_30x30_one_slice", (1, 64, 30, 30), 64, None, False, 6),
    ("c192_9x5_three_slices", (3, 192, 9, 5), 72, "relu6", False, 4),
    ("c64_56x56_wide_patch", (2, 64, 56, 56), 64, "relu", False, None),
    ("c128_28x28_ring2", (2, 128, 28, 28), 128, "relu", True, 2),
    ("c128_28x28_ring4", (2, 128, 28, 28), 128, "relu", True, 4),
    ("c128_28x28_ring6", (2, 128, 28, 28), 128, "relu", True, 6),
    ("c128_28x28_builtin", (4, 128, 28, 28), 128, "relu", True, None),
    ("c512_7x7_gelu", (3, 512, 7, 7), 128, "gelu", False, 8),
    ("c256_14x14_leaky_ring3", (2, 256, 14, 14), 128, "leaky", False, 3),
]


@pytest.mark.parametrize("case", HALO_CASES, ids=[c[0] for c in HALO_CASES])
def test_conv_halo_composite(case, monkeypatch):
    """3x3 stride-1 convs on the kernel that stages the input window in LDS:
    tiles spanning several images, ragged pixel and channel tails, one to
    eight 64-channel slices, non-square images, every weight-ring depth."""
    name, shape, k, act, res, ring = case
    if ring is not None:
        monkeypatch.setenv("BYOC_CONV_TILE", "h128x64s%d" % ring)
    else:  # the halo kernel wherever the shape allows, built-in ring
        monkeypatch.setenv("BYOC_CONV_HALO", "1")
    g = GraphBuilder("op_halo_" + name, 1300 + HALO_CASES.index(case))
    x = g.input("x", list(shape), "uniform")
    n, c, h, w = shape
    rname = g.input("res", [n, k, h, w], "normal") if res else None
    y = g.conv(x, k, 3, stride=1, pad=1, act=act, residual=rname, name="y")
    g.output(y)
    launches = _check_bf16(g.finish(), "conv halo " + name)
    names = [l["name"] for l in launches]
    assert any(nm.startswith("conv_halo_128x64") for nm in names), names
    if ring is not None:
        assert any(nm.startswith("conv_halo_128x64_s%d_" % ring) for nm in names), names


HALO64_CASES = [
    # name, (n, c, h, w), k, act, residual, weight-ring depth of the 64-pixel tile
    ("c512_7x7_multi_image_res", (3, 512, 7, 7), 128, "relu", True, 3),
    ("c128_7x7_ragged_k", (5, 128, 7, 7), 136, "relu", False, 2),
    ("c192_9x5_three_slices", (3, 192, 9, 5), 72, "relu6", False, 3),
    ("c64_30x30_one_slice", (1, 64, 30, 30), 64, None, False, 2),
    ("c384_8x8_gelu", (2, 384, 8, 8), 64, "gelu", False, 3),
]


@pytest.mark.parametrize("case", HALO64_CASES, ids=[c[0] for c in HALO64_CASES])
def test_conv_halo_64_composite(case, monkeypatch):
    """The windowed kernel's 64-pixel tile: within one ulp of the oracle and
    bit for bit the 128-pixel tile (the same summation order)."""
    name, shape, k, act, res, ring = case
    monkeypatch.setenv("BYOC_CONV_TILE", "h64x64s%d" % ring)
    g = GraphBuilder("op_halo64_" + name, 1350 + HALO64_CASES.index(case))
    x = g.input("x", list(shape), "uniform")
    n, c, h, w = shape
    rname = g.input("res", [n, k, h, w], "normal") if res else None
    y = g.conv(x, k, 3, stride=1, pad=1, act=act, residual=rname, name="y")
    g.output(y)
    wl = g.finish()
    launches = _check_bf16(wl, "conv halo 64 " + name)
    assert any(l["name"].startswith("conv_halo_64x64_s%d_" % ring) for l in launches), launches
    got, _ = _run_gpu(wl)
    monkeypatch.setenv("BYOC_CONV_TILE", "h128x64s%d" % ring)
    ref, launches = _run_gpu(wl)
    assert any(l["name"].startswith("conv_halo_128x64") for l in launches), launches
    for a, b in zip(got, ref):
        assert np.array_equal(a, b)


DW_CASES = [
    # name, (n, c, h, w), kernel, stride, pad, act, residual
    ("dw_s1_c96", (2, 96, 14, 14), 3, 1, 1, "relu6", False),
    ("dw_s2_c144", (1, 144, 28, 28), 3, 2, 1, "relu6", False),
    ("dw_s1_c40_res", (1, 40, 9, 7), 3, 1, 1, "relu6", True),
    # strips of 4 (stride 1) or 2 (stride 2) rows with ragged last strips,
    # several blocks along (column, channel group), odd sizes
    ("dw_s1_c32_ragged_rows", (3, 32, 113, 57), 3, 1, 1, "relu6", False),
    ("dw_s2_c96_odd", (2, 96, 113, 111), 3, 2, 1, "relu6", False),
    ("dw_s1_c960_7x7", (2, 960, 7, 7), 3, 1, 1, "relu6", True),
    ("dw_s2_asym_pad", (1, 24, 10, 9), 3, 2, (0, 0, 1, 1), None, False),
    ("dw_s1_leaky_no_pad", (2, 16, 6, 11), 3, 1, 0, "leaky", False),
    ("dw_s1_gelu", (1, 64, 5, 5), 3, 1, 1, "gelu", True),
    # not 3x3: the generic kernel
    ("dw_5x5_generic", (1, 48, 12, 12), 5, 1, 2, "relu", False),
    ("dw_3x3_s3_generic", (1, 8, 13, 13), 3, 3, 1, "relu", False),
]


@pytest.mark.parametrize("case", DW_CASES, ids=[c[0] for c in DW_CASES])
def test_depthwise_composite(case):
    name, shape, r, stride, pad, act, res = case
    g = GraphBuilder("op_" + name, 1100 + DW_CASES.index(case))
    x = g.input("x", list(shape), "uniform")
    n, c, h, w = shape
    pads = [pad] * 4 if isinstance(pad, int) else list(pad)
    p = (h + pads[0] + pads[2] - r) // stride + 1
    q = (w + pads[1] + pads[3] - r) // stride + 1
    rname = g.input("res", [n, c, p, q], "normal") if res else None
    y = g.conv(x, c, r, stride=stride, pad=pad, groups=c, act=act, residual=rname, name="y")
    g.output(y)
    launches = _check_bf16(g.finish(), "depthwise " + name)
    assert any(l["kind"] == "depthwise" for l in launches)


def _dw_graph(case, seed):
    name, shape, r, stride, pad, act, res = case
    g = GraphBuilder("op_" + name, seed)
    x = g.input("x", list(shape), "uniform")
    n, c, h, w = shape
    p = (h + 2 * pad - r) // stride + 1
    q = (w + 2 * pad - r) // stride + 1
    rname = g.input("res", [n, c, p, q], "normal") if res else None
    g.output(g.conv(x, c, r, stride=stride, pad=pad, groups=c, act=act, residual=rname, name="y"))
    return g.finish()


# every 3x3 case with symmetric padding, and MobileNetV2's unfused depthwise
# layers at batch 16 (many workgroups per XCD)
DW_STRIP_CASES = [c for c in DW_CASES if c[2] == 3 and c[3] in (1, 2) and isinstance(c[4], int)] + [
    ("dw_s1_c576_14x14_bs16", (16, 576, 14, 14), 3, 1, 1, "relu6", False),
    ("dw_s2_c576_14x14_bs16", (16, 576, 14, 14), 3, 2, 1, "relu6", False),
    ("dw_s1_c960_7x7_bs16", (16, 960, 7, 7), 3, 1, 1, "relu6", False),
]


@pytest.mark.parametrize("case", DW_STRIP_CASES, ids=[c[0] for c in DW_STRIP_CASES])
def test_depthwise_strip_heights_bitwise(case, monkeypatch):
    """Every strip height of the 3x3 strip kernel (2, 4, 8 output rows per
    thread at stride 1; 1, 2, 4 at stride 2) gives the same bits, and the
    default one is within one ulp of the oracle."""
    wl = _dw_graph(case, 1150 + DW_STRIP_CASES.index(case))
    monkeypatch.delenv("BYOC_DW_STRIP", raising=False)
    _check_bf16(wl, "depthwise strips " + case[0])
    ref, _ = _run_gpu(wl)
    for strip in ("2,1", "8,4"):
        monkeypatch.setenv("BYOC_DW_STRIP", strip)
        got, launches = _run_gpu(wl)
        assert any(l["kind"] == "depthwise" for l in launches)
        for a, b in zip(got, ref):
            assert np.array_equal(a, b), (case[0], strip)


DENSE_CASES = [
    ("fc_m1_k2048_n1000", 1, 2048, 1000, None, False),
    ("ffn1_m33_gelu", 33, 768, 3072, "gelu", False),
    ("ffn2_m64_res", 64, 3072, 768, None, True),
    ("m130_k100_n24_relu", 130, 104, 24, "relu", False),
]


@pytest.mark.parametrize("case", DENSE_CASES, ids=[c[0] for c in DENSE_CASES])
def test_dense_composite(case):
    name, m, kin, nout, act, res = case
    g = GraphBuilder("op_" + name, 1200 + DENSE_CASES.index(case))
    x = g.input("x", [m, kin], "normal")
    rname = g.input("res", [m, nout], "normal") if res else None
    y = g.dense(x, nout, act=act, residual=rname, w_std=0.05, b_std=0.05, name="y")
    g.output(y)
    _check_bf16(g.finish(), "dense " + name)


def _bf16_grid(lo_exp, hi_exp):
    """Every bfloat16 value v with 2^lo_exp <= |v| < 2^hi_exp, both signs, and 0."""
    mags = [(1.0 + m / 128.0) * 2.0 ** e for e in range(lo_exp, hi_exp) for m in range(128)]
    return np.array([0.0] + mags + [-v for v in mags], dtype=np.float32)


@pytest.mark.parametrize("rows", [32, 256], ids=["dense_rows", "implicit_gemm"])
def test_gelu_every_bf16_value(rows):
    """GELU of every bf16 value in +-[2^-12, 16) through a dense composite
    with identity weights (x . I = x exactly in fp32), so the output is the
    kernel's GELU of x rounded to bf16: within one bf16 ulp of the oracle's
    exact-erf GELU everywhere and equal to it almost everywhere (the float32
    evaluation may fall on the other side of a rounding boundary only where
    the exact value lies within its error of one).  32 rows take the few-row
    dense kernel, 256 the implicit-GEMM kernel's epilogue."""
    announce("gelu over every bf16 value, %d rows" % rows)
    vals = _bf16_grid(-12, 4)
    c = 64
    x = np.resize(vals, rows * c).reshape(rows, c).astype(np.float32)
    graph = {"format": "byoc-subgraph", "version": 1,
             "inputs": [{"name": "x", "shape": [rows, c], "dtype": "bf16", "layout": "ROWMAJOR"}],
             "constants": [{"name": "w", "index": 0, "shape": [c, c], "dtype": "f32"}],
             "nodes": [{"name": "y", "composite": "dense_gelu", "inputs": ["x", "w"], "out_dtype": "bf16"}],
             "outputs": [{"name": "y", "dtype": "bf16", "layout": "ROWMAJOR"}]}
    wl = workloads.Workload(graph, [np.eye(c, dtype=np.float32)], [x], rows * c * c, rows * c * c)
    gpu, launches = _run_gpu(wl)
    ref = oracle.run_graph(graph, wl.consts, wl.inputs, mode="bf16io")[0]
    ok = within_one_ulp(gpu[0], ref)
    assert ok.all(), (x[~ok][:5], gpu[0][~ok][:5], ref[~ok][:5])
    same = np.mean(gpu[0] == ref)
    print("gelu: %.5f of the bf16 outputs equal the oracle's (launches %s)" % (same, [l["name"] for l in launches]))
    assert same >= 0.999


def test_pools_and_add():
    g = GraphBuilder("op_pools", 1300)
    x = g.input("x", [2, 64, 29, 29], "normal")
    z = g.input("z", [2, 64, 15, 15], "normal")
    p = g.max_pool(x, 3, 2, 1, name="mp")
    a = g.add(p, z, act="relu", name="add")
    gp = g.global_avg_pool(a, name="gap")
    g.output(p)
    g.output(a)
    g.output(gp)
    _check_bf16(g.finish(), "maxpool+add_relu+gap")


def test_odd_channel_pool_and_gap():
    g = GraphBuilder("op_pools_odd", 1301)
    x = g.input("x", [3, 12, 7, 9], "normal")
    p = g.max_pool(x, 3, 1, 1, name="mp")
    gp = g.global_avg_pool(x, name="gap")
    g.output(p)
    g.output(gp)
    _check_bf16(g.finish(), "maxpool s1 + gap, C=12")


def test_f32_input_cast_and_f32_output():
    g = GraphBuilder("op_cast", 1400)
    x = g.input("x", [1, 3, 17, 17], "uniform", dtype="f32")
    y = g.conv(x, 16, 3, stride=1, pad=1, act="relu", name="y")
    g.output(y, dtype="f32")
    _check_bf16(g.finish(), "f32 input -> bf16 conv -> f32 output")


def test_rowmajor_cast_paths():
    # K not a multiple of 8: boundary pads the rows; f32 output is cast back
    g = GraphBuilder("op_rows", 1401)
    x = g.input("x", [5, 30], "normal", dtype="f32")
    y = g.dense(x, 20, act="relu", w_std=0.1, name="y")
    g.output(y, dtype="f32")
    g.output(x, dtype="bf16")
    _check_bf16(g.finish(), "rows f32 [5,30] -> dense 20")


# ---------------------------------------------------------------------------
# fp32 graphs


def _check_f32(wl, case):
    announce(case)
    gpu, _ = _run_gpu(wl)
    ref = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="exact")
    for g, o in zip(gpu, ref):
        assert rel_err(g, o) <= F32_TOL, (case, rel_err(g, o))


def test_f32_single_composite_config():
    _check_f32(workloads.conv_f32(), "conv_f32 1x16x32x32 -> 32")


F32_CONV_CASES = [
    # name, (n, c, h, w), k, r, stride, pad, act, residual: the
    # register-blocked kernel (3x3 and 1x1: odd channel counts, output
    # channels not a multiple of its 4-channel block, strides, residual) and
    # the direct kernel (other kernel sizes)
    ("s2_res_leaky_k13", (2, 64, 41, 40), 13, 3, 2, 1, "leaky", True),
    ("k5_asym_pad_direct", (1, 6, 23, 19), 20, 5, 1, (2, 0, 1, 3), "relu6", False),
    ("1x1_odd_channels", (1, 301, 9, 30), 16, 1, 1, 0, None, True),
    ("wide_rows", (1, 4, 5, 300), 8, 3, 1, 1, "relu", False),
    ("tiny_odd", (3, 5, 4, 4), 7, 3, 1, 1, "relu", False),
]


@pytest.mark.parametrize("case", F32_CONV_CASES, ids=[c[0] for c in F32_CONV_CASES])
def test_f32_conv_cases(case):
    name, shape, k, r, stride, pad, act, res = case
    g = GraphBuilder("op_f32_" + name, 1550 + F32_CONV_CASES.index(case), dtype="f32")
    x = g.input("x", list(shape), "uniform")
    rname = None
    if res:
        n, c, h, w = shape
        pads = [pad] * 4 if isinstance(pad, int) else list(pad)
        p = (h + pads[0] + pads[2] - r) // stride + 1
        q = (w + pads[1] + pads[3] - r) // stride + 1
        rname = g.input("res", [n, k, p, q], "normal")
    y = g.conv(x, k, r, stride=stride, pad=pad, act=act, residual=rname, bn=False, w_std=0.2, name="y")
    g.output(y)
    _check_f32(g.finish(), "f32 conv " + name)


def test_f32_other_ops():
    g = GraphBuilder("op_f32", 1500, dtype="f32")
    x = g.input("x", [2, 8, 11, 11], "uniform")
    a = g.conv(x, 8, 3, stride=2, pad=1, groups=8, act="relu6", bn=False, w_std=0.3, name="dw")
    p = g.max_pool(x, 3, 2, 1, name="mp")
    s = g.add(a, p, act="relu", name="s")
    gp = g.global_avg_pool(s, name="gap")
    d = g.dense(gp, 10, act="gelu", w_std=0.3, name="fc")
    g.output(d)
    g.output(s)
    _check_f32(g.finish(), "fp32 dw/maxpool/add/gap/dense")


STEM_CASES = [
    # name, (n, c, h, w), r, stride, pad, act, (pool size, stride, pad), input dtype
    ("resnet_stem_ragged", (2, 3, 45, 45), 7, 2, 3, "relu", (3, 2, 1), "bf16"),
    ("stem_f32_c1", (1, 1, 32, 30), 7, 2, 3, "relu", (3, 2, 1), "f32"),
    ("stem_3x3_s1_pool2", (2, 4, 20, 21), 3, 1, 1, None, (2, 2, 0), "bf16"),
    ("stem_5x5_s2_pool3_s1", (1, 3, 24, 24), 5, 2, 2, "relu6", (3, 1, 1), "bf16"),
    ("resnet_stem_f32_aligned", (2, 3, 48, 48), 7, 2, 3, "relu", (3, 2, 1), "f32"),
    ("stem_leaky", (2, 3, 40, 40), 7, 2, 3, "leaky", (3, 2, 1), "bf16"),
]


@pytest.mark.parametrize("case", STEM_CASES, ids=[c[0] for c in STEM_CASES])
def test_fused_stem_conv_maxpool(case):
    """A few-channel NCHW input feeding conv -> max pool runs as one fused
    kernel (no layout transform, no full-resolution conv output) and matches
    the unfused oracle chain."""
    name, shape, r, stride, pad, act, (ps, pst, ppad), dt = case
    g = GraphBuilder("stem_" + name, 1600 + STEM_CASES.index(case))
    x = g.input("x", list(shape), "uniform", dtype=dt)
    y = g.conv(x, 64, r, stride=stride, pad=pad, act=act, name="conv")
    p = g.max_pool(y, ps, pst, ppad, name="pool")
    g.output(p)
    launches = _check_bf16(g.finish(), "stem " + name)
    names = [l["name"] for l in launches]
    assert names[0] == "stem_conv_maxpool" and "nchw_to_nhwc" not in names, names


DENSE_ROWS_CASES = [
    # name, rows, k, n, act, residual
    ("m1_k2048_n1000", 1, 2048, 1000, None, False),
    ("m32_k2048_n1000_relu", 32, 2048, 1000, "relu", False),
    ("m33_k1000_n24_gelu_res", 33, 1000, 24, "gelu", True),
    ("m64_k64_n40_relu6", 64, 64, 40, "relu6", False),
    ("m16_k4200_n16_res", 16, 4200, 16, None, True),  # more k-steps than one pass of the waves
    ("m32_k1024_n1000_leaky", 32, 1024, 1000, "leaky", False),
]


@pytest.mark.parametrize("case", DENSE_ROWS_CASES, ids=[c[0] for c in DENSE_ROWS_CASES])
def test_dense_rows(case):
    """Few-row dense composites run on the dense-rows kernel (reduction split
    over the waves of a workgroup) and match the oracle."""
    name, rows, k, n, act, res = case
    g = GraphBuilder("dense_rows_" + name, 1800 + DENSE_ROWS_CASES.index(case))
    x = g.input("x", [rows, k], "normal", dtype="bf16")
    r = g.input("r", [rows, n], "normal", dtype="bf16") if res else None
    y = g.dense(x, n, act=act, residual=r, name="fc")
    g.output(y)
    launches = _check_bf16(g.finish(), "dense rows " + name)
    assert any(l["name"].startswith("dense_rows") for l in launches), [l["name"] for l in launches]


# (case, workgroups): each workgroup walks several tiles, so the patch
# prefetch of the next tile and the tile loop's LDS reuse are exercised
STEM_LOOP_CASES = [
    (("resnet_stem_12_tiles", (3, 3, 64, 64), 7, 2, 3, "relu", (3, 2, 1), "bf16"), 3),
    (("resnet_stem_ragged_8_tiles", (2, 3, 45, 45), 7, 2, 3, "relu", (3, 2, 1), "bf16"), 3),
    (("stem_f32_8_tiles", (2, 3, 48, 48), 7, 2, 3, "gelu", (3, 2, 1), "f32"), 2),
]


@pytest.mark.parametrize("case,grid", STEM_LOOP_CASES, ids=[c[0][0] for c in STEM_LOOP_CASES])
def test_fused_stem_tile_loop(case, grid, monkeypatch):
    """Fewer persistent workgroups than tiles: results match the oracle
    for every tile a workgroup computes after its first."""
    monkeypatch.setenv("BYOC_STEM_GRID", str(grid))
    name, shape, r, stride, pad, act, (ps, pst, ppad), dt = case
    g = GraphBuilder("stem_loop_" + name, 1700 + [c[0] for c in STEM_LOOP_CASES].index(case))
    x = g.input("x", list(shape), "uniform", dtype=dt)
    y = g.conv(x, 64, r, stride=stride, pad=pad, act=act, name="conv")
    p = g.max_pool(y, ps, pst, ppad, name="pool")
    g.output(p)
    launches = _check_bf16(g.finish(), "stem loop %s grid %d" % (name, grid))
    assert launches[0]["name"] == "stem_conv_maxpool", launches[0]


def test_leaky_slopes_depthwise_add_and_f32():
    """The leaky ReLU's slope reaches every other kernel: a non-default slope
    on the implicit GEMM, the depthwise conv, the standalone add, and the
    fp32 graph's direct conv and add."""
    g = GraphBuilder("op_leaky", 1900)
    x = g.input("x", [2, 48, 12, 12], "normal")
    a = g.conv(x, 48, 3, act="leaky", alpha=0.25, name="a")
    d = g.conv(a, 48, 3, groups=48, act="leaky", alpha=0.05, name="dw")
    s = g.add(a, d, act="leaky", name="s")
    g.output(s)
    g.output(a)
    wl = g.finish()
    for n in wl.graph["nodes"]:
        if n["name"] == "s":
            n["attrs"]["alpha"] = 0.3
    _check_bf16(wl, "leaky slopes: conv, depthwise, add")
    g = GraphBuilder("op_leaky_f32", 1901, dtype="f32")
    x = g.input("x", [2, 8, 11, 11], "normal")
    a = g.conv(x, 8, 3, act="leaky", alpha=0.2, bn=False, w_std=0.3, name="a")
    s = g.add(a, x, act="leaky", name="s")
    g.output(s)
    _check_f32(g.finish(), "fp32 leaky conv and add")


AVGPOOL_CASES = [
    # name, (n, c, h, w), size, stride, pad, count_include_pad
    ("3x3_s1_p1", (2, 64, 17, 17), 3, 1, 1, False),
    ("3x3_s1_p1_incl", (1, 40, 9, 7), 3, 1, 1, True),
    ("3x3_s2_p0", (2, 24, 15, 16), 3, 2, 0, False),
]


@pytest.mark.parametrize("case", AVGPOOL_CASES, ids=[c[0] for c in AVGPOOL_CASES])
def test_avg_pool_window(case):
    name, shape, size, stride, pad, incl = case
    g = GraphBuilder("op_avgpool_" + name, 2000 + AVGPOOL_CASES.index(case))
    x = g.input("x", list(shape), "normal")
    y = g.avg_pool(x, size, stride, pad, name="y")
    g.nodes[-1]["attrs"]["count_include_pad"] = incl
    g.output(y)
    _check_bf16(g.finish(), "avg pool " + name)


def test_concat_in_place_and_copied():
    """A concatenation of conv, max-pool and avg-pool outputs (written in
    place into their channel slices), a value also read elsewhere and a
    graph input (copied in), with rectangular 1x7 / 7x1 / 1x3 kernels; the
    concatenation feeds a conv and is a graph output."""
    g = GraphBuilder("op_concat", 2100)
    x = g.input("x", [2, 32, 13, 11], "uniform")
    z = g.input("z", [2, 16, 13, 11], "normal")
    a = g.conv(x, 24, (1, 7), name="a")
    b = g.conv(g.conv(x, 16, (7, 1), name="b0"), 40, (1, 3), name="b")
    m = g.max_pool(x, 3, 1, 1, name="m")
    p = g.avg_pool(x, 3, 1, 1, name="p")
    shared = g.conv(x, 8, 1, name="shared")
    c = g.concat([a, b, m, z, shared, p], name="cat")
    y = g.conv(c, 48, 3, name="y")
    u = g.conv(shared, 8, 1, name="u")
    g.output(y)
    g.output(c)
    g.output(u)
    launches = _check_bf16(g.finish(), "concat in place and copied")
    names = [l["name"] for l in launches]
    # z (a graph input) and shared (read twice) are copied; the rest in place
    assert names.count("concat_copy") == 2, names


def test_concat_all_in_place():
    g = GraphBuilder("op_concat_inplace", 2101)
    x = g.input("x", [1, 64, 8, 8], "uniform")
    c = g.concat([g.conv(x, 64, 1, name="a"), g.conv(x, 96, 3, name="b"), g.conv(x, 32, (3, 1), name="c")],
                 name="cat")
    g.output(g.conv(c, 16, 1, name="y"))
    launches = _check_bf16(g.finish(), "concat all in place")
    assert "concat_copy" not in [l["name"] for l in launches]


POST_ADD_PATHS = [
    ("default", {}),
    ("halo", {"BYOC_CONV_TILE": "h128x64s3"}),
    ("register_staged", {"BYOC_CONV_TILE": "64x64"}),
    ("split_k", {"BYOC_CONV_TILE": "64x64", "BYOC_CONV_SPLIT": "2"}),
]


@pytest.mark.parametrize("path", POST_ADD_PATHS, ids=[p[0] for p in POST_ADD_PATHS])
def test_post_activation_add_folds_into_conv(path, monkeypatch):
    """An add after a conv's activation (DarkNet's residual) runs inside the
    conv's epilogue on every conv kernel, bit-identical to the two launches."""
    name, env = path
    g = GraphBuilder("op_post_add", 1950)
    x = g.input("x", [2, 64, 14, 13], "normal")
    a = g.conv(x, 32, 1, act="leaky", name="a")
    b = g.conv(a, 64, 3, act="leaky", name="b")
    s = g.add(x, b, name="s")          # the conv is the second operand
    c = g.conv(s, 32, 1, act="relu", name="c")
    d = g.conv(c, 64, 3, act="leaky", name="d")
    t = g.add(d, s, name="t")          # the conv is the first operand
    g.output(t)
    wl = g.finish()
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    launches = _check_bf16(wl, "post-activation add, %s path" % name)
    names = [l["name"] for l in launches]
    assert not any(n.startswith("add_") for n in names), names
    fused, _ = _run_gpu(wl)
    monkeypatch.setenv("BYOC_FUSE_POST_ADD", "0")
    plain, plain_launches = _run_gpu(wl)
    assert sum(1 for l in plain_launches if l["name"].startswith("add_")) == 2
    assert np.array_equal(fused[0], plain[0])


def test_post_activation_add_not_folded():
    """The fold needs the conv's output to be read by the add alone, and the
    add to carry no activation of its own; otherwise both launches stay."""
    g = GraphBuilder("op_post_add_kept", 1960)
    x = g.input("x", [1, 32, 9, 11], "normal")
    b = g.conv(x, 32, 3, act="leaky", name="b")
    s = g.add(x, b, name="s")            # b is also a graph output
    c = g.conv(s, 32, 3, act="relu", name="c")
    t = g.add(c, s, act="relu", name="t")  # the add has an activation
    g.output(t)
    g.output(b)
    launches = _check_bf16(g.finish(), "post-activation adds that stay separate")
    assert sum(1 for l in launches if l["name"].startswith("add_")) == 2
