"""The partial-quantization pass (Sec. 3.2, Fig. 4a) and the int8 schema
checks of the C library, on the CPU."""

import copy

import numpy as np
import pytest

from oracle import quant as OQ
from paper_2105_03215_amd import capi, quantize, workloads
from test_oracle_quant import _tiny_int8_graph


@pytest.mark.parametrize("lo,hi", [(-1.3, 2.7), (0.0, 6.0), (-4.0, -1.0), (0.5, 3.0), (-0.001, 0.0)])
def test_affine_params_cover_the_range_and_zero(lo, hi):
    s, z = quantize.affine_params(lo, hi)
    assert s > 0 and -128 <= z <= 127
    assert OQ.dequantize(z, s, z) == 0.0  # zero (the padding value) is a code
    lo2, hi2 = min(lo, 0.0), max(hi, 0.0)
    for v in (lo2, hi2):
        back = OQ.dequantize(OQ.quantize(np.float32(v), s, z), s, z)
        assert abs(float(back) - v) <= s * 0.5 + 1e-6 * max(1.0, abs(v))
    assert quantize.affine_params(0.0, 0.0) == (1.0, 0)


def test_quantize_graph_rewrites_and_validates():
    wl = workloads.build("resnet50_v1", n=1, hw=64)
    rng = np.random.default_rng(0)
    ranges = {d["name"]: (0.0, 1.0) for d in wl.graph["inputs"]}
    for n in wl.graph["nodes"]:
        ranges[n["name"]] = (-float(rng.uniform(0, 3)), float(rng.uniform(1, 9)))
    qg = quantize.quantize_graph(wl.graph, ranges)
    assert all(n["out_dtype"] == "int8" for n in qg["nodes"])
    assert all("quant" in n for n in qg["nodes"])
    pools = [n for n in qg["nodes"] if n["composite"] == "max_pool2d"]
    by_name = {n["name"]: n for n in qg["nodes"]}
    for p in pools:
        assert p["quant"] == by_name[p["inputs"][0]]["quant"]
    assert wl.graph["nodes"][0]["out_dtype"] != "int8"  # the float function is left alone
    capi.validate(qg, wl.consts)
    cal = quantize.calibration_graph(wl.graph)
    assert [o["name"] for o in cal["outputs"]] == [n["name"] for n in wl.graph["nodes"]]
    capi.validate(cal, wl.consts)


def _mut(fn):
    g, consts = _tiny_int8_graph()
    g = copy.deepcopy(g)
    fn(g)
    return g, consts


@pytest.mark.parametrize("mutate,status,needle", [
    (lambda g: g["nodes"][0].pop("quant"), "PARSE", "needs quant"),
    (lambda g: g["inputs"][0].pop("quant"), "SHAPE", "no quant parameters"),
    (lambda g: g["nodes"][2].__setitem__("quant", {"scale": 0.05, "zero_point": -128}), "SHAPE", "keeps its input"),
    (lambda g: g["nodes"][0]["quant"].__setitem__("zero_point", 200), "PARSE", "zero_point"),
    (lambda g: g["nodes"][0]["quant"].__setitem__("scale", -1.0), "PARSE", "scale"),
    (lambda g: g["nodes"][0].__setitem__("composite", "conv2d_bias_gelu"), "UNSUPPORTED", "gelu"),
    (lambda g: g["nodes"][1].__setitem__("out_dtype", "bf16"), "UNSUPPORTED", "mixed out_dtype"),
])
def test_int8_schema_errors(mutate, status, needle):
    g, consts = _mut(mutate)
    with pytest.raises(capi.ByocError) as ei:
        capi.validate(g, consts)
    assert status in str(ei.value) and needle in str(ei.value)


def test_int8_schema_accepts_inherited_pool_quant():
    g, consts = _mut(lambda g: g["nodes"][2].pop("quant"))
    capi.validate(g, consts)


def test_int8_schema_accepts_leaky():
    """Leaky ReLU has an int8 form (on the offset from the zero point)."""
    g, consts = _mut(lambda g: g["nodes"][0].__setitem__("composite", g["nodes"][0]["composite"] + "_leaky")
                     if not g["nodes"][0]["composite"].endswith(("relu", "relu6")) else
                     g["nodes"][0].__setitem__("composite", g["nodes"][0]["composite"].rsplit("_", 1)[0] + "_leaky"))
    assert g["nodes"][0]["composite"].endswith("_leaky")
    capi.validate(g, consts)


def test_quant_only_in_int8_graphs():
    g, consts = _tiny_int8_graph()
    gf = copy.deepcopy(g)
    for n in gf["nodes"]:
        n["out_dtype"] = "bf16"
    with pytest.raises(capi.ByocError) as ei:
        capi.validate(gf, consts)
    assert "only in int8 graphs" in str(ei.value)
