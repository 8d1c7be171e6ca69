"""Contract tests of the C ABI that need no GPU: the library loads, exports
every entry point the header declares, and rejects malformed or inconsistent
subgraphs on the host (validation precedes any device call)."""

import copy
import json
import os
import re

import numpy as np
import pytest

from paper_2105_03215_amd import capi, workloads
from paper_2105_03215_amd.capi import ByocError, validate

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "byoc.h")


@pytest.fixture(scope="module")
def lib():
    return capi.load_library()


def test_exports_every_declared_symbol(lib):
    with open(HEADER) as f:
        text = f.read()
    declared = set(re.findall(r"^\s*(?:byoc_status|const char\*)\s+(byoc_\w+)\s*\(", text, re.M))
    assert declared == set(capi.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


def test_workloads_validate():
    for name in ["conv_f32", "resnet18_block", "mobilenet_v2"]:
        wl = workloads.build(name)
        validate(wl.graph, wl.consts)
    wl = workloads.build("resnet50_v1", n=2)
    validate(wl.json, wl.consts)
    wl = workloads.build("bert_ffn", batch=1, seq=8, layers=2)
    validate(wl.graph, wl.consts)


def _small():
    wl = workloads.resnet18_block(n=1, c=8, hw=6)
    return copy.deepcopy(wl.graph), wl.consts


def _expect(graph, consts, status, fragment):
    with pytest.raises(ByocError) as ei:
        validate(graph, consts)
    assert ei.value.status_name == status, str(ei.value)
    assert fragment in str(ei.value), str(ei.value)


def test_malformed_json():
    g, c = _small()
    _expect(json.dumps(g)[:-3], c, "PARSE", "JSON")
    _expect("[1, 2]", c, "PARSE", "top level")
    _expect('{"format": "x", "version": 1}', c, "PARSE", "format")


def test_schema_errors():
    g, c = _small()
    g2 = copy.deepcopy(g)
    g2["version"] = 2
    _expect(g2, c, "UNSUPPORTED", "version")
    g2 = copy.deepcopy(g)
    g2["nodes"][0]["composite"] = "conv3d_bias_relu"
    _expect(g2, c, "UNSUPPORTED", "node 0")
    g2 = copy.deepcopy(g)
    g2["nodes"][1]["inputs"][0] = "nope"
    _expect(g2, c, "PARSE", "unknown or later value 'nope'")
    g2 = copy.deepcopy(g)
    g2["nodes"][0]["inputs"] = g2["nodes"][0]["inputs"][:2]
    _expect(g2, c, "PARSE", "expects 3 inputs")
    g2 = copy.deepcopy(g)
    g2["nodes"][0]["attrs"]["dilation"] = [2, 2]
    _expect(g2, c, "UNSUPPORTED", "dilation")
    g2 = copy.deepcopy(g)
    g2["nodes"][1]["out_dtype"] = "f32"
    _expect(g2, c, "UNSUPPORTED", "mixed out_dtype")
    g2 = copy.deepcopy(g)
    g2["nodes"][1]["name"] = g2["nodes"][0]["name"]
    _expect(g2, c, "PARSE", "duplicate name")
    g2 = copy.deepcopy(g)
    g2["outputs"][0]["name"] = "conv1.w"
    _expect(g2, c, "UNSUPPORTED", "constant cannot be a subgraph output")


def test_constant_mismatches():
    g, c = _small()
    bad = list(c)
    bad[0] = np.zeros((8, 8, 3, 1), np.float32)
    _expect(g, bad, "SHAPE", "passed shape [8,8,3,1] != declared [8,8,3,3]")
    _expect(g, c[:2], "INVALID_ARG", "outside the 2 constants passed")
    g2 = copy.deepcopy(g)
    g2["constants"][1]["shape"] = [9]
    bad = list(c)
    bad[1] = np.zeros(9, np.float32)
    _expect(g2, bad, "SHAPE", "bias shape [9] != [8]")
    g2 = copy.deepcopy(g)
    g2["nodes"][0]["inputs"][1] = "x"
    _expect(g2, c, "UNSUPPORTED", "must be a constant")


def test_shape_errors():
    g, c = _small()
    g2 = copy.deepcopy(g)
    g2["nodes"][1]["inputs"][3] = "x"
    g2["nodes"][1]["attrs"]["strides"] = [2, 2]
    _expect(g2, c, "SHAPE", "residual shape")
    g2 = copy.deepcopy(g)
    g2["nodes"][0]["attrs"]["groups"] = 2
    _expect(g2, c, "SHAPE", "groups 2")
    g2 = copy.deepcopy(g)
    g2["inputs"][0]["shape"] = [1, 8, 6]
    _expect(g2, c, "UNSUPPORTED", "rank must be 2 or 4")


def test_pool_and_add_rules():
    g = {"format": "byoc-subgraph", "version": 1,
         "inputs": [{"name": "x", "shape": [1, 8, 5, 5], "dtype": "bf16"}],
         "nodes": [{"name": "p", "composite": "max_pool2d", "inputs": ["x"],
                    "attrs": {"pool_size": [3, 3], "strides": [2, 2], "padding": [3, 3, 3, 3]},
                    "out_dtype": "bf16"}],
         "outputs": [{"name": "p"}]}
    _expect(g, [], "UNSUPPORTED", "padding must be smaller")
    g["nodes"][0]["attrs"]["padding"] = [1, 1, 1, 1]
    validate(g, [])
    g["nodes"].append({"name": "a", "composite": "add_relu", "inputs": ["p", "x"], "out_dtype": "bf16"})
    _expect(g, [], "SHAPE", "operand shapes")


def test_create_without_device_reports_device_error():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    wl = workloads.conv_f32(n=1, c=4, hw=6, k=3)
    with pytest.raises(ByocError) as ei:
        capi.Subgraph(wl.graph, wl.consts)
    assert ei.value.status_name in ("DEVICE", "INVALID_ARG")
