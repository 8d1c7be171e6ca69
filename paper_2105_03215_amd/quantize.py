"""Partial quantization of an offloaded function (Sec. 3.2, Fig. 4a).

The accelerator backend inserts quantize / dequantize nodes into a
partitioned function so that the accelerator computes on fixed-point codes
while the rest of the model keeps floating tensors.  The scale S and zero
point Z of every tensor come either from calibration data at compile time or
from the real data at run time.  This module is the compile-time form:

* ``calibrate`` runs the float function on calibration inputs through the
  executor itself (a copy of the function whose outputs are every node) and
  records each tensor's range;
* ``affine_params`` turns a range into int8 (S, Z): the range is widened to
  contain 0 (so that zero, the padding value, is a code) and mapped onto
  [-128, 127];
* ``quantize_graph`` rewrites the serialized function into its int8 form:
  every node computes on codes ("out_dtype": "int8") and carries its
  tensor's (S, Z), inputs are quantized and outputs dequantized at the
  boundary by the executor.  A max pool keeps its input's parameters.

Weights need no calibration: the executor quantizes them per output channel
when it builds the engine.
"""

import copy
import json

import numpy as np

from . import capi


def affine_params(lo, hi):
    """int8 (scale, zero point) of the range [lo, hi] widened to hold 0."""
    lo, hi = min(float(lo), 0.0), max(float(hi), 0.0)
    if hi - lo <= 0.0:
        return 1.0, 0
    scale = (hi - lo) / 255.0
    zp = int(np.clip(np.rint(-128.0 - lo / scale), -128, 127))
    return scale, zp


def _load(graph):
    return json.loads(graph) if isinstance(graph, (str, bytes)) else graph


def calibration_graph(graph):
    """The float function with every node (and the original outputs) as an
    f32 output, in node order."""
    g = copy.deepcopy(_load(graph))
    g["outputs"] = [{"name": n["name"], "dtype": "f32"} for n in g["nodes"]]
    return g


def calibrate(graph, consts, batches, device=0):
    """Ranges {tensor name: (min, max)} of the inputs and node outputs of the
    float function over calibration batches (lists of device tensors, one
    per function input), computed by the executor."""
    import torch

    g = _load(graph)
    cg = calibration_graph(g)
    ranges = {}
    with capi.Subgraph(cg, consts, device=device) as sg:
        for inputs in batches:
            outs = []
            for i in range(sg.n_out):
                d = sg.io_desc(True, i)
                outs.append(torch.empty(d["shape"], dtype=torch.float32, device="cuda:%d" % device))
            sg.run(list(inputs), outs)
            torch.cuda.synchronize(device)
            merge_ranges(ranges, g, [t.float() for t in inputs], outs)
    return ranges


def merge_ranges(ranges, graph, inputs, node_values):
    """Widens ``ranges`` {tensor name: (min, max)} by one calibration batch:
    ``inputs`` in the order of the function's inputs and ``node_values`` in
    node order (arrays or tensors, any float type)."""
    g = _load(graph)

    def merge(name, t):
        lo, hi = float(t.min()), float(t.max())
        if name in ranges:
            lo, hi = min(lo, ranges[name][0]), max(hi, ranges[name][1])
        ranges[name] = (lo, hi)

    for desc, t in zip(g["inputs"], inputs):
        merge(desc["name"], t)
    for node, t in zip(g["nodes"], node_values):
        merge(node["name"], t)
    return ranges


def quantize_graph(graph, ranges):
    """The int8 form of a serialized function given each tensor's range."""
    g = copy.deepcopy(_load(graph))
    qp = {}
    for desc in g["inputs"]:
        s, z = affine_params(*ranges[desc["name"]])
        desc["quant"] = {"scale": s, "zero_point": z}
        qp[desc["name"]] = desc["quant"]
    for node in g["nodes"]:
        node["out_dtype"] = "int8"
        if node["composite"] == "max_pool2d":
            node["quant"] = dict(qp[node["inputs"][0]])
        else:
            s, z = affine_params(*ranges[node["name"]])
            node["quant"] = {"scale": s, "zero_point": z}
        qp[node["name"]] = node["quant"]
    for out in g["outputs"]:
        out.setdefault("dtype", "f32")
    return g
