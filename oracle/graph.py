"""Executor of a serialized subgraph, one composite at a time.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The serialized form is the JSON graph representation of Sec. 3.3 (Option 1):
one node per composite function with its pattern name, attributes and input
references.  The runtime behaviour follows Sec. 3.4 / Fig. 6: constants are
given once, inputs are read, the nodes run in order and the outputs are
written.

A composite is applied as separate steps, in this order (Sec. 3.1.1 groups an
operator with an optional bias_add and a trailing activation; the optional
residual add comes before the activation, as in a ResNet block):

    y = op(x, w);  y = bias_add(y, b);  y = add(y, residual);  y = act(y)

Pattern names: ``conv2d[_bias][_add][_relu|_relu6|_gelu|_leaky]``,
``dense[_bias][_add][_relu|_relu6|_gelu|_leaky]``, ``max_pool2d``,
``global_avg_pool2d``, ``avg_pool2d`` (window mean; attrs pool_size,
strides, padding, count_include_pad, default false: the divisor counts only
positions inside the image), ``concatenate`` (any number of inputs joined
along the channel axis), ``add[_relu|_relu6|_leaky]``; a leaky ReLU takes
its slope from ``attrs.alpha`` (default 0.1).  Inputs of a node are listed in
the order data, weight, bias, residual.

Precision semantics.  A node whose ``out_dtype`` is "bf16" belongs to a bf16
graph: its activations are bf16 values, its weights are rounded to bf16 (ties
to even) and its bias stays as given.  Both modes do all arithmetic in
float64; they differ only in the storage rounding of results:

* ``exact``  - no rounding of node outputs.
* ``bf16io`` - every node output declared bf16 is rounded to bf16 before use,
  which is exactly the declared graph (bf16 storage between composites).

A graph input declared "f32" that feeds a bf16 node is rounded to bf16 at the
boundary (the partial-quantization cast of Sec. 3.2, Fig. 4a) in both modes.
"""

import json

import numpy as np

from . import ops
from .bf16 import round_bf16

_ACTS = ("relu6", "relu", "gelu", "leaky")


def load_graph(js):
    """Parse a JSON string (or accept an already parsed dict)."""
    if isinstance(js, (str, bytes)):
        return json.loads(js)
    return js


def parse_composite(name):
    """Split a pattern name into (op, has_bias, has_add, activation)."""
    if name in ("max_pool2d", "global_avg_pool2d", "avg_pool2d", "concatenate"):
        return name, False, False, None
    parts = name.split("_")
    op = parts[0]
    if op not in ("conv2d", "dense", "add"):
        raise ValueError("unknown composite %r" % name)
    rest = parts[1:]
    act = None
    if rest and rest[-1] in _ACTS:
        act = rest.pop()
    has_bias = has_add = False
    if op == "add":
        if rest:
            raise ValueError("unknown composite %r" % name)
        return op, False, True, act
    if rest and rest[0] == "bias":
        has_bias = True
        rest = rest[1:]
    if rest and rest[0] == "add":
        has_add = True
        rest = rest[1:]
    if rest:
        raise ValueError("unknown composite %r" % name)
    return op, has_bias, has_add, act


def _store(y, dtype, mode):
    if mode == "bf16io" and dtype == "bf16":
        return round_bf16(y)
    if mode not in ("bf16io", "exact"):
        raise ValueError("mode must be 'exact' or 'bf16io'")
    return y


def run_node(node, args, mode="bf16io"):
    """Compute one composite node.

    ``args`` are the node's inputs as float64 arrays in the order of
    ``node["inputs"]`` (data, weight, bias, residual), with weights as given
    in the constant list (not yet rounded).  Returns the node output after
    the storage rounding of ``mode``.
    """
    name = node["composite"]
    attrs = node.get("attrs", {})
    dtype = node.get("out_dtype", "f32")
    op, has_bias, has_add, act = parse_composite(name)
    args = [np.asarray(a, dtype=np.float64) for a in args]
    if op in ("conv2d", "dense"):
        x, w = args[0], args[1]
        if dtype == "bf16":
            w = round_bf16(w)
        if op == "conv2d":
            y = ops.conv2d(x, w, tuple(attrs.get("strides", (1, 1))),
                           tuple(attrs.get("padding", (0, 0, 0, 0))),
                           int(attrs.get("groups", 1)))
        else:
            y = ops.dense(x, w)
        i = 2
        if has_bias:
            y = ops.bias_add(y, args[i])
            i += 1
        if has_add:
            y = ops.add(y, args[i])
            i += 1
    elif op == "add":
        y = ops.add(args[0], args[1])
    elif op == "max_pool2d":
        y = ops.max_pool2d(args[0], tuple(attrs.get("pool_size", (3, 3))),
                           tuple(attrs.get("strides", (2, 2))),
                           tuple(attrs.get("padding", (1, 1, 1, 1))))
    elif op == "avg_pool2d":
        y = ops.avg_pool2d(args[0], tuple(attrs.get("pool_size", (3, 3))),
                           tuple(attrs.get("strides", (1, 1))),
                           tuple(attrs.get("padding", (1, 1, 1, 1))),
                           bool(attrs.get("count_include_pad", False)))
    elif op == "concatenate":
        y = ops.concatenate(args, axis=1)
    else:
        y = ops.global_avg_pool2d(args[0])
    if act is not None:
        if act == "leaky":
            y = ops.leaky_relu(y, float(attrs.get("alpha", 0.1)))
        else:
            y = ops.ACTIVATIONS[act](y)
    return _store(y, dtype, mode)


def _graph_dtype_of_consumers(graph, name):
    for node in graph["nodes"]:
        if name in node["inputs"]:
            return node.get("out_dtype", "f32")
    return None


def run_graph(graph, consts, inputs, mode="bf16io", keep=False):
    """Execute the subgraph on host arrays.

    graph   JSON string or parsed dict.
    consts  list of arrays indexed by each constant's ``index``.
    inputs  list of arrays in the order of ``graph["inputs"]``.
    Returns the list of outputs (float64, external layout) or, with
    ``keep=True``, the dict of every named value as well.
    """
    g = load_graph(graph)
    vals = {}
    if len(inputs) != len(g["inputs"]):
        raise ValueError("expected %d inputs" % len(g["inputs"]))
    for desc, arr in zip(g["inputs"], inputs):
        a = np.asarray(arr, dtype=np.float64)
        if list(a.shape) != list(desc["shape"]):
            raise ValueError("input %s: shape %s != %s" % (desc["name"], a.shape, desc["shape"]))
        consumer = _graph_dtype_of_consumers(g, desc["name"])
        if desc.get("dtype") == "bf16" or consumer == "bf16":
            a = round_bf16(a)
        vals[desc["name"]] = a
    for c in g.get("constants", []):
        vals[c["name"]] = np.asarray(consts[c["index"]], dtype=np.float64)
    for node in g["nodes"]:
        args = [vals[ref] for ref in node["inputs"]]
        vals[node["name"]] = run_node(node, args, mode)
    outs = []
    for o in g["outputs"]:
        y = vals[o["name"]]
        if o.get("dtype") == "bf16":
            y = round_bf16(y) if mode == "bf16io" else y
        outs.append(y)
    if keep:
        return outs, vals
    return outs
