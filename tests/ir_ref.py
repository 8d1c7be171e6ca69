"""Reference execution of operator-level graphs and of partitioned programs
for the partitioner tests (CPU, float64).

Operators follow the oracle's definitions (oracle.ops); the host-only
operators (sigmoid, softmax, multiply, reshape, transpose) are written out
here.  An offloaded function of a partitioned program runs through the
oracle's executor of the serialized form.
"""

import numpy as np

import oracle
from oracle import ops


def op_ref(node, args):
    op, a = node.op, node.attrs
    x = args[0]
    if op == "nn.conv2d":
        return ops.conv2d(x, args[1], tuple(a.get("strides", [1, 1])), tuple(a.get("padding", [0, 0, 0, 0])),
                          a.get("groups", 1))
    if op == "nn.dense":
        return ops.dense(x, args[1])
    if op == "nn.bias_add":
        return ops.bias_add(x, args[1])
    if op == "add":
        return ops.add(x, args[1])
    if op == "multiply":
        return np.asarray(x, np.float64) * np.asarray(args[1], np.float64)
    if op == "nn.relu":
        return ops.relu(x)
    if op == "clip":
        return np.clip(np.asarray(x, np.float64), a["a_min"], a["a_max"])
    if op == "nn.gelu":
        return ops.gelu(x)
    if op == "nn.leaky_relu":
        return ops.leaky_relu(x, float(a.get("alpha", 0.1)))
    if op == "sigmoid":
        return 1.0 / (1.0 + np.exp(-np.asarray(x, np.float64)))
    if op == "nn.softmax":
        z = np.asarray(x, np.float64)
        z = z - z.max(axis=a.get("axis", -1), keepdims=True)
        e = np.exp(z)
        return e / e.sum(axis=a.get("axis", -1), keepdims=True)
    if op == "nn.max_pool2d":
        return ops.max_pool2d(x, tuple(a["pool_size"]), tuple(a["strides"]), tuple(a.get("padding", [0, 0, 0, 0])))
    if op == "nn.avg_pool2d":
        return ops.avg_pool2d(x, tuple(a["pool_size"]), tuple(a.get("strides", [1, 1])),
                              tuple(a.get("padding", [0, 0, 0, 0])), bool(a.get("count_include_pad", False)))
    if op == "concatenate":
        return ops.concatenate(args, axis=1)
    if op == "nn.global_avg_pool2d":
        y = ops.global_avg_pool2d(x)
        return y.reshape(y.shape[0], y.shape[1], 1, 1)
    if op == "nn.batch_flatten":
        return np.asarray(x, np.float64).reshape(x.shape[0], -1)
    if op == "reshape":
        return np.asarray(x, np.float64).reshape(a["newshape"])
    if op == "transpose":
        return np.transpose(np.asarray(x, np.float64), a["axes"])
    raise ValueError(op)


def run_ir(g, inputs):
    """The unpartitioned graph, operator by operator."""
    vals = {}
    k = 0
    for n in g.nodes:
        if n.op == "input":
            vals[n.id] = np.asarray(inputs[k], np.float64)
            k += 1
        elif n.op == "const":
            vals[n.id] = np.asarray(n.value, np.float64)
        else:
            vals[n.id] = op_ref(n, [vals[i] for i in n.inputs])
    return [vals[o] for o in g.outputs]


def run_partitioned(part, inputs, mode="exact"):
    """The partitioned program: host steps by reference, offloaded
    functions through the oracle's executor of their serialized form."""
    g = part.graph
    vals = {}
    for nid, x in zip(g.inputs, inputs):
        vals[nid] = np.asarray(x, np.float64)
    for n in g.nodes:
        if n.op == "const":
            vals[n.id] = np.asarray(n.value, np.float64)
    for kind, ref in part.steps:
        if kind == "host":
            node = g.nodes[ref]
            y = op_ref(node, [vals[i] for i in node.inputs])
            if node.dtype == "bf16" and mode == "bf16io":
                y = oracle.round_bf16(y)
            vals[ref] = y
        else:
            fn = part.functions[ref]
            outs = oracle.run_graph(fn.graph, fn.consts, [vals[i] for i in fn.inputs], mode=mode)
            for oid, o in zip(fn.outputs, outs):
                vals[oid] = o
    return [vals[o] for o in g.outputs]
