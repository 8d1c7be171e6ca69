"""Runtime of a partitioned model (Sec. 3.4, Fig. 6).

A ``Partitioned`` program (see ``partition.py``) is a list of steps: host
operators and external calls of offloaded functions.  ``Module`` runs it:

* metadata module - on creation it loads every constant the host operators
  use into data entries on the device, and builds the execution engine of
  each offloaded function once (``byoc_subgraph_create`` with the function's
  JSON and constants; the engine packs its own copy), cached for every later
  inference;
* data entries - one device tensor per graph input, constant and step
  result, addressed by the operator-graph id assigned at partitioning;
  intermediates inside an offloaded function are the engine's own and never
  appear here;
* execution - the steps in order: a host operator reads its input entries,
  computes on the device with PyTorch and writes its entry; an external call
  hands its input entries and freshly allocated output entries to the
  engine's run on the module's stream.

Host operators compute in float32 and store in the node's dtype.  The
offloaded functions run only through the HIP library: there is no other
path for them.
"""

import math

import torch
import torch.nn.functional as F

from . import capi


def _tdt(dtype):
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def _pads(p):
    return [int(v) for v in p] if len(p) == 4 else [int(p[0]), int(p[1])] * 2


def _host_op(node, args):
    """One host operator on float32 device tensors."""
    op, a = node.op, node.attrs
    x = args[0]
    if op == "nn.conv2d":
        pt, pl, pb, pr = _pads(a.get("padding", [0, 0, 0, 0]))
        x = F.pad(x, (pl, pr, pt, pb))
        return F.conv2d(x, args[1], stride=tuple(a.get("strides", [1, 1])), groups=a.get("groups", 1))
    if op == "nn.dense":
        return x @ args[1].t().contiguous()
    if op == "nn.bias_add":
        return x + args[1].view([1, -1] + [1] * (x.dim() - 2))
    if op == "add":
        return x + args[1]
    if op == "multiply":
        return x * args[1]
    if op == "nn.relu":
        return torch.relu(x)
    if op == "clip":
        return torch.clamp(x, a["a_min"], a["a_max"])
    if op == "nn.leaky_relu":
        return F.leaky_relu(x, float(a.get("alpha", 0.1)))
    if op == "nn.gelu":
        return 0.5 * x * (1.0 + torch.erf(x / math.sqrt(2.0)))
    if op == "sigmoid":
        return torch.sigmoid(x)
    if op == "nn.softmax":
        return torch.softmax(x, dim=a.get("axis", -1))
    if op == "nn.max_pool2d":
        pt, pl, pb, pr = _pads(a.get("padding", [0, 0, 0, 0]))
        x = F.pad(x, (pl, pr, pt, pb), value=-math.inf)
        return F.max_pool2d(x, tuple(a["pool_size"]), stride=tuple(a["strides"]))
    if op == "nn.avg_pool2d":
        pt, pl, pb, pr = _pads(a.get("padding", [0, 0, 0, 0]))
        if (pt, pl) != (pb, pr):
            raise ValueError("nn.avg_pool2d on the host: asymmetric padding")
        return F.avg_pool2d(x, tuple(a["pool_size"]), stride=tuple(a.get("strides", [1, 1])), padding=(pt, pl),
                            count_include_pad=bool(a.get("count_include_pad", False)))
    if op == "concatenate":
        return torch.cat(list(args), dim=1)
    if op == "nn.global_avg_pool2d":
        return x.mean(dim=(2, 3), keepdim=True)
    if op == "nn.batch_flatten":
        return x.reshape(x.shape[0], -1)
    if op == "reshape":
        return x.reshape(tuple(a["newshape"]))
    if op == "transpose":
        return x.permute(*a["axes"]).contiguous()
    raise ValueError("no host implementation of %s" % op)


class Module:
    """Executable form of a partitioned model on one device.

    Every step result (host operator or function output) has a data entry
    allocated once at creation, as the paper's data entries are (fixed IDs,
    preallocated): a run writes them in place, so the tensors ``run``
    returns are valid until the next run, and each engine sees the same
    buffers on every run, which lets it replay its launch sequence as a HIP
    graph (``graph_replay``)."""

    def __init__(self, part, device="cuda:0", graph_replay=False):
        self.part = part
        self.device = torch.device(device)
        self.dev_index = self.device.index or 0
        g = part.graph
        # metadata module: constants used by host operators, as data entries
        used_by_host = set()
        for kind, ref in part.steps:
            if kind == "host":
                used_by_host.update(g.nodes[ref].inputs)
        self.const_entries = {}
        for n in g.nodes:
            if n.op == "const" and n.id in used_by_host:
                self.const_entries[n.id] = torch.from_numpy(n.value).to(self.device, torch.float32)
        # one cached execution engine per offloaded function
        self.engines = [capi.Subgraph(f.graph, f.consts, device=self.dev_index) for f in part.functions]
        if graph_replay:
            for e in self.engines:
                e.set_options(graph_replay=True)
        # data entries of every step result
        self.data = {}
        for kind, ref in part.steps:
            if kind == "host":
                node = g.nodes[ref]
                self.data[ref] = torch.empty(tuple(node.shape), dtype=_tdt(node.dtype), device=self.device)
            else:
                eng = self.engines[ref]
                for j, oid in enumerate(part.functions[ref].outputs):
                    d = eng.io_desc(1, j)
                    self.data[oid] = torch.empty(d["shape"], dtype=_tdt(d["dtype"]), device=self.device)

    def close(self):
        for e in self.engines:
            e.close()
        self.engines = []

    def run(self, inputs, stream=None):
        """Run one inference; ``inputs`` are device tensors in the order of
        the graph's inputs.  Returns the graph's outputs (device tensors)."""
        g = self.part.graph
        stream = stream or torch.cuda.current_stream(self.device)
        entries = dict(self.const_entries)
        entries.update(self.data)
        # the inputs' producers ran on the caller's current stream
        stream.wait_stream(torch.cuda.current_stream(self.device))
        with torch.cuda.stream(stream):
            for nid, t in zip(g.inputs, inputs):
                # converted on the run stream; a converted copy is a new
                # allocation of that stream's pool, the input itself may
                # belong to another stream's pool
                x = t.to(self.device, _tdt(g.nodes[nid].dtype)).contiguous()
                if x.data_ptr() == t.data_ptr() and x.device.type == "cuda":
                    x.record_stream(stream)
                entries[nid] = x
            for kind, ref in self.part.steps:
                if kind == "host":
                    node = g.nodes[ref]
                    args = [entries[i].float() for i in node.inputs]
                    self.data[ref].copy_(_host_op(node, args).reshape(self.data[ref].shape))
                else:
                    fn = self.part.functions[ref]
                    self.engines[ref].run([entries[i] for i in fn.inputs], [self.data[o] for o in fn.outputs],
                                          stream)
        return [entries[o] for o in g.outputs]
