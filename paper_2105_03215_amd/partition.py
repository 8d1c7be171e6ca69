"""Graph partitioning for the offloaded-subgraph executor (Sec. 3.1).

The compile-side step upstream of ``byoc_subgraph_create``: it takes a model
graph of operator-level nodes and produces the offloaded functions that the
executor runs, serialized in the JSON form of Sec. 3.3 (Option 1), plus the
host part of the graph that calls them.

* Operator-level graph (``Graph``): nodes named after the operators of the
  paper's high-level IR (``nn.conv2d``, ``nn.bias_add``, ``add``,
  ``nn.relu``, ``clip``, ``nn.leaky_relu``, ``nn.dense``, ``nn.max_pool2d``,
  ``nn.avg_pool2d``, ``concatenate``, ``nn.global_avg_pool2d``,
  ``nn.batch_flatten``, ...), each with its
  attributes, inferred shape and dtype; weights are constant nodes.
* Pattern-based grouping (Sec. 3.1.1): patterns built from ``wildcard()``,
  ``is_op(name)(*args)``, ``is_constant()``, ``.optional(fn)`` and ``|``;
  each match becomes one composite node named after its pattern.  An
  operator inside a match whose result is used outside it cannot be fused,
  so such matches are rejected.
* Annotation (Sec. 3.1.2): per-target predicates decide which composites
  and operators a target supports (here: every composite the executor
  implements, in float32 or bfloat16).
* Region merging (Sec. 3.1.2): supported nodes are merged greedily into
  regions, joining the regions of their producers whenever the graph of
  regions stays acyclic.
* Cost-based partitioning (Sec. 3.1.3): a region larger than a maximum
  number of operators is split in topological order; a region that fails
  the fallback criterion (by default ``CalcMAC(region) > 0``, the TensorRT
  rule of Sec. 4.1) stays on the host.
* Encapsulation and serialization (Sec. 3.1.3, 3.3): each offloaded region
  becomes a function with boundary inputs, constants and outputs, written in
  the executor's JSON schema.

Everything here is host-side Python over small graphs; nothing runs on the
device.
"""

import json

import numpy as np

# ---------------------------------------------------------------------------
# Operator-level graph
# ---------------------------------------------------------------------------


class Node:
    """One operator (or input / constant) of the operator-level graph."""

    def __init__(self, nid, op, inputs, attrs, shape, dtype, value=None, name=None):
        self.id = nid
        self.op = op
        self.inputs = list(inputs)
        self.attrs = dict(attrs)
        self.shape = tuple(int(d) for d in shape)
        self.dtype = dtype
        self.value = value
        self.name = name or "%s_%d" % (op.replace(".", "_"), nid)

    def __repr__(self):
        return "Node(%d, %s, %s)" % (self.id, self.op, list(self.inputs))


def _conv_out(h, r, stride, pb, pa):
    return (h + pb + pa - r) // stride + 1


def _pads(padding):
    return [int(v) for v in padding] if len(padding) == 4 else [int(padding[0]), int(padding[1])] * 2


def _infer(op, ins, attrs):
    """Output shape of an operator from its input shapes and attributes."""
    if op in ("nn.relu", "clip", "nn.gelu", "nn.leaky_relu", "sigmoid", "nn.softmax"):
        return ins[0]
    if op in ("add", "multiply"):
        if ins[0] != ins[1]:
            raise ValueError("%s: shapes %s and %s differ" % (op, ins[0], ins[1]))
        return ins[0]
    if op == "nn.bias_add":
        if len(ins[1]) != 1 or ins[1][0] != ins[0][1]:
            raise ValueError("nn.bias_add: bias %s does not match %s" % (ins[1], ins[0]))
        return ins[0]
    if op == "nn.conv2d":
        n, c, h, w = ins[0]
        k, cg, r, s = ins[1]
        g = attrs.get("groups", 1)
        if c != cg * g or k % g:
            raise ValueError("nn.conv2d: channels %d, weight %s, groups %d" % (c, ins[1], g))
        pt, pl, pb, pr = _pads(attrs.get("padding", [0, 0, 0, 0]))
        sh, sw = attrs.get("strides", [1, 1])
        return (n, k, _conv_out(h, r, sh, pt, pb), _conv_out(w, s, sw, pl, pr))
    if op == "nn.dense":
        m, kin = ins[0]
        nout, kin2 = ins[1]
        if kin != kin2:
            raise ValueError("nn.dense: %s x %s" % (ins[0], ins[1]))
        return (m, nout)
    if op == "nn.max_pool2d":
        n, c, h, w = ins[0]
        r, s = attrs["pool_size"]
        sh, sw = attrs["strides"]
        pt, pl, pb, pr = _pads(attrs.get("padding", [0, 0, 0, 0]))
        return (n, c, _conv_out(h, r, sh, pt, pb), _conv_out(w, s, sw, pl, pr))
    if op == "nn.avg_pool2d":
        n, c, h, w = ins[0]
        r, s = attrs["pool_size"]
        sh, sw = attrs.get("strides", [1, 1])
        pt, pl, pb, pr = _pads(attrs.get("padding", [0, 0, 0, 0]))
        return (n, c, _conv_out(h, r, sh, pt, pb), _conv_out(w, s, sw, pl, pr))
    if op == "concatenate":
        if attrs.get("axis", 1) != 1 or any(len(x) != 4 or (x[0], x[2], x[3]) != (ins[0][0], ins[0][2], ins[0][3])
                                            for x in ins):
            raise ValueError("concatenate: channel-axis join of NCHW tensors of one batch and image, got %s" % (ins,))
        return (ins[0][0], sum(x[1] for x in ins), ins[0][2], ins[0][3])
    if op == "nn.global_avg_pool2d":
        n, c = ins[0][:2]
        return (n, c, 1, 1)
    if op == "nn.batch_flatten":
        return (ins[0][0], int(np.prod(ins[0][1:])))
    if op == "reshape":
        shape = tuple(attrs["newshape"])
        if int(np.prod(shape)) != int(np.prod(ins[0])):
            raise ValueError("reshape: %s to %s" % (ins[0], shape))
        return shape
    if op == "transpose":
        return tuple(ins[0][a] for a in attrs["axes"])
    raise ValueError("unknown operator %s" % op)


class Graph:
    """Operator-level model graph; nodes are created in topological order."""

    def __init__(self):
        self.nodes = []
        self.inputs = []
        self.outputs = []

    def _add(self, op, inputs, attrs, shape, dtype, value=None, name=None):
        n = Node(len(self.nodes), op, inputs, attrs, shape, dtype, value, name)
        self.nodes.append(n)
        return n.id

    def input(self, name, shape, dtype="f32"):
        nid = self._add("input", [], {}, shape, dtype, name=name)
        self.inputs.append(nid)
        return nid

    def const(self, value, name=None):
        value = np.ascontiguousarray(value, dtype=np.float32)
        return self._add("const", [], {}, value.shape, "f32", value=value, name=name)

    def call(self, op, inputs, name=None, **attrs):
        dt = self.nodes[inputs[0]].dtype
        shape = _infer(op, [self.nodes[i].shape for i in inputs], attrs)
        return self._add(op, inputs, attrs, shape, dt, name=name)

    def output(self, nid):
        self.outputs.append(nid)

    def consumers(self):
        cons = {n.id: [] for n in self.nodes}
        for n in self.nodes:
            for i in n.inputs:
                cons[i].append(n.id)
        return cons


def macs(node, graph):
    """Multiply-accumulates of one operator (only conv2d and dense have any,
    as the paper's TensorRT study counts them, Sec. 4.1)."""
    if node.op == "nn.conv2d":
        n, k, p, q = node.shape
        _, cg, r, s = graph.nodes[node.inputs[1]].shape
        return n * k * p * q * cg * r * s
    if node.op == "nn.dense":
        m, nout = node.shape
        return m * nout * graph.nodes[node.inputs[0]].shape[1]
    return 0


# ---------------------------------------------------------------------------
# Patterns (Sec. 3.1.1)
# ---------------------------------------------------------------------------


class Pattern:
    """Matches a subgraph rooted at a node; records bound nodes by role."""

    def optional(self, fn):
        """``self`` alone or ``fn(self)``: the wrapped operator may be absent."""
        return AltPattern(fn(self), self)

    def __or__(self, other):
        return AltPattern(self, other)

    def match(self, g, nid, env):
        raise NotImplementedError


class WildcardPattern(Pattern):
    def __init__(self, role=None):
        self.role = role

    def match(self, g, nid, env):
        if self.role:
            env.setdefault("roles", {})[self.role] = nid
        env.setdefault("args", []).append(nid)
        return True


class ConstantPattern(WildcardPattern):
    def match(self, g, nid, env):
        return g.nodes[nid].op == "const" and super().match(g, nid, env)


class OpPattern(Pattern):
    def __init__(self, op, args, attrs=None, role=None):
        self.op = op
        self.args = args
        self.attrs = attrs or {}
        self.role = role

    def has_attr(self, **attrs):
        return OpPattern(self.op, self.args, dict(self.attrs, **attrs), self.role)

    def match(self, g, nid, env):
        n = g.nodes[nid]
        if n.op != self.op or len(n.inputs) != len(self.args):
            return False
        for k, v in self.attrs.items():
            if n.attrs.get(k) != v:
                return False
        for a, i in zip(self.args, n.inputs):
            if not a.match(g, i, env):
                return False
        env.setdefault("ops", []).append(nid)
        env.setdefault("by_op", {}).setdefault(self.op, []).append(nid)
        return True


class VariadicOpPattern(OpPattern):
    """An operator over any number (at least one) of arguments, each bound
    in order as a composite argument (e.g. ``concatenate``)."""

    def __init__(self, op):
        super().__init__(op, [])

    def match(self, g, nid, env):
        n = g.nodes[nid]
        if n.op != self.op or not n.inputs:
            return False
        for i in n.inputs:
            WildcardPattern().match(g, i, env)
        env.setdefault("ops", []).append(nid)
        env.setdefault("by_op", {}).setdefault(self.op, []).append(nid)
        return True


class AltPattern(Pattern):
    def __init__(self, first, second):
        self.first = first
        self.second = second

    def match(self, g, nid, env):
        trial = _copy_env(env)
        if self.first.match(g, nid, trial):
            env.clear()
            env.update(trial)
            return True
        return self.second.match(g, nid, env)


def _copy_env(env):
    out = {}
    for k, v in env.items():
        if isinstance(v, list):
            out[k] = list(v)
        elif isinstance(v, dict):
            out[k] = {kk: (list(vv) if isinstance(vv, list) else vv) for kk, vv in v.items()}
        else:
            out[k] = v
    return out


def wildcard(role=None):
    """Any input: a model input, a constant or another operator's result."""
    return WildcardPattern(role)


def is_constant(role=None):
    return ConstantPattern(role)


def is_op(op):
    """``is_op(name)(*args)``: an operator of that type over argument patterns."""
    return lambda *args: OpPattern(op, list(args))


# ---------------------------------------------------------------------------
# The executor's composite patterns
# ---------------------------------------------------------------------------

def _with_epilogue(core):
    """core -> optional bias_add -> optional residual add -> optional act."""
    biased = core.optional(lambda x: is_op("nn.bias_add")(x, is_constant("bias")))
    added = biased.optional(lambda x: is_op("add")(x, wildcard("residual")) |
                            is_op("add")(wildcard("residual"), x))
    return added.optional(lambda x: is_op("nn.relu")(x) |
                          is_op("clip")(x).has_attr(a_min=0.0, a_max=6.0) |
                          is_op("nn.gelu")(x) | is_op("nn.leaky_relu")(x))


def conv2d_pattern():
    return _with_epilogue(is_op("nn.conv2d")(wildcard("data"), is_constant("weight")))


def dense_pattern():
    return _with_epilogue(is_op("nn.dense")(wildcard("data"), is_constant("weight")))


def max_pool_pattern():
    return is_op("nn.max_pool2d")(wildcard("data"))


def avg_pool_pattern():
    return is_op("nn.avg_pool2d")(wildcard("data"))


def concat_pattern():
    return VariadicOpPattern("concatenate")


def global_avg_pool_pattern():
    return is_op("nn.batch_flatten")(is_op("nn.global_avg_pool2d")(wildcard("data")))


def add_pattern():
    return is_op("add")(wildcard("data"), wildcard("residual")).optional(
        lambda x: is_op("nn.relu")(x) | is_op("clip")(x).has_attr(a_min=0.0, a_max=6.0) |
        is_op("nn.leaky_relu")(x))


def _act_suffix(g, env):
    by = env.get("by_op", {})
    if "nn.relu" in by:
        return "_relu"
    if "clip" in by:
        return "_relu6"
    if "nn.gelu" in by:
        return "_gelu"
    if "nn.leaky_relu" in by:
        return "_leaky"
    return ""


def _gemm_name(base):
    def name(g, env):
        by = env.get("by_op", {})
        s = base
        if "nn.bias_add" in by:
            s += "_bias"
        if "add" in by:
            s += "_add"
        return s + _act_suffix(g, env)
    return name


# (pattern factory, composite naming) in priority order
PATTERN_TABLE = [
    (conv2d_pattern, _gemm_name("conv2d")),
    (dense_pattern, _gemm_name("dense")),
    (global_avg_pool_pattern, lambda g, env: "global_avg_pool2d"),
    (max_pool_pattern, lambda g, env: "max_pool2d"),
    (avg_pool_pattern, lambda g, env: "avg_pool2d"),
    (concat_pattern, lambda g, env: "concatenate"),
    (add_pattern, lambda g, env: "add" + _act_suffix(g, env)),
]


class Composite:
    """A matched operator sequence: its member operators, its root (whose
    result is the composite's), and its arguments by role."""

    def __init__(self, name, members, root, roles, arglist=None):
        self.name = name
        self.members = sorted(members)
        self.root = root
        self.roles = roles  # data, weight, bias, residual -> node id
        self.arglist = arglist  # variadic composites: every argument in order

    @property
    def args(self):
        if self.arglist is not None:
            return list(self.arglist)
        return [self.roles[r] for r in ("data", "weight", "bias", "residual") if r in self.roles]


def merge_composites(g, table=None):
    """Group operator sequences into composites (Sec. 3.1.1).

    Patterns are tried in table order; within a pattern, candidate roots in
    reverse topological order, so that a sequence is taken whole from its
    last operator.  A match is accepted when none of its operators belongs
    to an earlier match and no operator but its root has a consumer outside
    the match.  Returns {root id: Composite} and {member id: root id}."""
    table = PATTERN_TABLE if table is None else table
    cons = g.consumers()
    outs = set(g.outputs)
    comps, owner = {}, {}
    for factory, namer in table:
        pat = factory()
        for n in reversed(g.nodes):
            if n.op in ("input", "const") or n.id in owner:
                continue
            env = {}
            if not pat.match(g, n.id, env):
                continue
            members = set(env["ops"])
            if members & set(owner):
                continue
            inner_ok = all(m == n.id or (all(c in members for c in cons[m]) and m not in outs)
                           for m in members)
            if not inner_ok:
                continue
            name = namer(g, env)
            roles = dict(env.get("roles", {}))
            if name == "concatenate":
                roles["data"] = env["args"][0]
            comp = Composite(name, members, n.id, roles, list(env["args"]) if name == "concatenate" else None)
            if comp.name.startswith(("conv2d", "dense")) and "weight" not in comp.roles:
                continue
            comps[n.id] = comp
            for m in members:
                owner[m] = n.id
    return comps, owner


# ---------------------------------------------------------------------------
# Annotation (Sec. 3.1.2)
# ---------------------------------------------------------------------------

_SUPPORT = {}


def register_op_attr(name, target):
    """Decorator registering a predicate: does ``target`` support this
    composite (or operator) instance?"""
    def deco(fn):
        _SUPPORT[(target, name)] = fn
        return fn
    return deco


TARGET = "byoc.mi355x"
_DTYPES = ("f32", "bf16")


def _composite_family(name):
    for fam in ("conv2d", "dense", "max_pool2d", "global_avg_pool2d", "add"):
        if name == fam or name.startswith(fam + "_"):
            return fam
    return name


@register_op_attr("conv2d", TARGET)
def _conv_supported(g, comp):
    conv = g.nodes[[m for m in comp.members if g.nodes[m].op == "nn.conv2d"][0]]
    x = g.nodes[comp.roles["data"]]
    groups = conv.attrs.get("groups", 1)
    _, c, _, _ = x.shape
    k = conv.shape[1]
    r, s = g.nodes[comp.roles["weight"]].shape[2:]
    return (x.dtype in _DTYPES and conv.attrs.get("dilation", [1, 1]) == [1, 1] and r <= 15 and s <= 15 and
            (groups == 1 or groups == c == k))


@register_op_attr("dense", TARGET)
def _dense_supported(g, comp):
    return g.nodes[comp.roles["data"]].dtype in _DTYPES


@register_op_attr("max_pool2d", TARGET)
def _pool_supported(g, comp):
    return g.nodes[comp.roles["data"]].dtype in _DTYPES and len(g.nodes[comp.roles["data"]].shape) == 4


@register_op_attr("global_avg_pool2d", TARGET)
def _gap_supported(g, comp):
    return g.nodes[comp.roles["data"]].dtype in _DTYPES


@register_op_attr("avg_pool2d", TARGET)
def _avg_pool_supported(g, comp):
    x = g.nodes[comp.roles["data"]]
    return x.dtype == "bf16" and len(x.shape) == 4


@register_op_attr("concatenate", TARGET)
def _concat_supported(g, comp):
    xs = [g.nodes[a] for a in comp.args]
    return all(x.dtype == "bf16" and len(x.shape) == 4 and x.shape[1] % 8 == 0 for x in xs)


@register_op_attr("add", TARGET)
def _add_supported(g, comp):
    return g.nodes[comp.roles["data"]].dtype in _DTYPES


def annotate(g, comps, target=TARGET):
    """Root ids of the composites ``target`` supports.  Operators outside
    composites have no executor kernel of their own and stay on the host."""
    out = set()
    for root, comp in comps.items():
        fn = _SUPPORT.get((target, _composite_family(comp.name)))
        if fn is not None and fn(g, comp):
            out.add(root)
    return out


# ---------------------------------------------------------------------------
# Regions: greedy merge, cost-based split, host fallback (Sec. 3.1.2-3.1.3)
# ---------------------------------------------------------------------------


class Unit:
    """A schedulable piece of the grouped graph: one composite or one
    operator left ungrouped."""

    def __init__(self, uid, root, members, comp=None):
        self.id = uid
        self.root = root
        self.members = members
        self.comp = comp
        self.inputs = []  # unit ids it consumes

    @property
    def n_ops(self):
        return len(self.members)


def _units(g, comps, owner):
    units, of_node = [], {}
    for n in g.nodes:
        if n.op in ("input", "const"):
            continue
        if n.id in owner and owner[n.id] != n.id:
            continue  # a composite's member other than its root
        comp = comps.get(n.id)
        u = Unit(len(units), n.id, comp.members if comp else [n.id], comp)
        units.append(u)
        for m in u.members:
            of_node[m] = u.id
    for u in units:
        srcs = set()
        for m in u.members:
            for i in g.nodes[m].inputs:
                if i in of_node and of_node[i] != u.id:
                    srcs.add(of_node[i])
        u.inputs = sorted(srcs)
    return units, of_node


def _acyclic(units, assign):
    """Is the graph of groups (units contracted by ``assign``) acyclic?"""
    succ = {}
    for u in units:
        a = assign[u.id]
        for s in u.inputs:
            b = assign[s]
            if a != b:
                succ.setdefault(b, set()).add(a)
    groups = set(assign.values())
    indeg = {x: 0 for x in groups}
    for b, outs in succ.items():
        for a in outs:
            indeg[a] += 1
    ready = [x for x in groups if indeg[x] == 0]
    seen = 0
    while ready:
        x = ready.pop()
        seen += 1
        for a in succ.get(x, ()):
            indeg[a] -= 1
            if indeg[a] == 0:
                ready.append(a)
    return seen == len(groups)


def form_regions(units, supported):
    """Greedy merge of supported units (Sec. 3.1.2): in topological order,
    a supported unit joins the regions of its supported producers - all of
    them where the region graph stays acyclic, else the first that keeps it
    acyclic - or opens a region of its own.  Returns {unit id: group id};
    host units are groups of their own."""
    assign = {u.id: ("h", u.id) for u in units}
    next_region = 0
    for u in units:
        if u.id not in supported:
            continue
        cands = []
        for s in u.inputs:
            r = assign[s]
            if r[0] == "r" and r not in cands:
                cands.append(r)
        placed = False
        if cands:
            trial = dict(assign)
            target = cands[0]
            for uid, grp in trial.items():
                if grp in cands:
                    trial[uid] = target
            trial[u.id] = target
            if _acyclic(units, trial):
                assign = trial
                placed = True
            else:
                for r in cands:
                    trial = dict(assign)
                    trial[u.id] = r
                    if _acyclic(units, trial):
                        assign = trial
                        placed = True
                        break
        if not placed:
            assign[u.id] = ("r", next_region)
            next_region += 1
    return assign


def split_regions(units, assign, max_ops):
    """Cost-based split (Sec. 3.1.3): a region with more than ``max_ops``
    operators is cut, in topological order of its units, into consecutive
    pieces of at most ``max_ops`` operators (a composite is never cut)."""
    if not max_ops:
        return assign
    out = dict(assign)
    by_region = {}
    for u in units:
        if assign[u.id][0] == "r":
            by_region.setdefault(assign[u.id], []).append(u)
    fresh = max([g[1] for g in assign.values() if g[0] == "r"], default=-1) + 1
    for r, us in by_region.items():
        if sum(u.n_ops for u in us) <= max_ops:
            continue
        cur, count = r, 0
        for u in us:  # units are in topological order
            if count and count + u.n_ops > max_ops:
                cur = ("r", fresh)
                fresh += 1
                count = 0
            out[u.id] = cur
            count += u.n_ops
    return out


def calc_mac(g, units_in_region):
    return sum(macs(g.nodes[m], g) for u in units_in_region for m in u.members)


def host_fallback(g, units, assign, keep=None):
    """Regions failing ``keep(graph, units)`` (default CalcMAC > 0, the
    paper's TensorRT rule) go back to the host, unit by unit."""
    keep = keep or (lambda gr, us: calc_mac(gr, us) > 0)
    out = dict(assign)
    by_region = {}
    for u in units:
        if assign[u.id][0] == "r":
            by_region.setdefault(assign[u.id], []).append(u)
    for r, us in by_region.items():
        if not keep(g, us):
            for u in us:
                out[u.id] = ("h", u.id)
    return out


# ---------------------------------------------------------------------------
# Encapsulation and serialization (Sec. 3.1.3, Sec. 3.3 Option 1)
# ---------------------------------------------------------------------------


class Function:
    """An offloaded region: the JSON graph handed to byoc_subgraph_create,
    its constant list, and the operator-graph ids of its boundary tensors."""

    def __init__(self, name, graph_json, consts, inputs, outputs, units, n_ops, n_macs):
        self.name = name
        self.graph = graph_json
        self.consts = consts
        self.inputs = inputs    # node ids read from outside, in the JSON's input order
        self.outputs = outputs  # node ids used outside, in the JSON's output order
        self.units = units
        self.n_ops = n_ops
        self.macs = n_macs

    def json_bytes(self):
        return json.dumps(self.graph).encode()


def _layout(shape):
    return "NCHW" if len(shape) == 4 else "ROWMAJOR"


def _serialize(g, name, us, used_outside):
    """Write one region in the executor's schema: composites in topological
    order, inputs = tensors produced outside, outputs = results used
    outside; constants listed in first-use order."""
    members = {m for u in us for m in u.members}
    dtype = g.nodes[us[0].root].dtype
    tname = {}
    inputs, consts_ids, const_arrays, nodes_json, outputs = [], [], [], [], []

    def ref(nid):
        if nid in tname:
            return tname[nid]
        n = g.nodes[nid]
        if n.op == "const":
            cname = "c%d" % len(consts_ids)
            consts_ids.append(nid)
            const_arrays.append(n.value)
            tname[nid] = cname
            return cname
        if nid in members:
            raise ValueError("operator %d used before it is defined" % nid)
        iname = "in%d" % len(inputs)
        inputs.append(nid)
        tname[nid] = iname
        return iname

    for u in us:
        comp = u.comp
        args = [ref(a) for a in comp.args]
        attrs = {}
        if comp.name.startswith("conv2d"):
            conv = g.nodes[[m for m in comp.members if g.nodes[m].op == "nn.conv2d"][0]]
            attrs = {"strides": list(conv.attrs.get("strides", [1, 1])),
                     "padding": _pads(conv.attrs.get("padding", [0, 0, 0, 0])),
                     "dilation": [1, 1], "groups": conv.attrs.get("groups", 1)}
        if comp.name.endswith("_leaky"):
            act = g.nodes[[m for m in comp.members if g.nodes[m].op == "nn.leaky_relu"][0]]
            attrs["alpha"] = float(act.attrs.get("alpha", 0.1))
        elif comp.name == "max_pool2d":
            pool = g.nodes[comp.root]
            attrs = {"pool_size": list(pool.attrs["pool_size"]), "strides": list(pool.attrs["strides"]),
                     "padding": _pads(pool.attrs.get("padding", [0, 0, 0, 0]))}
        elif comp.name == "avg_pool2d":
            pool = g.nodes[comp.root]
            attrs = {"pool_size": list(pool.attrs["pool_size"]), "strides": list(pool.attrs.get("strides", [1, 1])),
                     "padding": _pads(pool.attrs.get("padding", [0, 0, 0, 0])),
                     "count_include_pad": bool(pool.attrs.get("count_include_pad", False))}
        elif comp.name == "concatenate":
            attrs = {"axis": 1}
        oname = "n%d" % len(nodes_json)
        nodes_json.append({"name": oname, "composite": comp.name, "inputs": args, "attrs": attrs,
                           "out_dtype": dtype})
        tname[u.root] = oname
    for u in us:
        if u.root in used_outside:
            outputs.append(u.root)
    const_desc = []
    for i, nid in enumerate(consts_ids):
        n = g.nodes[nid]
        d = {"name": "c%d" % i, "index": i, "shape": list(n.shape), "dtype": "f32",
             "layout": {4: "OIHW", 2: "OI", 1: "O"}.get(len(n.shape), "ROWMAJOR")}
        const_desc.append(d)
    graph_json = {
        "format": "byoc-subgraph", "version": 1, "meta": {"function": name},
        "inputs": [{"name": tname[i], "shape": list(g.nodes[i].shape), "dtype": g.nodes[i].dtype,
                    "layout": _layout(g.nodes[i].shape)} for i in inputs],
        "constants": const_desc,
        "nodes": nodes_json,
        "outputs": [{"name": tname[o], "dtype": dtype, "layout": _layout(g.nodes[o].shape)} for o in outputs],
    }
    return graph_json, const_arrays, inputs, outputs


class Partitioned:
    """Result of partitioning: the offloaded functions and the host program
    (a list of steps in topological order: ("host", node id) for an
    operator run on the host, ("call", function index) for an external call
    of an offloaded function)."""

    def __init__(self, graph, functions, steps, comps):
        self.graph = graph
        self.functions = functions
        self.steps = steps
        self.composites = comps

    def stats(self):
        g = self.graph
        ops = [n for n in g.nodes if n.op not in ("input", "const")]
        off_ops = sum(f.n_ops for f in self.functions)
        total_macs = sum(macs(n, g) for n in ops)
        off_macs = sum(f.macs for f in self.functions)
        return {"operators": len(ops), "offloaded_operators": off_ops, "functions": len(self.functions),
                "node_offload": off_ops / max(len(ops), 1),
                "mac_offload": off_macs / total_macs if total_macs else 0.0}


def partition(g, max_ops=None, keep=None, target=TARGET, table=None):
    """Run the whole flow of Sec. 3.1 on an operator-level graph."""
    comps, owner = merge_composites(g, table)
    units, of_node = _units(g, comps, owner)
    supported = {u.id for u in units if u.comp is not None and u.root in annotate(g, comps, target)}
    assign = form_regions(units, supported)
    assign = split_regions(units, assign, max_ops)
    assign = host_fallback(g, units, assign, keep)
    if not _acyclic(units, assign):
        raise AssertionError("partition produced a cyclic region graph")

    # group order: a topological order of the contracted graph, taking each
    # group when its last unit's turn comes (units are topologically sorted)
    cons = g.consumers()
    outs = set(g.outputs)
    groups = {}
    for u in units:
        groups.setdefault(assign[u.id], []).append(u)
    order = _group_order(units, assign)
    functions, steps = [], []
    for grp in order:
        us = groups[grp]
        if grp[0] == "h":
            for m in us[0].members:
                steps.append(("host", m))
            continue
        members = {m for u in us for m in u.members}
        used_outside = {m for m in members if m in outs or any(c not in members for c in cons[m])}
        name = "byoc_fn%d" % len(functions)
        gj, carr, fin, fout = _serialize(g, name, us, used_outside)
        functions.append(Function(name, gj, carr, fin, fout, us, len(members), calc_mac(g, us)))
        steps.append(("call", len(functions) - 1))
    return Partitioned(g, functions, steps, comps)


def _group_order(units, assign):
    succ, indeg = {}, {}
    first = {}
    for u in units:
        a = assign[u.id]
        indeg.setdefault(a, 0)
        first.setdefault(a, u.id)
        for s in u.inputs:
            b = assign[s]
            if a != b and a not in succ.setdefault(b, set()):
                succ[b].add(a)
                indeg[a] = indeg.get(a, 0) + 1
    ready = sorted([x for x, d in indeg.items() if d == 0], key=lambda x: first[x])
    order = []
    while ready:
        x = ready.pop(0)
        order.append(x)
        for a in sorted(succ.get(x, ()), key=lambda y: first[y]):
            indeg[a] -= 1
            if indeg[a] == 0:
                ready.append(a)
        ready.sort(key=lambda y: first[y])
    return order


# ---------------------------------------------------------------------------
# Operator-level form of a serialized subgraph
# ---------------------------------------------------------------------------


def lower_subgraph(graph, consts):
    """The operator-level graph of a composite graph in the executor's
    schema: each composite becomes its operator sequence (op, bias_add,
    add, activation).  With partition() this closes the loop: the patterns
    regroup exactly these sequences."""
    g = Graph()
    names = {}
    for d in graph["inputs"]:
        names[d["name"]] = g.input(d["name"], d["shape"], d["dtype"])
    for d in graph["constants"]:
        names[d["name"]] = g.const(np.asarray(consts[d["index"]], dtype=np.float32).reshape(d["shape"]),
                                   name=d["name"])
    for nd in graph["nodes"]:
        comp, ins, attrs = nd["composite"], [names[i] for i in nd["inputs"]], nd.get("attrs", {})
        if comp.startswith(("conv2d", "dense")):
            parts = comp.split("_")
            core = "nn.conv2d" if parts[0] == "conv2d" else "nn.dense"
            kw = {}
            if core == "nn.conv2d":
                kw = {"strides": list(attrs.get("strides", [1, 1])), "padding": _pads(attrs.get("padding", [0] * 4)),
                      "groups": attrs.get("groups", 1)}
            y = g.call(core, ins[:2], **kw)
            k = 2
            if "bias" in parts:
                y = g.call("nn.bias_add", [y, ins[k]])
                k += 1
            if "add" in parts:
                y = g.call("add", [y, ins[k]])
            act = parts[-1] if parts[-1] in ("relu", "relu6", "gelu", "leaky") else None
        elif comp == "max_pool2d":
            y = g.call("nn.max_pool2d", ins, pool_size=list(attrs["pool_size"]),
                       strides=list(attrs["strides"]), padding=_pads(attrs.get("padding", [0] * 4)))
            act = None
        elif comp == "global_avg_pool2d":
            y = g.call("nn.batch_flatten", [g.call("nn.global_avg_pool2d", ins)])
            act = None
        elif comp == "avg_pool2d":
            y = g.call("nn.avg_pool2d", ins, pool_size=list(attrs["pool_size"]), strides=list(attrs["strides"]),
                       padding=_pads(attrs.get("padding", [0] * 4)),
                       count_include_pad=bool(attrs.get("count_include_pad", False)))
            act = None
        elif comp == "concatenate":
            y = g.call("concatenate", ins, axis=1)
            act = None
        elif comp.startswith("add"):
            y = g.call("add", ins)
            act = comp.split("_")[1] if "_" in comp else None
        else:
            raise ValueError("unknown composite %s" % comp)
        if act == "relu":
            y = g.call("nn.relu", [y])
        elif act == "relu6":
            y = g.call("clip", [y], a_min=0.0, a_max=6.0)
        elif act == "gelu":
            y = g.call("nn.gelu", [y])
        elif act == "leaky":
            y = g.call("nn.leaky_relu", [y], alpha=float(attrs.get("alpha", 0.1)))
        names[nd["name"]] = y
    for o in graph["outputs"]:
        g.output(names[o["name"]])
    return g
