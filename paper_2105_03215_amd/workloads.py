"""Seeded synthetic subgraphs shaped like the paper's offloaded workloads.

The paper evaluates fully offloaded image classifiers (ResNet-18, ResNet-50,
MobileNetV2 among them; Table 1, Sec. 4.1) with trained weights on ImageNet.
Neither is available here, so every workload is synthetic: random weights of
the same architecture and random inputs of the same shape, drawn from fixed
seeds.  This module builds, for each workload, the serialized subgraph (the
JSON graph representation of Sec. 3.3, Option 1), the constant list handed
over once at engine creation (Sec. 3.4, metadata module) and the inputs.

It holds no operator arithmetic: it draws random numbers and folds a
batch-norm into conv weights using layer-wide statistics predicted by a
scalar second-moment model (see ``GraphBuilder``), not measured by running
the network.  The same arrays feed the HIP library and the CPU checker.

Seeding: tensor ``t`` of workload ``cid`` is drawn from
``np.random.default_rng(np.random.SeedSequence([cid, t]))``; tensor 0 is the
input, constants follow in creation order, and the batch-norm shift of the
i-th folded conv uses tensor id 1_000_000 + i.
"""

import json
import math

import numpy as np

CONFIG_IDS = {
    "conv_f32": 0,
    "resnet18_block": 1,
    "resnet50_v1": 2,
    "mobilenet_v2": 3,
    "bert_ffn": 4,
    "vgg19": 5,
    "darknet53": 6,
    "inception_v3": 7,
}

_BN_EPS = 1e-5
_BN_SHIFT_STD = 0.01
# mean square of a 3x3 max over ReLU outputs relative to its input's: the max
# of 9 independent standard normals has mean 1.485 and variance 0.357, so
# E[max^2] = 2.56 s^2 against E[relu^2] = s^2 / 2
_MAXPOOL_GAIN = 5.1
# 2x2 windows of neighbouring conv outputs are far from independent: the
# mean-square gain of a 2x2 max over them is taken as 2 (the independent
# bound would be 3.1)
_MAXPOOL_GAIN_2X2 = 2.0
# share of a non-negative activation's mean square that its spatial mean keeps
_GAP_GAIN = 0.5
_ADD_RELU_KEEP = 0.75


class Workload:
    """A serialized subgraph with its constants and inputs.

    graph   dict in the JSON schema accepted by ``byoc_subgraph_create``
    consts  list of float32 arrays, indexed by each constant's ``index``
    inputs  list of float32 arrays in the order of ``graph["inputs"]``
            (bf16-declared inputs hold values already representable in bf16)
    macs    multiply-accumulates of the conv and dense composites
    """

    def __init__(self, graph, consts, inputs, macs, conv_macs):
        self.graph = graph
        self.consts = consts
        self.inputs = inputs
        self.macs = macs
        self.conv_macs = conv_macs

    @property
    def json(self):
        return json.dumps(self.graph)

    @property
    def batch(self):
        return self.graph["inputs"][0]["shape"][0]


def to_bf16_values(a):
    """Round float32 values to bfloat16 (ties to even) and return float32.

    Input preparation only: a bf16-declared input must already hold bf16
    values, so the generator rounds its random draws once.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    u = (u + 0x7FFF + lsb) >> 16
    return (u.astype(np.uint32) << 16).view(np.float32)


class GraphBuilder:
    """Accumulates nodes and constants of one synthetic subgraph.

    Weight scales follow a scalar second-moment model: with zero-mean random
    weights, the mean square of a linear layer's output, averaged over output
    channels, is fan_in * var(w) * E[x^2] in expectation over the weight draw,
    whatever the correlations of the input; ReLU keeps half of it because the
    weight draw makes each channel's pre-activation symmetric.  A folded
    batch-norm uses these layer-wide statistics (mean 0, variance the
    predicted mean square) so that every normalized conv output has a mean
    square of about 1.
    """

    def __init__(self, name, cid, dtype="bf16"):
        self.name = name
        self.cid = cid
        self.dtype = dtype
        self.inputs = []
        self.input_arrays = []
        self.constants = []
        self.const_arrays = []
        self.nodes = []
        self.outputs = []
        self.shapes = {}
        self.m2 = {}
        self.mu = {}  # layer-wide mean of a tensor, where it is not ~0 (activation outputs, the image)
        self.next_tensor = 1
        self.n_folded = 0
        self.macs = 0
        self.conv_macs = 0

    # -- random draws ------------------------------------------------------
    def rng(self, tensor_id):
        return np.random.default_rng(np.random.SeedSequence([self.cid, tensor_id]))

    def _const(self, name, arr, layout):
        idx = len(self.const_arrays)
        self.constants.append({"name": name, "index": idx, "shape": list(arr.shape),
                               "dtype": "f32", "layout": layout})
        self.const_arrays.append(np.ascontiguousarray(arr, dtype=np.float32))
        return name

    # -- graph construction ------------------------------------------------
    def input(self, name, shape, dist="uniform", dtype=None, layout=None):
        dtype = dtype or self.dtype
        rng = self.rng(0 if not self.inputs else 100 + len(self.inputs))
        if dist == "uniform":
            a = rng.random(shape, dtype=np.float64).astype(np.float32)
            m2 = 1.0 / 3.0
        elif dist == "normal":
            a = rng.standard_normal(shape, dtype=np.float64).astype(np.float32)
            m2 = 1.0
        else:
            raise ValueError(dist)
        if dtype == "bf16":
            a = to_bf16_values(a)
        if layout is None:
            layout = "NCHW" if len(shape) == 4 else "ROWMAJOR"
        self.inputs.append({"name": name, "shape": list(shape), "dtype": dtype, "layout": layout})
        self.input_arrays.append(a)
        self.shapes[name] = list(shape)
        self.m2[name] = m2
        self.mu[name] = 0.5 if dist == "uniform" else 0.0
        return name

    def _after_add_act(self, m2_stream, m2_branch, act):
        if not act:
            return m2_stream + m2_branch
        # the stream is non-negative after its own ReLU and the branch is
        # symmetric: between half and all of the branch survives the ReLU
        return m2_stream + _ADD_RELU_KEEP * m2_branch

    def conv(self, x, k, r, stride=1, pad=None, groups=1, act="relu", bias=True, residual=None,
             bn=True, gamma=1.0, w_std=None, b_std=None, name=None, alpha=0.1):
        """Conv composite with He-normal weights and an optional folded BN.
        ``r`` is the kernel size, or (rows, columns) for a rectangular one."""
        n, c, h, w = self.shapes[x]
        r, sk = (r, r) if isinstance(r, int) else tuple(r)
        pad = [r // 2, sk // 2, r // 2, sk // 2] if pad is None else pad
        pads = [pad] * 4 if isinstance(pad, int) else list(pad)
        strides = [stride, stride] if isinstance(stride, int) else list(stride)
        cg = c // groups
        fan_in = cg * r * sk
        tid = self.next_tensor
        self.next_tensor += 2
        std = w_std if w_std is not None else math.sqrt(2.0 / fan_in)
        wt = self.rng(tid).normal(0.0, std, size=(k, cg, r, sk))
        m2_in = self.m2[x]
        if bn:
            var_pred = fan_in * std * std * m2_in
            beta = self.rng(1_000_000 + self.n_folded).normal(0.0, _BN_SHIFT_STD, size=k)
            self.n_folded += 1
            wt = wt * (gamma / math.sqrt(var_pred + _BN_EPS))
            b = beta
            m2 = gamma * gamma + _BN_SHIFT_STD ** 2
        else:
            bs = b_std if b_std is not None else 0.01
            b = self.rng(tid + 1).normal(0.0, bs, size=k)
            m2 = fan_in * std * std * m2_in + bs * bs
        name = name or "n%d" % len(self.nodes)
        wname = self._const(name + ".w", wt, "OIHW")
        ins = [x, wname]
        comp = "conv2d"
        if bias:
            ins.append(self._const(name + ".b", b, "O"))
            comp += "_bias"
        if residual is not None:
            ins.append(residual)
            comp += "_add"
            m2 = self._after_add_act(self.m2[residual], m2, act)
        elif act == "leaky":
            # the negative half keeps alpha^2 of its share; the output's mean
            # is (1 - alpha) sigma / sqrt(2 pi) for a symmetric pre-activation
            self.mu[name or "n%d" % len(self.nodes)] = (1.0 - alpha) * math.sqrt(m2 / (2.0 * math.pi))
            m2 = 0.5 * (1.0 + alpha * alpha) * m2
        elif act:
            if act in ("relu", "relu6"):
                self.mu[name] = math.sqrt(m2 / (2.0 * math.pi))
            m2 = 0.5 * m2
        if act:
            comp += "_" + act
        p = (h + pads[0] + pads[2] - r) // strides[0] + 1
        q = (w + pads[1] + pads[3] - sk) // strides[1] + 1
        attrs = {"strides": strides, "padding": pads, "dilation": [1, 1], "groups": groups}
        if act == "leaky":
            attrs["alpha"] = alpha
        self.nodes.append({"name": name, "composite": comp, "inputs": ins, "attrs": attrs,
                           "out_dtype": self.dtype})
        self.shapes[name] = [n, k, p, q]
        self.m2[name] = m2
        macs = n * k * p * q * cg * r * sk
        self.macs += macs
        self.conv_macs += macs
        return name

    def dense(self, x, n_out, act=None, residual=None, w_std=None, b_std=0.01, name=None):
        m, kin = self.shapes[x]
        tid = self.next_tensor
        self.next_tensor += 2
        std = w_std if w_std is not None else math.sqrt(2.0 / kin)
        wt = self.rng(tid).normal(0.0, std, size=(n_out, kin))
        b = self.rng(tid + 1).normal(0.0, b_std, size=n_out)
        name = name or "n%d" % len(self.nodes)
        ins = [x, self._const(name + ".w", wt, "OI"), self._const(name + ".b", b, "O")]
        comp = "dense_bias"
        m2 = kin * std * std * self.m2[x] + b_std * b_std
        if residual is not None:
            ins.append(residual)
            comp += "_add"
            m2 = self._after_add_act(self.m2[residual], m2, act)
        elif act:
            m2 = 0.5 * m2
        if act:
            comp += "_" + act
        self.nodes.append({"name": name, "composite": comp, "inputs": ins, "attrs": {},
                           "out_dtype": self.dtype})
        self.shapes[name] = [m, n_out]
        self.m2[name] = m2
        self.macs += m * n_out * kin
        return name

    def max_pool(self, x, size=3, stride=2, pad=1, name=None, gain=None):
        n, c, h, w = self.shapes[x]
        name = name or "n%d" % len(self.nodes)
        self.nodes.append({"name": name, "composite": "max_pool2d", "inputs": [x],
                           "attrs": {"pool_size": [size, size], "strides": [stride, stride],
                                     "padding": [pad] * 4},
                           "out_dtype": self.dtype})
        p = (h + 2 * pad - size) // stride + 1
        q = (w + 2 * pad - size) // stride + 1
        self.shapes[name] = [n, c, p, q]
        if gain is None:
            gain = _MAXPOOL_GAIN_2X2 if size == 2 else _MAXPOOL_GAIN
        self.m2[name] = gain * self.m2[x]
        return name

    def avg_pool(self, x, size=3, stride=1, pad=1, name=None):
        """Windowed average pool (padding not counted in the divisor)."""
        n, c, h, w = self.shapes[x]
        name = name or "n%d" % len(self.nodes)
        self.nodes.append({"name": name, "composite": "avg_pool2d", "inputs": [x],
                           "attrs": {"pool_size": [size, size], "strides": [stride, stride],
                                     "padding": [pad] * 4, "count_include_pad": False},
                           "out_dtype": self.dtype})
        self.shapes[name] = [n, c, (h + 2 * pad - size) // stride + 1, (w + 2 * pad - size) // stride + 1]
        mu = self.mu.get(x, 0.0)
        # the window mean keeps the mean and averages the rest over
        # correlated neighbours (taken to keep half of it)
        self.m2[name] = mu * mu + 0.5 * (self.m2[x] - mu * mu)
        self.mu[name] = mu
        return name

    def concat(self, xs, name=None):
        """Channel concatenation of NCHW tensors of one batch and image."""
        name = name or "n%d" % len(self.nodes)
        self.nodes.append({"name": name, "composite": "concatenate", "inputs": list(xs), "attrs": {"axis": 1},
                           "out_dtype": self.dtype})
        n, _, h, w = self.shapes[xs[0]]
        cs = [self.shapes[x][1] for x in xs]
        self.shapes[name] = [n, sum(cs), h, w]
        self.m2[name] = sum(c * self.m2[x] for c, x in zip(cs, xs)) / sum(cs)
        self.mu[name] = sum(c * self.mu.get(x, 0.0) for c, x in zip(cs, xs)) / sum(cs)
        return name

    def global_avg_pool(self, x, name=None):
        n, c, h, w = self.shapes[x]
        name = name or "n%d" % len(self.nodes)
        self.nodes.append({"name": name, "composite": "global_avg_pool2d", "inputs": [x],
                           "attrs": {}, "out_dtype": self.dtype})
        self.shapes[name] = [n, c]
        self.m2[name] = _GAP_GAIN * self.m2[x]
        return name

    def add(self, a, b, act=None, name=None):
        name = name or "n%d" % len(self.nodes)
        comp = "add" + ("_" + act if act else "")
        self.nodes.append({"name": name, "composite": comp, "inputs": [a, b], "attrs": {},
                           "out_dtype": self.dtype})
        self.shapes[name] = list(self.shapes[a])
        mu_a, mu_b = self.mu.get(a, 0.0), self.mu.get(b, 0.0)
        # E[(a + b)^2] = E[a^2] + E[b^2] + 2 E[a b]; the means of two
        # activated tensors add coherently (zero for zero-mean operands)
        self.m2[name] = self._after_add_act(self.m2[a], self.m2[b], act) + (0.0 if act else 2.0 * mu_a * mu_b)
        if not act:
            self.mu[name] = mu_a + mu_b
        return name

    def output(self, x, dtype=None, layout=None):
        shape = self.shapes[x]
        if layout is None:
            layout = "NCHW" if len(shape) == 4 else "ROWMAJOR"
        self.outputs.append({"name": x, "dtype": dtype or self.dtype, "layout": layout})

    def finish(self, meta=None):
        graph = {"format": "byoc-subgraph", "version": 1,
                 "meta": dict({"workload": self.name, "seed_config_id": self.cid}, **(meta or {})),
                 "inputs": self.inputs, "constants": self.constants, "nodes": self.nodes,
                 "outputs": self.outputs}
        return Workload(graph, self.const_arrays, self.input_arrays, self.macs, self.conv_macs)


# ---------------------------------------------------------------------------
# The five workloads
# ---------------------------------------------------------------------------

def conv_f32(n=1, c=16, hw=32, k=32):
    """One conv2d(3x3, s1, p1)+bias+ReLU composite in fp32.

    x U[0,1), W N(0, 0.1), b N(0, 0.01).
    """
    g = GraphBuilder("conv_f32", CONFIG_IDS["conv_f32"], dtype="f32")
    x = g.input("x", [n, c, hw, hw], "uniform")
    y = g.conv(x, k, 3, stride=1, pad=1, act="relu", bn=False, w_std=0.1, b_std=0.01, name="conv")
    g.output(y)
    return g.finish({"batch": n})


def resnet18_block(n=1, c=64, hw=56):
    """ResNet-18 basic block: conv3x3+bias+ReLU, conv3x3+bias, +x, ReLU (bf16)."""
    g = GraphBuilder("resnet18_block", CONFIG_IDS["resnet18_block"])
    x = g.input("x", [n, c, hw, hw], "uniform")
    a = g.conv(x, c, 3, act="relu", name="conv1")
    y = g.conv(a, c, 3, act="relu", residual=x, name="conv2")
    g.output(y)
    return g.finish({"batch": n})


def _bottleneck(g, x, mid, out, stride, downsample, stride_on, prefix):
    s1 = stride if stride_on == "1x1" else 1
    s3 = stride if stride_on == "3x3" else 1
    sc = x
    if downsample:
        sc = g.conv(x, out, 1, stride=stride, pad=0, act=None, name=prefix + ".down")
    a = g.conv(x, mid, 1, stride=s1, pad=0, act="relu", name=prefix + ".a")
    b = g.conv(a, mid, 3, stride=s3, pad=1, act="relu", name=prefix + ".b")
    return g.conv(b, out, 1, stride=1, pad=0, act="relu", residual=sc, name=prefix + ".c")


def resnet50(n=1, hw=224, variant="v1", input_dtype="bf16", num_classes=1000):
    """ResNet-50 v1 (stride on the first 1x1 of a downsampling block) or v1b
    (stride on the 3x3), batch-norm folded, max-pool, global average pool and
    the 2048->1000 classifier; bf16 activations."""
    g = GraphBuilder("resnet50_" + variant, CONFIG_IDS["resnet50_v1"])
    x = g.input("x", [n, 3, hw, hw], "uniform", dtype=input_dtype)
    y = g.conv(x, 64, 7, stride=2, pad=3, act="relu", name="stem")
    y = g.max_pool(y, 3, 2, 1, name="pool")
    stride_on = "1x1" if variant == "v1" else "3x3"
    cin = 64
    for si, (mid, blocks, stride) in enumerate([(64, 3, 1), (128, 4, 2), (256, 6, 2), (512, 3, 2)]):
        out = mid * 4
        for bi in range(blocks):
            st = stride if bi == 0 else 1
            y = _bottleneck(g, y, mid, out, st, bi == 0, stride_on, "s%d.b%d" % (si + 1, bi))
        cin = out
    y = g.global_avg_pool(y, name="gap")
    y = g.dense(y, num_classes, name="fc")
    g.output(y)
    del cin
    return g.finish({"batch": n, "variant": variant})


_MBV2_SETTINGS = [(1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 3, 2), (6, 64, 4, 2),
                  (6, 96, 3, 1), (6, 160, 3, 2), (6, 320, 1, 1)]


def mobilenet_v2(n=1, hw=224, input_dtype="bf16", num_classes=1000):
    """MobileNetV2-1.0: stem 3x3 s2 + ReLU6, 17 inverted residual blocks
    (1x1 expand + ReLU6, depthwise 3x3 + ReLU6, 1x1 linear project, residual
    when the shape is kept), 1x1 -> 1280 + ReLU6, GAP, 1280 -> 1000."""
    g = GraphBuilder("mobilenet_v2", CONFIG_IDS["mobilenet_v2"])
    x = g.input("x", [n, 3, hw, hw], "uniform", dtype=input_dtype)
    y = g.conv(x, 32, 3, stride=2, pad=1, act="relu6", name="stem")
    cin = 32
    bidx = 0
    for t, c, reps, s in _MBV2_SETTINGS:
        for i in range(reps):
            stride = s if i == 0 else 1
            hidden = cin * t
            pre = "ir%d" % bidx
            h = y
            if t != 1:
                h = g.conv(h, hidden, 1, pad=0, act="relu6", name=pre + ".expand")
            h = g.conv(h, hidden, 3, stride=stride, pad=1, groups=hidden, act="relu6",
                       name=pre + ".dw")
            res = y if (stride == 1 and cin == c) else None
            y = g.conv(h, c, 1, pad=0, act=None, residual=res, name=pre + ".project")
            cin = c
            bidx += 1
    y = g.conv(y, 1280, 1, pad=0, act="relu6", name="head")
    y = g.global_avg_pool(y, name="gap")
    y = g.dense(y, num_classes, name="fc")
    g.output(y)
    return g.finish({"batch": n})


def bert_ffn(batch=8, seq=128, hidden=768, ffn=3072, layers=12):
    """BERT-base-shaped FFN stack: x <- x + (GELU(x W1^T + b1) W2^T + b2), 12
    layers, tokens row-major [batch*seq, hidden]; x N(0,1), W and b N(0, 0.02)."""
    g = GraphBuilder("bert_ffn", CONFIG_IDS["bert_ffn"])
    x = g.input("x", [batch * seq, hidden], "normal")
    for layer in range(layers):
        h = g.dense(x, ffn, act="gelu", w_std=0.02, b_std=0.02, name="l%d.ffn1" % layer)
        x = g.dense(h, hidden, residual=x, w_std=0.02, b_std=0.02, name="l%d.ffn2" % layer)
    g.output(x)
    return g.finish({"batch": batch, "seq": seq})


_VGG19 = [64, 64, "M", 128, 128, "M", 256, 256, 256, 256, "M", 512, 512, 512, 512, "M",
          512, 512, 512, 512, "M"]


def vgg19(n=1, hw=224, input_dtype="bf16", num_classes=1000, fc=4096):
    """VGG19-shaped network (one of the fully offloaded rows of the paper's
    Table 1): 16 conv3x3 + ReLU layers in five stages separated by 2x2
    stride-2 max pools, then the classifier.  The first classifier layer
    reads the flattened NCHW feature map, which is exactly a convolution
    whose kernel covers the whole map (no padding) - written that way, its
    [N, 4096, 1, 1] output is flattened by a global average pool over the
    1x1 map; then 4096 -> 4096 + ReLU and 4096 -> classes.  Weights are
    He-normal with the same layer-wide folded normalization as the other
    networks (reading: keeps every activation O(1) with random weights)."""
    g = GraphBuilder("vgg19", CONFIG_IDS["vgg19"])
    x = g.input("x", [n, 3, hw, hw], "uniform", dtype=input_dtype)
    y = x
    for i, v in enumerate(_VGG19):
        if v == "M":
            y = g.max_pool(y, 2, 2, 0, name="pool%d" % i)
        else:
            y = g.conv(y, v, 3, act="relu", name="conv%d" % i)
    s = g.shapes[y][2]
    y = g.conv(y, fc, s, pad=0, act="relu", name="fc6")
    y = g.global_avg_pool(y, name="flatten")
    y = g.dense(y, fc, act="relu", name="fc7")
    y = g.dense(y, num_classes, name="fc8")
    g.output(y)
    return g.finish({"batch": n})


# DarkNet-53 (the YOLOv3 backbone): per stage, output channels and residual blocks
_DARKNET53 = [(64, 1), (128, 2), (256, 8), (512, 8), (1024, 4)]
# folded-BN scale of each residual branch's last conv: the branch adds after
# its leaky ReLU, whose output has a positive mean, so with unit scale the
# stream's mean grows coherently over a stage's blocks (to rms ~20 after 8
# blocks); a small branch scale, as trained residual networks have, keeps it O(1)
_DARKNET_BRANCH_GAMMA = 0.3


def darknet53(n=1, hw=256, input_dtype="bf16", num_classes=1000, alpha=0.1):
    """DarkNet-53-shaped network (a fully offloaded row of the paper's
    Table 1): a 3x3 conv with 32 channels, then five stages, each a 3x3
    stride-2 conv doubling the channels followed by residual blocks of a 1x1
    conv halving them and a 3x3 conv restoring them, every conv with folded
    batch norm and leaky ReLU (slope 0.1); the shortcut adds the block input
    to the block's activated output (a standalone add, after the activation;
    the branch's folded batch norm is scaled by 0.3, see above).
    Global average pool and a dense classifier; 52 convs + 1 dense.  Input
    256x256, the resolution of the published classifier."""
    g = GraphBuilder("darknet53", CONFIG_IDS["darknet53"])
    x = g.input("x", [n, 3, hw, hw], "uniform", dtype=input_dtype)
    y = g.conv(x, 32, 3, act="leaky", alpha=alpha, name="conv0")
    for si, (c, blocks) in enumerate(_DARKNET53):
        y = g.conv(y, c, 3, stride=2, act="leaky", alpha=alpha, name="s%d_down" % si)
        for b in range(blocks):
            h = g.conv(y, c // 2, 1, act="leaky", alpha=alpha, name="s%d_b%d_a" % (si, b))
            h = g.conv(h, c, 3, act="leaky", alpha=alpha, gamma=_DARKNET_BRANCH_GAMMA, name="s%d_b%d_b" % (si, b))
            y = g.add(y, h, name="s%d_b%d_add" % (si, b))
    y = g.global_avg_pool(y, name="pool")
    y = g.dense(y, num_classes, name="fc")
    g.output(y)
    return g.finish({"batch": n})


# mean-square gain of Inception's unpadded 3x3 stride-2 max pools over
# folded-normalized ReLU maps (measured on the float network with these
# weights: 1.5-2.9; the ResNet stem pool's 5.1 would shrink every later layer)
_INCEPTION_MAXPOOL_GAIN = 2.0


def _inception_a(g, x, pool_features, p):
    b1 = g.conv(x, 64, 1, name=p + ".b1")
    b5 = g.conv(g.conv(x, 48, 1, name=p + ".b5a"), 64, 5, name=p + ".b5b")
    b3 = g.conv(g.conv(g.conv(x, 64, 1, name=p + ".b3a"), 96, 3, name=p + ".b3b"), 96, 3, name=p + ".b3c")
    bp = g.conv(g.avg_pool(x, 3, 1, 1, name=p + ".pool"), pool_features, 1, name=p + ".bp")
    return g.concat([b1, b5, b3, bp], name=p)


def _inception_b(g, x, p):
    b3 = g.conv(x, 384, 3, stride=2, pad=0, name=p + ".b3")
    bd = g.conv(g.conv(g.conv(x, 64, 1, name=p + ".bda"), 96, 3, name=p + ".bdb"), 96, 3, stride=2, pad=0,
                name=p + ".bdc")
    bp = g.max_pool(x, 3, 2, 0, name=p + ".pool", gain=_INCEPTION_MAXPOOL_GAIN)
    return g.concat([b3, bd, bp], name=p)


def _inception_c(g, x, c7, p):
    b1 = g.conv(x, 192, 1, name=p + ".b1")
    b7 = g.conv(x, c7, 1, name=p + ".b7a")
    b7 = g.conv(b7, c7, (1, 7), name=p + ".b7b")
    b7 = g.conv(b7, 192, (7, 1), name=p + ".b7c")
    bd = g.conv(x, c7, 1, name=p + ".bda")
    for i, (ks, k) in enumerate([((7, 1), c7), ((1, 7), c7), ((7, 1), c7), ((1, 7), 192)]):
        bd = g.conv(bd, k, ks, name=p + ".bd%d" % i)
    bp = g.conv(g.avg_pool(x, 3, 1, 1, name=p + ".pool"), 192, 1, name=p + ".bp")
    return g.concat([b1, b7, bd, bp], name=p)


def _inception_d(g, x, p):
    b3 = g.conv(g.conv(x, 192, 1, name=p + ".b3a"), 320, 3, stride=2, pad=0, name=p + ".b3b")
    b7 = g.conv(x, 192, 1, name=p + ".b7a")
    b7 = g.conv(b7, 192, (1, 7), name=p + ".b7b")
    b7 = g.conv(b7, 192, (7, 1), name=p + ".b7c")
    b7 = g.conv(b7, 192, 3, stride=2, pad=0, name=p + ".b7d")
    bp = g.max_pool(x, 3, 2, 0, name=p + ".pool", gain=_INCEPTION_MAXPOOL_GAIN)
    return g.concat([b3, b7, bp], name=p)


def _inception_e(g, x, p):
    b1 = g.conv(x, 320, 1, name=p + ".b1")
    b3 = g.conv(x, 384, 1, name=p + ".b3a")
    b3a = g.conv(b3, 384, (1, 3), name=p + ".b3b1")
    b3b = g.conv(b3, 384, (3, 1), name=p + ".b3b2")
    bd = g.conv(g.conv(x, 448, 1, name=p + ".bda"), 384, 3, name=p + ".bdb")
    bda = g.conv(bd, 384, (1, 3), name=p + ".bdc1")
    bdb = g.conv(bd, 384, (3, 1), name=p + ".bdc2")
    bp = g.conv(g.avg_pool(x, 3, 1, 1, name=p + ".pool"), 192, 1, name=p + ".bp")
    # the branches' inner concatenations of the two split convs are part of
    # the block's one concatenation (the same channel order)
    return g.concat([b1, b3a, b3b, bda, bdb, bp], name=p)


def inception_v3(n=1, hw=299, input_dtype="bf16", num_classes=1000):
    """Inception V3-shaped network (a fully offloaded row of the paper's
    Table 1), inference form: the stem of 3x3 convs and max pools, three
    Inception-A blocks (35x35), the grid reduction B, four Inception-C blocks
    with factorized 1x7 / 7x1 convs (17x17), reduction D and two Inception-E
    blocks (8x8), global average pool and a dense classifier.  Every conv has
    folded batch norm and ReLU; the pool branches average 3x3 windows
    (stride 1, padding not counted).  Input 299x299."""
    g = GraphBuilder("inception_v3", CONFIG_IDS["inception_v3"])
    x = g.input("x", [n, 3, hw, hw], "uniform", dtype=input_dtype)
    y = g.conv(x, 32, 3, stride=2, pad=0, name="stem1")
    y = g.conv(y, 32, 3, pad=0, name="stem2")
    y = g.conv(y, 64, 3, name="stem3")
    y = g.max_pool(y, 3, 2, 0, name="stem_pool1", gain=_INCEPTION_MAXPOOL_GAIN)
    y = g.conv(y, 80, 1, name="stem4")
    y = g.conv(y, 192, 3, pad=0, name="stem5")
    y = g.max_pool(y, 3, 2, 0, name="stem_pool2", gain=_INCEPTION_MAXPOOL_GAIN)
    for i, pf in enumerate((32, 64, 64)):
        y = _inception_a(g, y, pf, "mixed5%s" % "bcd"[i])
    y = _inception_b(g, y, "mixed6a")
    for i, c7 in enumerate((128, 160, 160, 192)):
        y = _inception_c(g, y, c7, "mixed6%s" % "bcde"[i])
    y = _inception_d(g, y, "mixed7a")
    y = _inception_e(g, y, "mixed7b")
    y = _inception_e(g, y, "mixed7c")
    y = g.global_avg_pool(y, name="pool")
    y = g.dense(y, num_classes, name="fc")
    g.output(y)
    return g.finish({"batch": n})


def build(name, **kw):
    """Build a workload by name: conv_f32, resnet18_block, resnet50_v1,
    resnet50_v1b, mobilenet_v2, bert_ffn, vgg19, darknet53, inception_v3."""
    if name == "conv_f32":
        return conv_f32(**kw)
    if name == "resnet18_block":
        return resnet18_block(**kw)
    if name == "resnet50_v1":
        return resnet50(variant="v1", **kw)
    if name == "resnet50_v1b":
        return resnet50(variant="v1b", **kw)
    if name == "mobilenet_v2":
        return mobilenet_v2(**kw)
    if name == "bert_ffn":
        return bert_ffn(**kw)
    if name == "vgg19":
        return vgg19(**kw)
    if name == "darknet53":
        return darknet53(**kw)
    if name == "inception_v3":
        return inception_v3(**kw)
    raise ValueError("unknown workload %r" % name)
