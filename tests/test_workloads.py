"""The seeded synthetic workloads: shapes, op counts, determinism, scale."""

import numpy as np
import pytest

import oracle
from paper_2105_03215_amd import workloads


def _count(wl, prefix):
    return sum(1 for n in wl.graph["nodes"] if n["composite"].startswith(prefix))


def test_resnet50_v1_structure_and_work():
    wl = workloads.build("resnet50_v1", n=1)
    convs = [n for n in wl.graph["nodes"] if n["composite"].startswith("conv2d")]
    assert len(convs) == 53
    assert _count(wl, "max_pool2d") == 1 and _count(wl, "global_avg_pool2d") == 1
    assert _count(wl, "dense") == 1
    assert sum(1 for n in convs if "_add" in n["composite"]) == 16
    # 7.716 GFLOP per image for v1 (stride on the 1x1), 8.178 for v1b
    assert abs(2 * wl.macs / 1e9 - 7.716) < 0.01
    wlb = workloads.build("resnet50_v1b", n=1)
    assert abs(2 * wlb.macs / 1e9 - 8.178) < 0.01
    assert wl.graph["outputs"][0]["name"] == "fc"


def test_mobilenet_v2_structure():
    wl = workloads.build("mobilenet_v2", n=1)
    dw = [n for n in wl.graph["nodes"] if n["composite"].startswith("conv2d") and n["attrs"]["groups"] > 1]
    assert len(dw) == 17
    assert _count(wl, "conv2d") - len(dw) == 35
    assert sum(1 for n in wl.graph["nodes"] if "_add" in n["composite"]) == 10
    assert all(n["composite"] == "conv2d_bias_relu6" for n in dw)


def test_bert_ffn_structure():
    wl = workloads.build("bert_ffn")
    assert wl.graph["inputs"][0]["shape"] == [1024, 768]
    assert _count(wl, "dense_bias_gelu") == 12 and _count(wl, "dense_bias_add") == 12
    assert abs(2 * wl.macs / 1024 / 1e6 - 113.2) < 0.1


def test_vgg19_structure_and_work():
    wl = workloads.vgg19(n=1)
    comps = [n["composite"] for n in wl.graph["nodes"]]
    assert comps.count("conv2d_bias_relu") == 17  # 16 conv3x3 + the full-map fc6
    assert comps.count("max_pool2d") == 5
    assert comps[-3:] == ["global_avg_pool2d", "dense_bias_relu", "dense_bias"]
    # 19.63 G multiply-adds per 224x224 image (the usual VGG19 count)
    assert abs(wl.macs / 1e9 - 19.63) < 0.01


def test_full_map_conv_is_flatten_then_dense():
    """The reading behind fc6: a convolution whose kernel covers the whole
    feature map (no padding) equals a dense layer on the NCHW-flattened map."""
    import oracle
    rng = np.random.default_rng(0)
    x = rng.standard_normal((3, 5, 4, 4))
    w = rng.standard_normal((7, 5, 4, 4))
    a = oracle.ops.conv2d(x, w)[:, :, 0, 0]
    b = oracle.ops.dense(x.reshape(3, -1), w.reshape(7, -1))
    assert np.max(np.abs(a - b)) < 1e-12


def test_deterministic_and_distinct_seeds():
    a = workloads.build("resnet18_block")
    b = workloads.build("resnet18_block")
    assert a.json == b.json
    for x, y in zip(a.consts + a.inputs, b.consts + b.inputs):
        assert np.array_equal(x, y)
    assert not np.array_equal(a.consts[0], a.consts[2])


def test_bf16_inputs_are_representable():
    wl = workloads.build("resnet18_block")
    x = wl.inputs[0]
    assert x.dtype == np.float32
    assert np.all((x.view(np.uint32) & 0xFFFF) == 0)
    assert 0.0 <= x.min() and x.max() <= 1.0


@pytest.mark.slow
def test_darknet53_structure_and_work():
    wl = workloads.darknet53(n=1)
    comps = [n["composite"] for n in wl.graph["nodes"]]
    assert comps.count("conv2d_bias_leaky") == 52 and comps.count("add") == 23
    assert comps[-2:] == ["global_avg_pool2d", "dense_bias"]
    assert all(n["attrs"]["alpha"] == 0.1 for n in wl.graph["nodes"] if n["composite"].endswith("_leaky"))
    # 18.6 GFLOP per 256x256 image (the published DarkNet-53 count is 18.7 BFLOP)
    assert abs(2 * wl.macs / 1e9 - 18.57) < 0.01
    # the shortcut adds the block input to the activated branch
    adds = [n for n in wl.graph["nodes"] if n["composite"] == "add"]
    by = {n["name"]: n for n in wl.graph["nodes"]}
    assert all(by[a["inputs"][1]]["composite"] == "conv2d_bias_leaky" for a in adds)


def test_inception_v3_structure_and_work():
    wl = workloads.inception_v3(n=1)
    comps = [n["composite"] for n in wl.graph["nodes"]]
    assert comps.count("conv2d_bias_relu") == 94 and comps.count("concatenate") == 11
    assert comps.count("avg_pool2d") == 9 and comps.count("max_pool2d") == 4
    # block output channels of the published network, from the node list
    wshape = {c["name"]: wl.consts[c["index"]].shape for c in wl.graph["constants"]}
    ch = {"x": 3}
    for n in wl.graph["nodes"]:
        if n["composite"].startswith(("conv2d", "dense")):
            ch[n["name"]] = wshape[n["inputs"][1]][0]
        elif n["composite"] == "concatenate":
            ch[n["name"]] = sum(ch[i] for i in n["inputs"])
        else:
            ch[n["name"]] = ch[n["inputs"][0]]
    assert {k: ch[k] for k in ("mixed5b", "mixed5c", "mixed5d", "mixed6a", "mixed6e", "mixed7a", "mixed7b",
                               "mixed7c")} == {"mixed5b": 256, "mixed5c": 288, "mixed5d": 288, "mixed6a": 768,
                                               "mixed6e": 768, "mixed7a": 1280, "mixed7b": 2048, "mixed7c": 2048}
    # 5.71 G multiply-adds per 299x299 image (the usual Inception V3 count)
    assert abs(wl.macs / 1e9 - 5.713) < 0.01
    rect = [n for n in wl.graph["nodes"] if n["composite"].startswith("conv2d")
            and wl.consts[[c["index"] for c in wl.graph["constants"] if c["name"] == n["inputs"][1]][0]].shape[2:]
            in ((1, 7), (7, 1), (1, 3), (3, 1))]
    assert len(rect) == 4 * 6 + 2 + 2 * 4


@pytest.mark.parametrize("name", ["resnet50_v1", "mobilenet_v2", "resnet18_block", "vgg19", "darknet53",
                                  "inception_v3"])
def test_activations_stay_order_one(name):
    kw = {"vgg19": {"hw": 112}, "darknet53": {"hw": 128}, "inception_v3": {"hw": 139}}.get(name, {})
    wl = workloads.build(name, **kw)
    outs, vals = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="bf16io", keep=True)
    names = [n["name"] for n in wl.graph["nodes"]]
    peak = max(float(np.abs(vals[n]).max()) for n in names)
    rms_out = float(np.sqrt(np.mean(outs[0] ** 2)))
    assert peak < 32, peak
    assert 0.1 < rms_out < 4, rms_out
