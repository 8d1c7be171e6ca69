"""Fused MobileNetV2 inverted-residual blocks: [1x1 expand + ReLU6 ->]
depthwise 3x3 + ReLU6 -> 1x1 project [+ the block input], planned as one
launch whose expanded and depthwise tensors never leave LDS.

Checked on every compiled kind (expansion 1; stride 1 and 2; 16 to 96
output channels) at MobileNetV2's own and at ragged image sizes:

* the fused run equals, bit for bit, the separate launches with every conv
  on the single-reduction-group implicit-GEMM kernel without split-K (the
  same summation order and the same bf16 rounding of each composite);
* one block is within the bf16 tolerance of the oracle (bf16io);
* the whole MobileNetV2 with its early blocks fused equals the unfused plan
  bit for bit, and the fusion rule picks the blocks with enough tiles.
"""

import pytest
import torch

import oracle
from paper_2105_03215_amd import capi, runtime
from paper_2105_03215_amd.workloads import GraphBuilder
from parity_util import BF16_TOL, announce, rel_err

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
ENV = ("BYOC_FUSE_IR", "BYOC_FUSE_BLOCK", "BYOC_CONV_TILE", "BYOC_CONV_SPLIT", "BYOC_CONV_HALO", "BYOC_IR_VARIANT")
FUSED = {"BYOC_FUSE_IR": "1"}
UNFUSED_KG1 = {"BYOC_FUSE_IR": "0", "BYOC_CONV_TILE": "d64x64s2t256k1", "BYOC_CONV_SPLIT": "1"}

CASES = [
    # name, batch, input channels, expansion, output channels, height, width (of the input), stride
    ("noexp_32_16_ragged_20x37", 2, 32, 1, 16, 20, 37, 1),
    ("s2_16_96_24_ragged_31x26", 2, 16, 6, 24, 31, 26, 2),
    ("s1_24_144_24_28x28", 2, 24, 6, 24, 28, 28, 1),
    ("s2_24_144_32_ragged_19x22", 1, 24, 6, 32, 19, 22, 2),
    ("s1_32_192_32_ragged_13x29", 2, 32, 6, 32, 13, 29, 1),
    ("s2_32_192_64_28x28", 2, 32, 6, 64, 28, 28, 2),
    ("s1_64_384_64_14x14", 3, 64, 6, 64, 14, 14, 1),
    ("s1_64_384_96_ragged_9x11", 2, 64, 6, 96, 9, 11, 1),
    # the later blocks: the window two or three slices deep, expanded width up to 960
    ("s1_96_576_96_14x14", 2, 96, 6, 96, 14, 14, 1),
    ("s2_96_576_160_ragged_13x11", 1, 96, 6, 160, 13, 11, 2),
    ("s1_160_960_160_7x7", 3, 160, 6, 160, 7, 7, 1),
    ("s1_160_960_320_ragged_9x6", 2, 160, 6, 320, 9, 6, 1),
]


def _blocks(case, n_blocks=2):
    """The block, then (when its output keeps a supported shape) one more
    with the residual, as MobileNetV2 chains them."""
    name, n, cin, t, cout, h, w, stride = case
    g = GraphBuilder("ir_" + name, 3300 + (CASES.index(case) if case in CASES else 9))
    y = g.input("x", [n, cin, h, w], "uniform")
    c_in = cin
    for i in range(n_blocks):
        st = stride if i == 0 else 1
        te = t if i == 0 else 6
        hidden = c_in * te
        hh = y
        if te != 1:
            hh = g.conv(hh, hidden, 1, pad=0, act="relu6", name="b%d.expand" % i)
        hh = g.conv(hh, hidden, 3, stride=st, pad=1, groups=hidden, act="relu6", name="b%d.dw" % i)
        res = y if (st == 1 and c_in == cout) else None
        y = g.conv(hh, cout, 1, pad=0, act=None, residual=res, name="b%d.project" % i)
        c_in = cout
        if cout > 160:  # the next block's input would not fit the fused kernel's window
            break
    g.output(y)
    return g.finish()


def _run(wl, monkeypatch, env, options=None):
    for k in ENV:
        monkeypatch.delenv(k, raising=False)
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    sg = capi.Subgraph(wl.graph, wl.consts, device=0)
    s = torch.cuda.Stream(device=DEV)
    try:
        if options:
            sg.set_options(**options)
        ins = runtime.inputs_for(sg, wl.inputs, DEV)
        outs = runtime.outputs_for(sg, DEV)
        outs[0].fill_(float("nan"))
        torch.cuda.synchronize()
        for _ in range(2 if options else 1):
            sg.run(ins, outs, s)
        s.synchronize()
        return outs[0].clone(), [l["name"] for l in sg.launches()]
    finally:
        sg.close()


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_fused_ir_block_matches_unfused_and_oracle(case, monkeypatch):
    announce("fused inverted-residual block " + case[0])
    wl = _blocks(case)
    fused, names = _run(wl, monkeypatch, FUSED)
    assert sum(nm.startswith("ir_block_") for nm in names) >= 1, names
    plain, pnames = _run(wl, monkeypatch, UNFUSED_KG1)
    assert not any(nm.startswith("ir_block_") for nm in pnames), pnames
    assert torch.equal(_bits(fused), _bits(plain))
    wl = _blocks(case, n_blocks=1)
    fused, names = _run(wl, monkeypatch, FUSED)
    assert sum(nm.startswith("ir_block_") for nm in names) == 1, names
    assert not any(nm.startswith(("depthwise", "conv_")) for nm in names), names
    ref = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="bf16io")[0]
    err = rel_err(runtime.to_host_f64(fused), ref)
    print("%s: max rel err %.3e" % (case[0], err), flush=True)
    assert err <= BF16_TOL


VARIANT_CASES = [CASES[0], CASES[1], CASES[2], CASES[5], CASES[6], CASES[7], CASES[8], CASES[9], CASES[10],
                 CASES[11]]


@pytest.mark.parametrize("case", VARIANT_CASES, ids=[c[0] for c in VARIANT_CASES])
def test_every_ir_variant_and_autotune_bitwise(case, monkeypatch):
    """Every tile variant of a kind gives the same bits, also when the
    autotune picks among them under graph replay."""
    announce("inverted-residual variants " + case[0])
    wl = _blocks(case, n_blocks=1)
    ref, names0 = _run(wl, monkeypatch, dict(FUSED, BYOC_IR_VARIANT="0"))
    seen = {tuple(n for n in names0 if n.startswith("ir_block_"))}
    for v in (1, 2):
        out, names = _run(wl, monkeypatch, dict(FUSED, BYOC_IR_VARIANT=str(v)))
        seen.add(tuple(n for n in names if n.startswith("ir_block_")))
        assert torch.equal(_bits(out), _bits(ref)), v
    assert len(seen) == 3, seen
    out, _ = _run(wl, monkeypatch, FUSED, options={"autotune": True, "graph_replay": True})
    assert torch.equal(_bits(out), _bits(ref))


def test_mobilenet_v2_fused_equals_unfused_bitwise(monkeypatch):
    """MobileNetV2 (batch 2, 160x160) with every supported block fused
    equals the unfused plan bit for bit, both with every other conv on the
    same single-group tile without split-K."""
    announce("mobilenet_v2 bs2 160: fused inverted-residual blocks vs unfused, bitwise")
    from paper_2105_03215_amd import workloads
    wl = workloads.build("mobilenet_v2", n=2, hw=160)
    fused, names = _run(wl, monkeypatch, dict(UNFUSED_KG1, BYOC_FUSE_IR="1"))
    n_ir = sum(n.startswith("ir_block_") for n in names)
    assert n_ir == 17, names  # every block
    plain, pnames = _run(wl, monkeypatch, UNFUSED_KG1)
    assert not any(n.startswith("ir_block_") for n in pnames)
    assert torch.equal(_bits(fused), _bits(plain))


def test_ir_fusion_rule(monkeypatch):
    """By default every supported block with at most 64 input channels
    fuses, at any batch: MobileNetV2 at batch 16 and at batch 1 fuses its
    eleven blocks up to 64 -> 96 channels; BYOC_FUSE_IR=1 fuses all 17
    (the wider ones too), BYOC_FUSE_IR=0 none."""
    announce("inverted-residual fusion rule")
    from paper_2105_03215_amd import workloads
    wl = workloads.build("mobilenet_v2", n=16)
    _, names = _run(wl, monkeypatch, {})
    assert sum(n.startswith("ir_block_") for n in names) == 11, names
    _, names = _run(wl, monkeypatch, {"BYOC_FUSE_IR": "1"})
    assert sum(n.startswith("ir_block_") for n in names) == 17, names
    _, names = _run(wl, monkeypatch, {"BYOC_FUSE_IR": "0"})
    assert not any(n.startswith("ir_block_") for n in names)
    wl = workloads.build("mobilenet_v2", n=1)
    _, names = _run(wl, monkeypatch, {})
    assert sum(n.startswith("ir_block_") for n in names) == 11, names
