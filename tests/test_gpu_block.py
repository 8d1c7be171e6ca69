"""Fused bottleneck blocks: 1x1 reduce -> 3x3 -> 1x1 expand + the block
input (or + a 1x1 projection of it), planned as one launch whose
intermediates never leave LDS.

Checked on ResNet-50 stage shapes and on ragged ones (image sizes that are
not multiples of the kernel's output tile), two blocks chained (a projection
block, stride 1 or 2, is followed by an identity one):

* the fused run equals, bit for bit, the three unfused launches on the
  single-reduction-group implicit-GEMM kernel without split-K (the same
  summation order and the same bf16 rounding of each composite's output);
* every tile variant of the fused kernel gives the same bits, also when the
  autotune picks among them under graph replay;
* one block's output is within the bf16 tolerance of the oracle (bf16io).
  (Two chained blocks on these inputs sit at the tolerance itself - 1.003e-2
  on the 56x56 case, for the fused and the unfused launches alike - from the
  bf16 storage of four composites in a row; the bit equality above carries
  the per-composite one-ulp checks of the unfused kernels over to them.)

The int8 form of the same blocks (scales and zero points calibrated on the
oracle's values of one image; the intermediates' zero point after the ReLU is
-128, so the 3x3's padding is a nonzero code) must equal both the unfused
int8 launches and the int8 oracle bit for bit, with every tile variant.
"""


import numpy as np
import pytest
import torch

import oracle
from oracle import quant as OQ
from paper_2105_03215_amd import capi, runtime
from paper_2105_03215_amd.workloads import GraphBuilder
from parity_util import BF16_TOL, announce, oracle_calibrated_int8, rel_err

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
ENV = ("BYOC_FUSE_BLOCK", "BYOC_CONV_TILE", "BYOC_CONV_SPLIT", "BYOC_BLOCK_VARIANT", "BYOC_CONV_HALO")
# these blocks are small: fuse them whatever their tile count
FUSED = {"BYOC_FUSE_BLOCK": "1"}
# the unfused reference: every conv on one tile of the single-group kernel, no split-K
UNFUSED_KG1 = {"BYOC_FUSE_BLOCK": "0", "BYOC_CONV_TILE": "d64x64s2t256k1", "BYOC_CONV_SPLIT": "1"}

CASES = [
    # name, batch, input channels, mid channels, output channels, height, width (of the input), stride
    ("s1_56x56", 2, 256, 64, 256, 56, 56, 1),
    ("s1_ragged_30x19", 1, 256, 64, 256, 30, 19, 1),
    ("s2_28x28", 2, 512, 128, 512, 28, 28, 1),
    ("s2_ragged_13x9", 3, 512, 128, 512, 13, 9, 1),
    ("proj_56x56", 2, 64, 64, 256, 56, 56, 1),
    ("proj_ragged_30x19", 1, 64, 64, 256, 30, 19, 1),
    ("proj_s2_56x56", 2, 256, 128, 512, 56, 56, 2),
    ("proj_s2_ragged_27x19", 1, 256, 128, 512, 27, 19, 2),
]


def _blocks(case, n_blocks=2):
    name, n, cin, mid, cout, h, w, stride = case
    g = GraphBuilder("block_" + name, 3100 + (CASES.index(case) if case in CASES else 9))
    y = g.input("x", [n, cin, h, w], "uniform")
    for i in range(n_blocks):
        r = y
        st = stride if i == 0 else 1
        if g.shapes[y][1] != cout or st != 1:  # the projection shortcut
            r = g.conv(y, cout, 1, stride=st, pad=0, act=None, name="b%d.p" % i)
        a = g.conv(y, mid, 1, stride=st, pad=0, act="relu", name="b%d.a" % i)
        b = g.conv(a, mid, 3, pad=1, act="relu", name="b%d.b" % i)
        y = g.conv(b, cout, 1, pad=0, act="relu", residual=r, name="b%d.c" % i)
    g.output(y)
    return g.finish()


def _run(wl, monkeypatch, env, options=None, graph=None):
    for k in ENV:
        monkeypatch.delenv(k, raising=False)
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    sg = capi.Subgraph(graph if graph is not None else wl.graph, wl.consts, device=0)
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


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_fused_block_matches_unfused_and_oracle(case, monkeypatch):
    announce("fused block " + case[0])
    wl = _blocks(case)
    fused, names = _run(wl, monkeypatch, FUSED)
    assert sum(nm.startswith("bottleneck_") for nm in names) == 2, names
    assert not any(nm.startswith("conv_") for nm in names), names
    plain, pnames = _run(wl, monkeypatch, UNFUSED_KG1)
    assert not any(nm.startswith("bottleneck_") for nm in pnames), pnames
    assert torch.equal(fused.view(torch.int16), plain.view(torch.int16))
    wl = _blocks(case, n_blocks=1)
    fused, _ = _run(wl, monkeypatch, FUSED)
    ref = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="bf16io")[0]
    err = rel_err(runtime.to_host_f64(fused), ref)
    print("%s: max rel err %.3e" % (case[0], err), flush=True)
    assert err <= BF16_TOL


VARIANT_CASES = [CASES[0], CASES[2], CASES[4], CASES[6]]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_every_block_variant_and_autotune_bitwise(case, monkeypatch):
    announce("block variants " + case[0])
    wl = _blocks(case)
    ref, names0 = _run(wl, monkeypatch, dict(FUSED, BYOC_BLOCK_VARIANT="0"))
    seen = {tuple(n for n in names0 if n.startswith("bottleneck_"))}
    for v in (1, 2, 3):  # 3: the small-batch tile (4 x 7 pixels, 4 waves)
        out, names = _run(wl, monkeypatch, dict(FUSED, BYOC_BLOCK_VARIANT=str(v)))
        seen.add(tuple(n for n in names if n.startswith("bottleneck_")))
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), v
    assert len(seen) == 4, seen  # the variants are distinct kernels
    out, _ = _run(wl, monkeypatch, FUSED, options={"autotune": True, "graph_replay": True})
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))


def test_block_fusion_rule(monkeypatch):
    """Three launches where fusion is off (BYOC_FUSE_BLOCK=0) and for a width
    pair without a fused kernel; one launch by default for a supported bf16
    block at any batch (batch 1 at 28x28: 28 tiles of 4 x 7 pixels)."""
    announce("block fusion rule")
    wl = _blocks(("odd", 1, 192, 48, 192, 14, 14, 1), n_blocks=1)
    _, names = _run(wl, monkeypatch, FUSED)
    assert not any(n.startswith("bottleneck_") for n in names), names
    wl = _blocks(CASES[0], n_blocks=1)
    _, names = _run(wl, monkeypatch, {"BYOC_FUSE_BLOCK": "0"})
    assert not any(n.startswith("bottleneck_") for n in names), names
    _, names = _run(wl, monkeypatch, {})
    assert sum(n.startswith("bottleneck_") for n in names) == 1, names
    wl = _blocks(("s2_bs1", 1, 512, 128, 512, 28, 28, 1), n_blocks=1)
    _, names = _run(wl, monkeypatch, {})
    assert sum(n.startswith("bottleneck_") for n in names) == 1, names


def test_resnet50_fused_equals_unfused_bitwise(monkeypatch):
    """The whole ResNet-50 v1 graph with every supported block fused
    (batch 4, fusion forced) equals the unfused plan bit for bit, both with
    every other conv on the same single-group tile without split-K."""
    announce("resnet50_v1 bs4: fused blocks vs unfused, bitwise")
    from paper_2105_03215_amd import workloads
    wl = workloads.build("resnet50_v1", n=4)
    fused, names = _run(wl, monkeypatch, dict(UNFUSED_KG1, BYOC_FUSE_BLOCK="1"))
    assert sum(n.startswith("bottleneck_") for n in names) == 7, names  # stages 1 and 2
    plain, pnames = _run(wl, monkeypatch, UNFUSED_KG1)
    assert not any(n.startswith("bottleneck_") for n in pnames)
    assert torch.equal(fused.view(torch.int16) if fused.dtype == torch.bfloat16 else fused,
                       plain.view(torch.int16) if plain.dtype == torch.bfloat16 else plain)


def _int8(wl):
    return oracle_calibrated_int8(wl.graph, wl.consts, [np.ascontiguousarray(a[:1]) for a in wl.inputs])


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_int8_fused_block_exact(case, monkeypatch):
    """int8: fused == unfused == the int8 oracle, bit for bit (two chained blocks)."""
    announce("int8 fused block " + case[0])
    wl = _blocks(case)
    qg = _int8(wl)
    fused, names = _run(wl, monkeypatch, FUSED, graph=qg)
    assert sum(nm.startswith("bottleneck_i8_") for nm in names) == 2, names
    assert not any(nm.startswith("conv_i8") for nm in names), names
    plain, pnames = _run(wl, monkeypatch, {"BYOC_FUSE_BLOCK": "0"}, graph=qg)
    assert not any(nm.startswith("bottleneck_") for nm in pnames), pnames
    assert torch.equal(fused, plain)
    ref = OQ.run_quantized_graph(qg, wl.consts, wl.inputs)[0]
    assert np.array_equal(runtime.to_host_f64(fused), ref.astype(np.float64))


@pytest.mark.parametrize("case", VARIANT_CASES, ids=[c[0] for c in VARIANT_CASES])
def test_int8_every_block_variant_and_autotune(case, monkeypatch):
    announce("int8 block variants " + case[0])
    wl = _blocks(case)
    qg = _int8(wl)
    ref, names0 = _run(wl, monkeypatch, dict(FUSED, BYOC_BLOCK_VARIANT="0"), graph=qg)
    seen = {tuple(n for n in names0 if n.startswith("bottleneck_i8_"))}
    for v in (1, 2):
        out, names = _run(wl, monkeypatch, dict(FUSED, BYOC_BLOCK_VARIANT=str(v)), graph=qg)
        seen.add(tuple(n for n in names if n.startswith("bottleneck_i8_")))
        assert torch.equal(out, ref), v
    assert len(seen) == 3, seen
    out, _ = _run(wl, monkeypatch, FUSED, options={"autotune": True, "graph_replay": True}, graph=qg)
    assert torch.equal(out, ref)
