"""Every bf16 implicit-GEMM kernel variant at batch-32 ResNet-50 layer shapes.

The engine's autotune picks, per conv launch, the fastest of the variants
whose results are bit-for-bit those of the built-in choice: every tile of the
HBM->LDS pipelined kernel (32x64 ... 256x128 pixels x channels), ring depths
1-4, 4 or 8 waves, the register-staged kernel, and any XCD placement of the
tiles, all within the reduction-order class of the built-in choice (one
reduction group, or two or four groups that split the stages).  The 3x3 halo kernel
(input window staged in LDS) sums in its own order; its weight rings and its
two tiles (128 or 64 pixels x 64 channels) are its variants.  Here each variant is forced through the tile override on three
layers at their batch-32 shapes and checked:

* within one bf16 ulp of the oracle (plus 2^-16 of the summed term
  magnitudes) - the first variant of every class against the oracle, and
* bit for bit equal to the first variant of its class (so every variant the
  autotune can choose is held to the same bar).
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2105_03215_amd import capi, runtime
from paper_2105_03215_amd.workloads import GraphBuilder
from parity_util import announce, term_scale_graph, within_one_ulp

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
LDS_LIMIT = 160 * 1024

# (bm, bn) per workgroup shape: 4 waves, 8 waves, two or four 4-wave reduction groups
TILES_W4 = [(128, 128), (128, 64), (64, 128), (64, 64), (32, 64), (64, 256), (256, 64)]
TILES_W8 = [(128, 128), (128, 64), (64, 128), (128, 256), (256, 128)]
TILES_KG2 = [(128, 128), (128, 64), (64, 128), (64, 64), (32, 64)]
TILES_KG4 = [(64, 64), (32, 64)]


def dma_variants(m_rows):
    """(override string, kgroups) of every pipelined-kernel variant."""
    out = []
    for tiles, threads, kg in ((TILES_W4, 256, 1), (TILES_W8, 512, 1), (TILES_KG2, 512, 2), (TILES_KG4, 1024, 4)):
        for bm, bn in tiles:
            if bm == 32 and m_rows >= 48:
                continue
            for ns in range(1, 5):
                if (bm + bn) * 128 * ns * kg + 64 * 16 > LDS_LIMIT:
                    continue
                out.append(("d%dx%ds%dt%dk%d" % (bm, bn, ns, threads, kg), kg,
                            "conv_dma_%dx%d_s%d_w%d_k%d" % (bm, bn, ns, threads // 64, kg)))
    return out


LAYERS = [
    # name, (n, c, h, w), k, r, act, residual
    ("s3_3x3", (32, 256, 14, 14), 256, 3, "relu", False),
    ("s4_3x3", (32, 512, 7, 7), 512, 3, "relu", False),
    ("s1_1x1_expand_res", (32, 64, 56, 56), 256, 1, "relu", True),
]


def _layer(case):
    name, shape, k, r, act, res = case
    g = GraphBuilder("variants_" + name, 3000 + LAYERS.index(case))
    x = g.input("x", list(shape), "uniform")
    n, c, h, w = shape
    rname = g.input("res", [n, k, h, w], "normal") if res else None
    y = g.conv(x, k, r, stride=1, pad=(r - 1) // 2, act=act, residual=rname, name="y")
    g.output(y)
    return g.finish()


def _run_forced(wl, env, monkeypatch):
    monkeypatch.delenv("BYOC_CONV_TILE", raising=False)
    monkeypatch.delenv("BYOC_CONV_XCD", raising=False)
    monkeypatch.delenv("BYOC_CONV_HALO", raising=False)
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    sg = capi.Subgraph(wl.graph, wl.consts, device=0)
    try:
        ins = runtime.inputs_for(sg, wl.inputs, DEV)
        outs = runtime.outputs_for(sg, DEV)
        outs[0].fill_(float("nan"))
        sg.run(ins, outs)
        torch.cuda.synchronize()
        names = [l["name"] for l in sg.launches() if l["kind"] in ("conv_mfma", "reduce")]
        return outs[0], names
    finally:
        sg.close()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("case", LAYERS, ids=[c[0] for c in LAYERS])
def test_every_variant(case, monkeypatch):
    name, shape, k, r, act, res = case
    wl = _layer(case)
    n, c, h, w = shape
    m_rows = n * h * w
    ref = oracle.run_graph(wl.graph, wl.consts, wl.inputs, mode="bf16io")[0]
    scale = term_scale_graph(wl.graph, wl.consts, wl.inputs)[0]

    firsts = {}
    checked = 0

    def check(label, env, cls, expect_name):
        nonlocal checked
        announce("variant %s %s" % (name, label))
        out, names = _run_forced(wl, env, monkeypatch)
        assert len(names) == 1 and names[0].startswith(expect_name), (label, names)
        if cls not in firsts:
            g = runtime.to_host_f64(out)
            ok = within_one_ulp(g, ref, scale)
            assert ok.all(), "%s %s: %d elements beyond one ulp" % (name, label, int((~ok).sum()))
            firsts[cls] = out
        else:
            assert torch.equal(out.view(torch.int16), firsts[cls].view(torch.int16)), (name, label)
        checked += 1

    for ov, kg, expect in dma_variants(m_rows):
        check(ov, {"BYOC_CONV_TILE": ov}, "kg%d" % kg, expect)
    # the register-staged kernel (one reduction group)
    check("regs 64x64", {"BYOC_CONV_TILE": "64x64x16"}, "kg1", "conv_mfma_64x64_mf16")
    # every XCD placement of one tile
    for py in (0, 1, 2, 4, 8):
        check("xcd %d" % py, {"BYOC_CONV_TILE": "d128x64s2t512k1", "BYOC_CONV_XCD": str(py)}, "kg1",
              "conv_dma_128x64_s2_w8_k1")
    # 3x3 layers: the halo kernel's weight rings (its own reduction order)
    if r == 3 and c % 64 == 0:
        for ring in (2, 3, 4, 6, 8):
            check("halo ring %d" % ring, {"BYOC_CONV_TILE": "h128x64s%d" % ring}, "halo",
                  "conv_halo_128x64_s%d" % ring)
        for ring in (2, 3):
            check("halo 64x64 ring %d" % ring, {"BYOC_CONV_TILE": "h64x64s%d" % ring}, "halo",
                  "conv_halo_64x64_s%d" % ring)
    print("%s: %d variants checked, classes %s" % (name, checked, sorted(firsts)), flush=True)
