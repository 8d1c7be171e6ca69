"""AddressSanitizer / UndefinedBehaviorSanitizer build of the library's host
side - the JSON reader, the schema checks and the launch planner - driven on
the CPU over every workload of this repository (bf16, fp32 and int8 forms)
and over a few hundred malformed variants of serialized subgraphs.

The host sources (json.cpp, graph.cpp, capi.cpp, engine.cpp) are compiled
with g++ and the sanitizers; the HIP kernel objects of the regular build are
linked in uninstrumented (their host launchers are never reached here).
byoc_subgraph_create plans the launch sequence before it looks for a device,
so on this GPU-less host every valid case runs the whole planner and then
returns BYOC_ERR_DEVICE.  Any sanitizer report, crash or leak fails the
test."""

import copy
import hashlib
import json
import os
import random
import shutil
import subprocess

import pytest

from paper_2105_03215_amd import build as B
from paper_2105_03215_amd import quantize, workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DRIVER = os.path.join(ROOT, "tests", "sanitize", "byoc_plan_driver.cpp")
HOST_SOURCES = ["json.cpp", "graph.cpp", "capi.cpp", "engine.cpp"]
CXXFLAGS = ["-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
            "-fno-sanitize-recover=undefined", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
            "-I" + os.path.join(ROOT, "include")]

pytestmark = [pytest.mark.slow,
              pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="host-only sanitizer run (a GPU is visible)"),
              pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")]

ST_OK, ST_DEVICE, ST_INTERNAL = 0, 5, 7


def _hip_objects():
    objs = [os.path.join(B.OBJ, os.path.splitext(s)[0] + ".o") for s in B.SOURCES if s.endswith(".hip")]
    missing = [o for o in objs if not os.path.exists(o)]
    if missing:
        pytest.skip("HIP objects not built (run the package build first): %s" % missing[0])
    return objs


def _build_driver():
    h = hashlib.sha256()
    for name in sorted(os.listdir(B.CSRC)):
        if name.endswith((".cpp", ".h")):
            with open(os.path.join(B.CSRC, name), "rb") as f:
                h.update(name.encode() + f.read())
    for p in (DRIVER, os.path.join(ROOT, "include", "byoc.h")):
        with open(p, "rb") as f:
            h.update(f.read())
    h.update(" ".join(CXXFLAGS).encode())
    out_dir = os.path.join("/tmp", "byoc_sanitize_" + h.hexdigest()[:16])
    os.makedirs(out_dir, exist_ok=True)
    objs = []
    procs = []
    for src in HOST_SOURCES + [DRIVER]:
        path = src if os.path.isabs(src) else os.path.join(B.CSRC, src)
        obj = os.path.join(out_dir, os.path.splitext(os.path.basename(path))[0] + ".o")
        objs.append(obj)
        if not os.path.exists(obj):
            procs.append((path, subprocess.Popen(["g++"] + CXXFLAGS + ["-c", path, "-o", obj + ".tmp"],
                                                 stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
    for path, p in procs:
        out, _ = p.communicate()
        assert p.returncode == 0, "g++ failed on %s:\n%s" % (path, out)
    for obj in objs:
        if os.path.exists(obj + ".tmp"):
            os.replace(obj + ".tmp", obj)
    exe = os.path.join(out_dir, "byoc_plan_driver")
    r = subprocess.run(["g++", "-fsanitize=address,undefined", "-static-libasan", "-o", exe] + objs +
                       _hip_objects() + ["-L/opt/rocm/lib", "-Wl,-rpath,/opt/rocm/lib", "-lamdhip64"],
                       capture_output=True, text=True)
    assert r.returncode == 0, "link failed:\n" + r.stdout + r.stderr
    return exe, out_dir


def _const_lines(wl):
    by_index = sorted(wl.graph["constants"], key=lambda c: c["index"])
    lines = []
    for c in by_index:
        a = wl.consts[c["index"]]
        lines.append(" ".join(["0", str(a.ndim)] + [str(d) for d in a.shape]))
    return "\n".join(lines) + "\n"


def _int8(wl):
    ranges = {d["name"]: (-1.0, 2.0) for d in wl.graph["inputs"]}
    for k, n in enumerate(wl.graph["nodes"]):
        ranges[n["name"]] = (-0.5 - 0.01 * k, 3.0 + 0.02 * k)
    return quantize.quantize_graph(wl.graph, ranges)


def _valid_cases():
    cases = [
        ("conv_f32", workloads.build("conv_f32")),
        ("resnet18_block", workloads.build("resnet18_block")),
        ("resnet50_v1_bs1", workloads.build("resnet50_v1", n=1)),
        ("resnet50_v1_bs32", workloads.build("resnet50_v1", n=32)),
        ("resnet50_v1b_bs2", workloads.build("resnet50_v1b", n=2)),
        ("resnet50_f32_input", workloads.resnet50(n=2, input_dtype="f32")),
        ("mobilenet_v2_bs16", workloads.build("mobilenet_v2", n=16)),
        ("bert_ffn", workloads.build("bert_ffn")),
        ("vgg19_64", workloads.build("vgg19", n=2, hw=64)),
        ("darknet53_128", workloads.build("darknet53", n=1, hw=128)),
        ("inception_v3", workloads.build("inception_v3", n=1)),
    ]
    out = []
    for name, wl in cases:
        out.append((name, wl.graph, _const_lines(wl)))
    for name, wl in (("resnet50_v1_int8", workloads.build("resnet50_v1", n=2, hw=96)),
                     ("mobilenet_v2_int8", workloads.build("mobilenet_v2", n=1, hw=64)),
                     ("darknet53_int8", workloads.build("darknet53", n=1, hw=64)),
                     ("vgg19_int8", workloads.build("vgg19", n=1, hw=64))):
        out.append((name, _int8(wl), _const_lines(wl)))
    return out


def _mutants(base, consts, rng, count):
    """Malformed variants of a serialized subgraph: truncations, byte flips,
    dropped or retyped fields, out-of-range numbers."""
    text = json.dumps(base)
    out = []
    for i in range(count):
        kind = i % 6
        if kind == 0:
            out.append(text[:rng.randrange(len(text))])
        elif kind == 1:
            b = bytearray(text.encode())
            for _ in range(rng.randint(1, 4)):
                b[rng.randrange(len(b))] = rng.choice(b'{}[]":,0123456789-eE.tfn \x00\xff')
            out.append(bytes(b).decode("latin-1"))
        else:
            g = copy.deepcopy(base)
            node = rng.choice(g["nodes"])
            if kind == 2:
                node.pop(rng.choice(sorted(node)), None)
            elif kind == 3:
                attrs = node.setdefault("attrs", {})
                key = rng.choice(["strides", "padding", "groups", "dilation", "pool_size", "alpha"])
                attrs[key] = rng.choice([[0, 0], [-1, 2], [1 << 31, 1], [1, 1, 1], "x", None, 1e30, -3, [],
                                         [2 ** 40, 2 ** 40, 0, 0]])
            elif kind == 4:
                d = rng.choice(g["inputs"] + g["constants"])
                d["shape"] = rng.choice([[], [0], [-4, 3], [1 << 31, 2, 2, 2], [1, 2, 3, 4, 5, 6, 7, 8, 9],
                                         [2 ** 20, 2 ** 20, 2 ** 20, 1]])
            else:
                node["inputs"] = rng.choice([[], ["nope"], node["inputs"][:1], node["inputs"] * 2,
                                             [node["name"]]])
            out.append(json.dumps(g))
    return [(m, consts) for m in out]


def test_host_side_under_asan_ubsan(tmp_path):
    exe, _ = _build_driver()
    valid = _valid_cases()
    rng = random.Random(20250)
    cases = []
    for name, graph, consts in valid:
        cases.append((name, json.dumps(graph), consts, True))
    base_names = {"resnet18_block", "resnet50_v1_int8", "inception_v3", "bert_ffn"}
    for name, graph, consts in valid:
        if name in base_names:
            for k, (m, c) in enumerate(_mutants(graph, consts, rng, 60)):
                cases.append(("%s_mut%d" % (name, k), m, c, False))
    lst = []
    for name, text, consts, _ in cases:
        jp = tmp_path / (name + ".json")
        cp = tmp_path / (name + ".consts")
        jp.write_bytes(text.encode("latin-1", "replace") if isinstance(text, str) else text)
        cp.write_text(consts)
        lst.append("%s %s" % (jp, cp))
    (tmp_path / "list.txt").write_text("\n".join(lst) + "\n")
    supp = tmp_path / "lsan.supp"
    supp.write_text("leak:libamdhip64\nleak:libhsa-runtime64\nleak:librocprofiler\nleak:libdrm\n")
    env = dict(os.environ,
               ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               LSAN_OPTIONS="suppressions=%s" % supp)
    r = subprocess.run([exe, str(tmp_path / "list.txt")], capture_output=True, text=True, env=env, timeout=900)
    report = r.stdout[-4000:] + r.stderr[-8000:]
    assert r.returncode == 0, report
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, report
    lines = [ln for ln in r.stdout.splitlines() if " validate=" in ln]
    assert len(lines) == len(cases)
    status = {}
    for ln in lines:
        path = ln.split(" ", 1)[0]
        v = int(ln.split("validate=")[1].split()[0])
        c = int(ln.split("create=")[1].split()[0])
        status[os.path.splitext(os.path.basename(path))[0]] = (v, c, ln)
    for name, _, _, ok in cases:
        v, c, ln = status[name]
        assert c != ST_INTERNAL, ln
        if ok:
            # valid: accepted by the parser, planned, then no device here
            assert v == ST_OK and c == ST_DEVICE and "no HIP device" in ln, ln
        elif v != ST_OK:
            assert c == v, ln  # create reports the parser's error first
