"""ctypes binding of include/byoc.h (argument marshalling only).

Every computation runs in the HIP library; PyTorch supplies device memory
and streams.  Loading fails loudly when the built library is missing.
"""

import ctypes
import json as _json
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libbyoc.so")

BYOC_OK = 0
F32, BF16 = 0, 1
NCHW, NHWC, ROWMAJOR = 0, 1, 2
KIND_NAMES = ["conv_mfma", "conv_f32", "depthwise", "maxpool", "avgpool", "add", "transform",
              "reduce", "conv_i8"]
STATUS_NAMES = ["OK", "INVALID_ARG", "PARSE", "UNSUPPORTED", "SHAPE", "DEVICE", "OOM", "INTERNAL"]

# Every entry point declared in include/byoc.h.
EXPORTS = ["byoc_subgraph_validate", "byoc_subgraph_create", "byoc_subgraph_run",
           "byoc_subgraph_destroy", "byoc_subgraph_num_io", "byoc_subgraph_io_desc",
           "byoc_subgraph_stats", "byoc_subgraph_num_launches", "byoc_subgraph_launch_info",
           "byoc_subgraph_profile_begin", "byoc_subgraph_profile_end",
           "byoc_subgraph_set_options", "byoc_subgraph_run_static", "byoc_last_error"]
OPT_GRAPH_REPLAY = 1
OPT_AUTOTUNE = 2


class ByocConst(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.POINTER(ctypes.c_int64))]


class TensorDesc(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("layout", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("shape", ctypes.c_int64 * 8)]


class LaunchInfo(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("node", ctypes.c_int32), ("flops", ctypes.c_int64),
                ("bytes", ctypes.c_int64), ("name", ctypes.c_char * 64)]


class ByocError(RuntimeError):
    def __init__(self, status, message):
        self.status = status
        self.status_name = STATUS_NAMES[status] if 0 <= status < len(STATUS_NAMES) else str(status)
        super().__init__("byoc %s: %s" % (self.status_name, message))


_lib = None


def load_library(path=LIB_PATH):
    """Load libbyoc.so once; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("HIP library %s is missing: build it with "
                           "`python -m paper_2105_03215_amd.build`" % path)
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32, i64, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    sig = {
        "byoc_subgraph_validate": [ctypes.c_char_p, sz, ctypes.POINTER(ByocConst), i32],
        "byoc_subgraph_create": [ctypes.c_char_p, sz, ctypes.POINTER(ByocConst), i32, i32,
                                 ctypes.POINTER(P)],
        "byoc_subgraph_run": [P, ctypes.POINTER(P), i32, ctypes.POINTER(P), i32, P],
        "byoc_subgraph_run_static": [P, ctypes.POINTER(P), i32, ctypes.POINTER(P), i32, P],
        "byoc_subgraph_destroy": [P],
        "byoc_subgraph_num_io": [P, ctypes.POINTER(i32), ctypes.POINTER(i32)],
        "byoc_subgraph_io_desc": [P, i32, i32, ctypes.POINTER(TensorDesc)],
        "byoc_subgraph_stats": [P, ctypes.POINTER(i64), ctypes.POINTER(i64), ctypes.POINTER(i64)],
        "byoc_subgraph_num_launches": [P, ctypes.POINTER(i32)],
        "byoc_subgraph_launch_info": [P, i32, ctypes.POINTER(LaunchInfo)],
        "byoc_subgraph_profile_begin": [P, i32],
        "byoc_subgraph_set_options": [P, i32],
        "byoc_subgraph_profile_end": [P, ctypes.POINTER(ctypes.c_float), i32, ctypes.POINTER(i32)],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.byoc_last_error.argtypes = []
    lib.byoc_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status):
    if status != BYOC_OK:
        msg = load_library().byoc_last_error().decode("utf-8", "replace")
        raise ByocError(status, msg)


def _json_bytes(graph):
    if isinstance(graph, (bytes, bytearray)):
        return bytes(graph)
    if isinstance(graph, str):
        return graph.encode("utf-8")
    return _json.dumps(graph).encode("utf-8")


class _Consts:
    """Host constant arrays marshalled into a byoc_const array (kept alive)."""

    def __init__(self, consts):
        self.arrays = []
        self.shapes = []
        n = len(consts)
        self.c = (ByocConst * max(n, 1))()
        for i, a in enumerate(consts):
            if hasattr(a, "detach"):  # torch tensor on the host
                import torch
                if a.dtype == torch.bfloat16:
                    a = a.contiguous().view(torch.int16).numpy().view(np.uint16)
                else:
                    a = a.detach().cpu().numpy()
            a = np.asarray(a)
            if a.dtype == np.uint16:
                dt = BF16
            else:
                a = a.astype(np.float32, copy=False)
                dt = F32
            a = np.ascontiguousarray(a)
            shape = (ctypes.c_int64 * max(a.ndim, 1))(*a.shape)
            self.arrays.append(a)
            self.shapes.append(shape)
            self.c[i] = ByocConst(a.ctypes.data, dt, a.ndim, shape)
        self.n = n


def validate(graph, consts):
    """Host-only check of a serialized subgraph against its constants."""
    lib = load_library()
    js = _json_bytes(graph)
    cs = _Consts(consts)
    _check(lib.byoc_subgraph_validate(js, len(js), cs.c, cs.n))


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


_ELEM_DTYPE = {"bf16": "torch.bfloat16", "f32": "torch.float32"}


def _check_tensor(t, desc, device, what):
    """Raises ByocError unless the torch tensor t matches the declared
    description (dtype, element count) and is a contiguous tensor on the
    engine's device.  Ints (raw device pointers) and None are not checked."""
    if t is None or isinstance(t, int):
        return
    want = _ELEM_DTYPE[desc["dtype"]]
    n = int(np.prod(desc["shape"])) if desc["shape"] else 1
    problems = []
    if str(t.dtype) != want:
        problems.append("dtype %s, declared %s" % (t.dtype, want))
    if t.numel() != n:
        problems.append("%d elements, declared %d %s" % (t.numel(), n, list(desc["shape"])))
    if t.device.type != "cuda" or (t.device.index if t.device.index is not None else 0) != int(device):
        problems.append("on %s, engine on cuda:%d" % (t.device, int(device)))
    if not t.is_contiguous():
        problems.append("not contiguous")
    if problems:
        raise ByocError(1, "%s: %s" % (what, "; ".join(problems)))


class Subgraph:
    """An execution engine for one serialized subgraph on one HIP device."""

    def __init__(self, graph, consts, device=0):
        self.lib = load_library()
        js = _json_bytes(graph)
        cs = _Consts(consts)
        h = ctypes.c_void_p()
        _check(self.lib.byoc_subgraph_create(js, len(js), cs.c, cs.n, int(device), ctypes.byref(h)))
        self.handle = h
        self.device = device
        self._options = 0
        n_in, n_out = ctypes.c_int32(), ctypes.c_int32()
        _check(self.lib.byoc_subgraph_num_io(h, ctypes.byref(n_in), ctypes.byref(n_out)))
        self.n_in, self.n_out = n_in.value, n_out.value
        self._descs = ([self.io_desc(0, i) for i in range(self.n_in)],
                       [self.io_desc(1, j) for j in range(self.n_out)])

    def io_desc(self, is_output, idx):
        d = TensorDesc()
        _check(self.lib.byoc_subgraph_io_desc(self.handle, int(is_output), int(idx), ctypes.byref(d)))
        return {"dtype": "bf16" if d.dtype == BF16 else "f32",
                "layout": ["NCHW", "NHWC", "ROWMAJOR"][d.layout],
                "shape": [d.shape[i] for i in range(d.ndim)]}

    def stats(self):
        m, w, a = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        _check(self.lib.byoc_subgraph_stats(self.handle, ctypes.byref(m), ctypes.byref(w), ctypes.byref(a)))
        return {"macs": m.value, "weight_bytes": w.value, "arena_bytes": a.value}

    def launches(self):
        n = ctypes.c_int32()
        _check(self.lib.byoc_subgraph_num_launches(self.handle, ctypes.byref(n)))
        out = []
        for i in range(n.value):
            li = LaunchInfo()
            _check(self.lib.byoc_subgraph_launch_info(self.handle, i, ctypes.byref(li)))
            out.append({"kind": KIND_NAMES[li.kind], "node": li.node, "flops": li.flops,
                        "bytes": li.bytes, "name": li.name.decode()})
        return out

    def _marshal(self, inputs, outputs, stream):
        """Pointer arrays and the raw stream of a run.  Torch tensors are
        checked against the declared dtype, element count, device and
        contiguity (a wrong buffer would make the kernels read or write out
        of bounds); raw integer pointers are passed through as they are."""
        if len(inputs) != self.n_in or len(outputs) != self.n_out:
            raise ByocError(1, "expected %d inputs and %d outputs, got %d and %d"
                            % (self.n_in, self.n_out, len(inputs), len(outputs)))
        for what, ts, descs in (("input", inputs, self._descs[0]), ("output", outputs, self._descs[1])):
            for i, (t, d) in enumerate(zip(ts, descs)):
                _check_tensor(t, d, self.device, "%s %d" % (what, i))
        ins = (ctypes.c_void_p * max(len(inputs), 1))(*[_ptr(t) for t in inputs])
        outs = (ctypes.c_void_p * max(len(outputs), 1))(*[_ptr(t) for t in outputs])
        if stream is None:
            import torch
            s = torch.cuda.current_stream(self.device).cuda_stream
        elif isinstance(stream, int):
            s = stream
        else:
            s = stream.cuda_stream
        return ins, outs, ctypes.c_void_p(s)

    def run(self, inputs, outputs, stream=None):
        """Enqueue one run on `stream` (a torch.cuda.Stream, a raw hipStream_t
        int, or None for torch's current stream)."""
        ins, outs, s = self._marshal(inputs, outputs, stream)
        _check(self.lib.byoc_subgraph_run(self.handle, ins, len(inputs), outs, len(outputs), s))

    def run_static(self, inputs, outputs, stream=None):
        """run() with the intermediates in the library's static per-device
        scratch (allocates nothing; direct launches)."""
        ins, outs, s = self._marshal(inputs, outputs, stream)
        _check(self.lib.byoc_subgraph_run_static(self.handle, ins, len(inputs), outs, len(outputs), s))

    def set_options(self, graph_replay=None, autotune=None):
        """Turn engine options on or off; None keeps an option as it is.

        graph_replay: HIP-graph replay of the launch sequence.
        autotune: time the result-identical kernel variants of every conv /
        dense composite on the device now and keep the fastest (off restores
        the built-in choice)."""
        flags = self._options
        if graph_replay is not None:
            flags = (flags | OPT_GRAPH_REPLAY) if graph_replay else (flags & ~OPT_GRAPH_REPLAY)
        if autotune is not None:
            flags = (flags | OPT_AUTOTUNE) if autotune else (flags & ~OPT_AUTOTUNE)
        _check(self.lib.byoc_subgraph_set_options(self.handle, flags))
        self._options = flags

    def profile_begin(self, max_runs):
        _check(self.lib.byoc_subgraph_profile_begin(self.handle, int(max_runs)))

    def profile_end(self):
        n = len(self.launches())
        ms = (ctypes.c_float * max(n, 1))()
        runs = ctypes.c_int32()
        _check(self.lib.byoc_subgraph_profile_end(self.handle, ms, n, ctypes.byref(runs)))
        return [ms[i] for i in range(n)], runs.value

    def close(self):
        if getattr(self, "handle", None):
            _check(self.lib.byoc_subgraph_destroy(self.handle))
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
