"""Torch helpers around the C ABI: device buffers for a subgraph's declared
inputs and outputs, host <-> device conversion.  Torch only allocates memory
and provides streams; all subgraph arithmetic runs in the HIP library."""

import numpy as np
import torch

from .capi import Subgraph  # noqa: F401


def torch_dtype(name):
    return torch.bfloat16 if name == "bf16" else torch.float32


def to_device(arr, dtype_name, device):
    """Host float array -> device tensor of the declared dtype.  bf16-declared
    arrays must hold bf16-representable values (the conversion is exact)."""
    t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32))
    return t.to(device=device, dtype=torch_dtype(dtype_name)).contiguous()


def to_host_f64(t):
    return t.detach().to(device="cpu", dtype=torch.float32).numpy().astype(np.float64)


def inputs_for(sg, arrays, device):
    return [to_device(a, sg.io_desc(0, i)["dtype"], device) for i, a in enumerate(arrays)]


def outputs_for(sg, device):
    outs = []
    for j in range(sg.n_out):
        d = sg.io_desc(1, j)
        outs.append(torch.empty(d["shape"], dtype=torch_dtype(d["dtype"]), device=device))
    return outs


def run_once(sg, arrays, device="cuda:0"):
    """Upload, run on the current stream, synchronise and return host float64 outputs."""
    ins = inputs_for(sg, arrays, device)
    outs = outputs_for(sg, device)
    sg.run(ins, outs)
    torch.cuda.synchronize(device)
    return [to_host_f64(o) for o in outs]
