"""MI355X (gfx950) executor for offloaded accelerator subgraphs.

The runtime half of the Bring-Your-Own-Codegen flow (Chen et al., arXiv
2105.03215, Sec. 3.4): a serialized chain of composite operators (conv2d /
dense with fused bias, residual add and activation; depthwise conv; pooling;
add) is turned once into an execution engine (packed constants, planned
arena, launch sequence of hand-written HIP kernels) and then run on
caller-owned device tensors on a caller stream.

Modules: ``capi`` (ctypes binding of include/byoc.h), ``runtime`` (torch
tensor helpers), ``workloads`` (seeded synthetic subgraphs), ``build``.
"""

from .capi import ByocError, Subgraph, load_library, validate  # noqa: F401
