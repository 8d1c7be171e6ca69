"""CPU oracle for executing an offloaded accelerator subgraph.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports this package:
only the test suite, the smoke check and the CPU-baseline leg of the benchmark
may call it.  It shares no code with the HIP library (different language, its
own JSON reading, its own bf16 rounding) and must stay that way.

What it computes.  An offloaded subgraph is the chain of composite functions
produced by pattern grouping (Sec. 3.1.1 of Chen et al., "Bring Your Own
Codegen to Deep Learning Compiler", arXiv 2105.03215): each composite is an
operator (Conv2D or Dense) optionally followed by a bias add and an
activation, serialized as a JSON node list carrying operator name, attributes
and dataflow (Sec. 3.3, Option 1).  The runtime reads the subgraph inputs,
executes the function and writes its outputs (Sec. 3.4, Fig. 6).  The paper
names the operators by their Relay names only; this package writes out their
standard definitions (cross-correlation convolution with zero padding, dense
as x W^T, max pooling with -inf padding, global average pooling, ReLU, ReLU6,
exact-erf GELU) in float64 NumPy, op by op and unfused.

Modules
-------
bf16   round-to-nearest-even of float64 values to bfloat16, done directly on
       the significand so there is no double rounding through float32.
ops    the operator definitions in float64.
graph  the JSON subgraph reader and executor, modes "exact" and "bf16io".
brute  pure-Python scalar loops of the same definitions, for tiny shapes.
quant  the affine int8 (partial quantization) definitions and an executor
       of int8 subgraphs.

Every function is pinned by a CPU test against something other than itself
(brute force, closed forms, library routines, invariants); see tests/.
"""

from .bf16 import round_bf16, bf16_bits  # noqa: F401
from . import ops, graph, brute, quant  # noqa: F401
from .graph import run_graph, run_node, load_graph  # noqa: F401
