"""Shared helpers of the GPU parity tests: the tolerance metric of the
comparison, a one-ulp check for single composites, and device plumbing."""

import sys

import numpy as np

BF16_TOL = 1e-2   # max |gpu - oracle| / (|oracle| + 1), bf16 graphs
F32_TOL = 1e-4    # the same metric for fp32 graphs


def rel_err(gpu, ref):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    if gpu.size == 0:
        return 0.0
    return float(np.max(np.abs(gpu - ref) / (np.abs(ref) + 1.0)))


def bf16_ulp(v):
    """Spacing of bfloat16 numbers at |v| (normal range)."""
    a = np.maximum(np.abs(np.asarray(v, dtype=np.float64)), 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(a)) - 7)


def within_one_ulp(gpu, ref, scale=None):
    """True where the GPU value is within one bf16 ulp of the oracle's, plus
    2^-16 of the summed term magnitudes ``scale`` (sum |x||w| + |b| + |res|,
    see ``term_scale``): the fp32 accumulation error of a correct kernel is
    far below that slack, so only outputs whose terms cancel can use it."""
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    slack = 0.0 if scale is None else 2.0 ** -16 * np.asarray(scale, dtype=np.float64)
    return np.abs(gpu - ref) <= bf16_ulp(ref) * 1.0001 + slack + 1e-30


def term_scale_node(node, args):
    """Magnitude of the terms summed by one composite: the node evaluated in
    exact mode on the absolute values of its inputs and constants."""
    import oracle
    return oracle.run_node(node, [np.abs(np.asarray(a, dtype=np.float64)) for a in args], mode="exact")


def term_scale_graph(graph, consts, inputs):
    import oracle
    return oracle.run_graph(graph, [np.abs(np.asarray(c, dtype=np.float64)) for c in consts],
                            [np.abs(np.asarray(a, dtype=np.float64)) for a in inputs], mode="exact")


def announce(msg):
    print("[gpu case] " + msg, flush=True)
    sys.stdout.flush()
