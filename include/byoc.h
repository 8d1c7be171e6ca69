/*
 * byoc.h - C ABI of an MI355X (gfx950) executor for offloaded accelerator
 * subgraphs.
 *
 * Model.  In the Bring-Your-Own-Codegen flow (Chen et al., arXiv 2105.03215)
 * a partitioner groups operator sequences into composite functions
 * (Sec. 3.1.1: Conv2D, optional bias_add, activation), merges supported
 * operators into regions and encapsulates each region as a function bound
 * to an accelerator (Sec. 3.1.3).  The accelerator's code generator
 * serializes the function, by default as a JSON graph carrying operator
 * names, attributes and dataflow (Sec. 3.3, Option 1).  At run time the
 * constants are loaded once (metadata module, Sec. 3.4), the accelerator's
 * execution engine is built once and cached, and every invocation reads the
 * inputs from pre-allocated data entries, executes the function and writes
 * the outputs (Sec. 3.4, Fig. 6(b)(c)).  Intermediate results of the
 * function are owned by the accelerator engine, not by the data entries.
 *
 * This library is that accelerator engine:
 *   byoc_subgraph_create  = engine initialisation (parse, validate, plan,
 *                           upload and pack constants, allocate the
 *                           intermediate arena); done once per graph;
 *   byoc_subgraph_run     = one invocation on caller-owned device buffers,
 *                           enqueued on a caller stream;
 *   byoc_subgraph_destroy = release.
 *
 * Serialized format (schema "byoc-subgraph", version 1), a JSON object:
 *   "inputs":    [{"name", "shape", "dtype": "f32"|"bf16", "layout": "NCHW"|"ROWMAJOR"}]
 *   "constants": [{"name", "index", "shape", "dtype"}]   index into the
 *                constant array passed to create; conv weights OIHW, dense
 *                weights [out, in], biases [out]
 *   "nodes":     [{"name", "composite", "inputs": [names], "attrs", "out_dtype"}]
 *   "outputs":   [{"name", "dtype", "layout"}]
 * Composite names (the pattern names of Sec. 3.1.1; a composite applies
 * op -> bias -> residual add -> activation):
 *   conv2d[_bias][_add][_relu|_relu6|_gelu|_leaky]   inputs data, weight[, bias][, residual]
 *       attrs strides [sh,sw], padding [top,left,bottom,right], dilation [1,1],
 *       groups (1, or groups == in channels == out channels: depthwise)
 *   dense[_bias][_add][_relu|_relu6|_gelu|_leaky]    data [M,K], weight [N,K]
 *   max_pool2d        attrs pool_size, strides, padding (padding acts as -inf)
 *   avg_pool2d        attrs pool_size, strides (default 1), padding,
 *                     count_include_pad (default false: the divisor counts
 *                     the window positions inside the image); bf16 graphs
 *   global_avg_pool2d output [N, C]
 *   concatenate       one or more NCHW inputs of one batch and image joined
 *                     along channels (attrs axis 1), each with a multiple of
 *                     8 channels; bf16 graphs
 *   add[_relu|_relu6|_leaky] two tensors of one shape
 * A leaky ReLU (suffix _leaky) takes its slope from attrs alpha in [0, 1)
 * (default 0.1).
 * All nodes of a graph share one out_dtype, the graph's compute type:
 *   "bf16": bf16 activations, weights rounded to bf16 (nearest, ties to
 *           even), fp32 bias, fp32 accumulation, each node's output rounded
 *           to bf16; an "f32" input is rounded to bf16 at the boundary
 *           (the partial-quantization cast of Sec. 3.2, Fig. 4a);
 *   "f32":  fp32 throughout, true fp32 products;
 *   "int8": partial quantization (Sec. 3.2, Fig. 4a).  Every input and
 *           node carries "quant": {"scale": S > 0, "zero_point": Z in
 *           [-128, 127]} for the affine codes of its tensor, T = S (T_q - Z).
 *           Inputs are quantized at the boundary in fp32 arithmetic,
 *           q = clip(rint(x * fl32(1/S)) + Z); outputs are dequantized to
 *           their declared "f32" or "bf16" dtype, S (q - Z).  Weights are
 *           quantized per output channel, symmetric (S_w = max|W|/127);
 *           biases become int32 in the accumulator's scale.  Conv and dense
 *           accumulate exactly in int32 on int8 MFMA; every rescaling is
 *           rint(fl32(fl32(a) * m)) in float32, ties to even, saturated to
 *           +-2^20; activations act in code space (ReLU >= Z, ReLU6 <= Z +
 *           rint(6/S); leaky ReLU maps a negative offset t = q - Z to
 *           rint(fl32(t * alpha))).  A max pool keeps its input's S and Z;
 *           depthwise convs sum exactly on the vector ALU.  Not in int8
 *           graphs: GELU, windowed average pools, concatenation.
 * Internally activations of bf16 graphs are NHWC with channels padded to a
 * multiple of 8 (the layout-transform nodes of Sec. 3.2, Fig. 4b, sit at
 * the function boundary); callers always see the declared layouts.
 *
 * Errors.  Every call returns a status; on failure byoc_last_error() gives a
 * message naming the node and field.  The message is thread-local and valid
 * until the next byoc_* call on the same thread.  Argument and graph errors
 * are detected on the host before any device work.  Device faults of a run
 * surface at the caller's next synchronisation of the stream.
 */
#ifndef BYOC_H
#define BYOC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct byoc_subgraph byoc_subgraph; /* opaque engine handle */

typedef enum {
  BYOC_OK = 0,
  BYOC_ERR_INVALID_ARG = 1, /* NULL pointer, bad count or index          */
  BYOC_ERR_PARSE = 2,       /* malformed JSON or schema violation         */
  BYOC_ERR_UNSUPPORTED = 3, /* valid JSON naming something not supported */
  BYOC_ERR_SHAPE = 4,       /* shapes, dtypes or constants do not match   */
  BYOC_ERR_DEVICE = 5,      /* a HIP runtime call failed                  */
  BYOC_ERR_OOM = 6,         /* device allocation failed                   */
  BYOC_ERR_INTERNAL = 7
} byoc_status;

typedef enum { BYOC_F32 = 0, BYOC_BF16 = 1 } byoc_dtype;
typedef enum { BYOC_NCHW = 0, BYOC_NHWC = 1, BYOC_ROWMAJOR = 2 } byoc_layout;

/* One constant handed to create: host memory, C-contiguous, in the layout
 * the JSON declares (OIHW conv weights, [out,in] dense weights, [out]
 * biases).  dtype is a byoc_dtype; bf16 data are raw 16-bit patterns.
 * The library copies the data during create; the caller keeps ownership. */
typedef struct {
  const void* data;
  int32_t dtype;
  int32_t ndim;
  const int64_t* shape;
} byoc_const;

/* Declared dtype, layout and shape of a subgraph input or output. */
typedef struct {
  int32_t dtype;  /* byoc_dtype  */
  int32_t layout; /* byoc_layout */
  int32_t ndim;
  int32_t reserved;
  int64_t shape[8];
} byoc_tensor_desc;

/* Kind of a device launch in the run sequence (for profiling). */
typedef enum {
  BYOC_K_CONV_MFMA = 0, /* implicit-GEMM conv / dense on bf16 MFMA      */
  BYOC_K_CONV_F32 = 1,  /* fp32 direct conv / dense                     */
  BYOC_K_DEPTHWISE = 2, /* depthwise conv, vector ALU                   */
  BYOC_K_MAXPOOL = 3,
  BYOC_K_AVGPOOL = 4,
  BYOC_K_ADD = 5,       /* standalone elementwise add                   */
  BYOC_K_TRANSFORM = 6, /* boundary layout / dtype transform            */
  BYOC_K_REDUCE = 7,    /* split-K reduction with the fused epilogue    */
  BYOC_K_CONV_I8 = 8    /* implicit-GEMM conv / dense on int8 MFMA      */
} byoc_kernel_kind;

/* One entry of the launch sequence a run enqueues. */
typedef struct {
  int32_t kind;       /* byoc_kernel_kind                                   */
  int32_t node;       /* index of the JSON node, -1 for boundary transforms */
  int64_t flops;      /* algorithmic flops (2 x MACs for conv / dense)      */
  int64_t bytes;      /* algorithmic HBM bytes: inputs, weights, residual
                         read once and output written once                  */
  char name[64];      /* kernel name and tile configuration                 */
} byoc_launch_info;

/* Parse and check a serialized subgraph against its constants, on the host
 * only (no device call).  json need not be NUL-terminated (len bytes).
 * consts[i] is the constant whose JSON "index" is i.  Returns BYOC_OK or
 * the first error found. */
byoc_status byoc_subgraph_validate(const char* json, size_t len, const byoc_const* consts,
                                   int32_t n_consts);

/* Build the execution engine for a subgraph on HIP device `device`
 * (Sec. 3.4: constants loaded once, engine initialised once and cached):
 * validates, plans the launch sequence and the intermediate arena, uploads
 * and packs the constants, allocates device memory, and synchronises.  On
 * success *out owns all device memory of the engine; on failure *out is
 * NULL and nothing leaks.  Shapes, including the batch, are fixed per
 * engine. */
byoc_status byoc_subgraph_create(const char* json, size_t len, const byoc_const* consts,
                                 int32_t n_consts, int32_t device, byoc_subgraph** out);

/* Enqueue one invocation on `stream` (a hipStream_t; NULL = the null
 * stream) and return without synchronising.  inputs[i] / outputs[j] are
 * device pointers to contiguous buffers with the dtype, layout and shape
 * reported by byoc_subgraph_io_desc, in JSON order; outputs must not
 * overlap inputs or each other.  No allocation, no host-device copy.  The
 * engine's arena is shared by its runs: calls on one engine must be
 * serialised on one stream, or use one engine per concurrent stream. */
byoc_status byoc_subgraph_run(byoc_subgraph* g, const void* const* inputs, int32_t n_in,
                              void* const* outputs, int32_t n_out, void* stream);

/* Capacity of the static scratch that byoc_subgraph_run_static uses. */
#define BYOC_STATIC_SCRATCH_BYTES ((int64_t)64 << 20)

/* For callers that cannot allocate device memory while they run (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * byoc_subgraph_run with the engine's intermediates (activations between
 * composites, split-K partial sums, concatenation buffers) placed in a
 * static scratch array of BYOC_STATIC_SCRATCH_BYTES that the library holds
 * on every GPU it runs on until the process ends, instead of the engine's
 * own arena.  Arguments, layouts and ownership as for byoc_subgraph_run;
 * always direct launches (no graph replay, no profiling events), and no
 * allocation, no host-device copy and no synchronisation of any kind.  The
 * first call on a device looks up that device's scratch address once.
 * Engines whose intermediates need more than BYOC_STATIC_SCRATCH_BYTES
 * (byoc_subgraph_stats' arena_bytes) are rejected with
 * BYOC_ERR_INVALID_ARG before anything is enqueued.  Every call on one GPU,
 * from any engine, shares that GPU's scratch, which keeps the last call's
 * contents (nothing in it needs clearing: every intermediate is written
 * before it is read): calls that overlap on one GPU - on two streams, or
 * from two threads - race and must be serialised by the caller.  Outputs
 * are bit-for-bit those of byoc_subgraph_run.  byoc_subgraph_destroy does
 * not wait for these runs: synchronise their stream first. */
byoc_status byoc_subgraph_run_static(byoc_subgraph* g, const void* const* inputs, int32_t n_in,
                                     void* const* outputs, int32_t n_out, void* stream);

/* Wait for the last run enqueued by byoc_subgraph_run (on whatever stream
 * it was enqueued), then free every allocation of the engine and the
 * handle; other streams and the rest of the device are not synchronised.
 * NULL is a no-op returning BYOC_OK. */
byoc_status byoc_subgraph_destroy(byoc_subgraph* g);

/* Number of subgraph inputs and outputs. */
byoc_status byoc_subgraph_num_io(const byoc_subgraph* g, int32_t* n_in, int32_t* n_out);

/* Declared description of input (is_output = 0) or output (1) number idx. */
byoc_status byoc_subgraph_io_desc(const byoc_subgraph* g, int32_t is_output, int32_t idx,
                                  byoc_tensor_desc* desc);

/* Multiply-accumulates of the conv and dense composites (the cost measure
 * of the paper's TensorRT fallback rule, Sec. 4.1), bytes of packed
 * constants and bytes of the intermediate arena.  Any pointer may be NULL. */
byoc_status byoc_subgraph_stats(const byoc_subgraph* g, int64_t* macs, int64_t* weight_bytes,
                                int64_t* arena_bytes);

/* Number of device launches one run enqueues, and their descriptions. */
byoc_status byoc_subgraph_num_launches(const byoc_subgraph* g, int32_t* n);
byoc_status byoc_subgraph_launch_info(const byoc_subgraph* g, int32_t i, byoc_launch_info* info);

/* Per-launch timing.  byoc_subgraph_profile_begin(g, max_runs) allocates
 * HIP events for max_runs runs; each following run records an event on its
 * stream before its first launch and after every launch.  profile_end
 * synchronises on the last recorded event, writes into ms[i] (n >= number
 * of launches) the summed duration of launch i over the recorded runs,
 * stores that run count in *runs, and frees the events.  Runs past
 * max_runs are not recorded. */
byoc_status byoc_subgraph_profile_begin(byoc_subgraph* g, int32_t max_runs);
byoc_status byoc_subgraph_profile_end(byoc_subgraph* g, float* ms, int32_t n, int32_t* runs);

/* Engine options (bit flags) for byoc_subgraph_set_options. */
enum { BYOC_OPT_GRAPH_REPLAY = 1, BYOC_OPT_AUTOTUNE = 2 };

/* Set engine options (default 0).  BYOC_OPT_GRAPH_REPLAY: run() records its
 * launch sequence as a HIP graph the first time it sees a (stream, inputs,
 * outputs) combination and afterwards replays that graph - one graph launch
 * instead of one launch per kernel - while the combination repeats; a new
 * combination is recorded again.  Recording and instantiating allocate host
 * and device memory on those runs, so an allocation-free run() needs the
 * option off.  Runs on the NULL stream, runs while profiling and runs on a
 * stream that is already being captured by the caller use direct launches.
 * BYOC_OPT_AUTOTUNE: when the bit is turned on, this call times on the
 * device (synchronously, on a stream of its own, with scratch input and
 * output buffers it allocates and frees) every kernel variant the engine
 * has for each convolution / dense composite whose results are bit-for-bit
 * those of the built-in choice (same tile reduction order, no split-K
 * change) and keeps the fastest; turning it off restores the built-in
 * choice.  The computed values never change, only the speed.  Unknown flag
 * bits are rejected with BYOC_ERR_INVALID_ARG. */
byoc_status byoc_subgraph_set_options(byoc_subgraph* g, int32_t flags);

/* Thread-local text of the last error ("" if none). */
const char* byoc_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* BYOC_H */
