// Execution engine of one offloaded subgraph: the plan (launch sequence,
// arena layout, packed constants) built once at creation and replayed by
// every run (Sec. 3.4: the accelerator engine is initialised once, cached,
// and each invocation reads inputs, executes and writes outputs).
#pragma once

#include <hip/hip_runtime.h>

#include <string>
#include <vector>

#include "graph.h"
#include "kernels.h"

namespace byoc {

// Where a tensor lives during a run.
struct Ref {
  enum Kind : uint8_t { None, Arena, Input, Output, Weights } kind = None;
  int idx = -1;       // arena buffer id, input or output number
  int64_t off = 0;    // byte offset (weights region; within the buffer for an arena slice)
};

struct Launch {
  enum Op {
    ConvMfma, SplitReduce, ConvF32, Depthwise, MaxPoolBf16, AvgPoolBf16, MaxPoolF32, AvgPoolF32,
    AddBf16, AddF32, NchwToNhwc, NhwcToNchw, RowsToPadded, PaddedToRows, Cast, StemConvPool, DenseRows,
    ConvI8, MaxPoolI8, AvgPoolI8, AddI8, QuantizeI8, DequantizeI8, AvgPoolWinBf16, CopyChannels, QuantizeIm2colI8,
    DepthwiseI8, Bottleneck, IrBlock
  } op;
  byoc_launch_info info{};
  Ref x, w, bias, res, y, partial, other;
  ConvParams conv{};
  ConvTile tile{};
  ConvTile tile_default{};  // built-in choice (autotune may replace `tile`)
  ConvF32Params cf{};
  DwParams dw{};
  PoolParams pool{};
  StemParams stem{};
  QConvParams qc{};  // int8 conv / dense (qc.g holds the geometry; tile in `tile`)
  QAddParams qa{};   // int8 add
  QDwParams qd{};    // int8 depthwise conv
  // fused bottleneck block (Bottleneck): geometry and activations in bn,
  // the 1x1 reduce's weights and bias in w / bias, the 3x3's in w2 / b2,
  // the 1x1 expand's in w3 / b3, the projection's in wp / bp; res is x
  BottleneckParams bn{};
  // fused inverted-residual block (IrBlock): geometry in ir, the expand's
  // weights and bias in w / bias, the depthwise's in w2 / b2, the project's
  // in w3 / b3
  IrParams ir{};
  Ref w2, b2, w3, b3, wp, bp;
  int bnF = 0, bnC = 0, bnCout = 0, bnS = 1;
  bool bnI8 = false;  // on int8 codes (w*, b* hold the int8 conv's weights and tables)
  float qscale = 0.f;            // quantize: fl32(1 / S); dequantize: fl32(S)
  int qzero = 0;                 // quantize / dequantize zero point
  int qzx = 0, qzy = 0;          // int8 average pool: zero points
  float qm = 0.f;                //   and rescaling factor
  int64_t n = 0;
  int act = 0;
  float alpha = 0.f;  // leaky ReLU slope
  bool src_bf16 = false, dst_bf16 = false;
  bool count_include_pad = false;  // windowed average pool
  int N = 0, C = 0, H = 0, W = 0, Cp = 0, M = 0, K = 0, Kp = 0;
};

struct ArenaBuf {
  int64_t bytes = 0;
  int first = 0, last = 0;  // launch indices of definition and last use
  int64_t off = -1;
};

struct Engine {
  Graph graph;
  int device = 0;
  std::vector<Launch> launches;
  std::vector<ArenaBuf> bufs;
  char* arena = nullptr;
  int64_t arena_bytes = 0;
  char* weights = nullptr;
  int64_t weight_bytes = 0;
  // graph replay (BYOC_OPT_GRAPH_REPLAY)
  int options = 0;
  hipGraphExec_t gexec = nullptr;
  hipStream_t g_stream = nullptr;
  std::vector<const void*> g_in;
  std::vector<void*> g_out;
  // profiling
  std::vector<hipEvent_t> events;
  int prof_max_runs = 0;
  int prof_runs = 0;
  hipStream_t prof_last_stream = nullptr;
  // marks the end of the last run() on its stream; destroy waits for it
  hipEvent_t done = nullptr;
  // two-stream execution: launch i runs on the caller's stream (lstream 0)
  // or on the engine's side stream (1) and first waits for the event of
  // launch lwait[i] (>= 0) on the other stream; lrecord[i]: an event is
  // recorded after launch i
  bool two_streams = false;
  hipStream_t side = nullptr;
  std::vector<int8_t> lstream, lrecord;
  std::vector<int> lwait;
  std::vector<hipEvent_t> lev;
  hipEvent_t fork_ev = nullptr, join_ev = nullptr;
};

// Builds the plan and device state.  On failure releases everything.
Status engine_create(Graph&& g, const byoc_const* consts, int32_t n_consts, int device,
                     Engine** out);
Status engine_run(Engine* e, const void* const* inputs, int32_t n_in, void* const* outputs,
                  int32_t n_out, hipStream_t stream);
// run() with the intermediates in the library's static per-device scratch
// instead of the engine's arena: direct launches, no allocation of any kind.
Status engine_run_static(Engine* e, const void* const* inputs, int32_t n_in, void* const* outputs,
                         int32_t n_out, hipStream_t stream);
Status engine_destroy(Engine* e);
Status engine_set_options(Engine* e, int flags);
Status engine_profile_begin(Engine* e, int max_runs);
Status engine_profile_end(Engine* e, float* ms, int n, int* runs);

}  // namespace byoc
