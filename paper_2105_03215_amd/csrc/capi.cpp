// The extern "C" boundary of include/byoc.h.
#include <cstring>
#include <new>
#include <string>

#include "engine.h"
#include "graph.h"

struct byoc_subgraph {
  byoc::Engine* engine;
};

namespace {

thread_local std::string g_last_error;

byoc_status fail(const byoc::Status& st) {
  g_last_error = st.msg;
  return st.code;
}

byoc_status fail(byoc_status code, const char* msg) {
  g_last_error = msg;
  return code;
}

}  // namespace

extern "C" {

const char* byoc_last_error(void) { return g_last_error.c_str(); }

byoc_status byoc_subgraph_validate(const char* json, size_t len, const byoc_const* consts,
                                   int32_t n_consts) {
  g_last_error.clear();
  byoc::Graph g;
  byoc::Status st = byoc::parse_graph(json, len, consts, n_consts, &g);
  return st.ok() ? BYOC_OK : fail(st);
}

byoc_status byoc_subgraph_create(const char* json, size_t len, const byoc_const* consts,
                                 int32_t n_consts, int32_t device, byoc_subgraph** out) {
  g_last_error.clear();
  if (!out) return fail(BYOC_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  try {
    byoc::Graph g;
    byoc::Status st = byoc::parse_graph(json, len, consts, n_consts, &g);
    if (!st.ok()) return fail(st);
    byoc::Engine* e = nullptr;
    st = byoc::engine_create(std::move(g), consts, n_consts, device, &e);
    if (!st.ok()) return fail(st);
    byoc_subgraph* h = new byoc_subgraph{e};
    *out = h;
    return BYOC_OK;
  } catch (const std::bad_alloc&) {
    return fail(BYOC_ERR_OOM, "host allocation failed");
  } catch (...) {
    return fail(BYOC_ERR_INTERNAL, "unexpected exception in create");
  }
}

byoc_status byoc_subgraph_run(byoc_subgraph* g, const void* const* inputs, int32_t n_in,
                              void* const* outputs, int32_t n_out, void* stream) {
  g_last_error.clear();
  if (!g || !g->engine) return fail(BYOC_ERR_INVALID_ARG, "subgraph handle is NULL");
  byoc::Status st = byoc::engine_run(g->engine, inputs, n_in, outputs, n_out, (hipStream_t)stream);
  return st.ok() ? BYOC_OK : fail(st);
}

byoc_status byoc_subgraph_run_static(byoc_subgraph* g, const void* const* inputs, int32_t n_in,
                                     void* const* outputs, int32_t n_out, void* stream) {
  g_last_error.clear();
  if (!g || !g->engine) return fail(BYOC_ERR_INVALID_ARG, "subgraph handle is NULL");
  byoc::Status st = byoc::engine_run_static(g->engine, inputs, n_in, outputs, n_out, (hipStream_t)stream);
  return st.ok() ? BYOC_OK : fail(st);
}

byoc_status byoc_subgraph_destroy(byoc_subgraph* g) {
  g_last_error.clear();
  if (!g) return BYOC_OK;
  byoc::Status st = byoc::engine_destroy(g->engine);
  delete g;
  return st.ok() ? BYOC_OK : fail(st);
}

byoc_status byoc_subgraph_num_io(const byoc_subgraph* g, int32_t* n_in, int32_t* n_out) {
  g_last_error.clear();
  if (!g || !g->engine) return fail(BYOC_ERR_INVALID_ARG, "subgraph handle is NULL");
  if (n_in) *n_in = (int32_t)g->engine->graph.inputs.size();
  if (n_out) *n_out = (int32_t)g->engine->graph.outputs.size();
  return BYOC_OK;
}

byoc_status byoc_subgraph_io_desc(const byoc_subgraph* g, int32_t is_output, int32_t idx,
                                  byoc_tensor_desc* desc) {
  g_last_error.clear();
  if (!g || !g->engine) return fail(BYOC_ERR_INVALID_ARG, "subgraph handle is NULL");
  if (!desc) return fail(BYOC_ERR_INVALID_ARG, "desc is NULL");
  const byoc::Graph& gr = g->engine->graph;
  const auto& list = is_output ? gr.outputs : gr.inputs;
  if (idx < 0 || idx >= (int32_t)list.size()) return fail(BYOC_ERR_INVALID_ARG, "index out of range");
  const byoc::IoDesc& io = list[idx];
  const auto& shape = gr.values[io.value].shape;
  std::memset(desc, 0, sizeof(*desc));
  desc->dtype = (int32_t)io.dtype;
  desc->layout = (int32_t)io.layout;
  desc->ndim = (int32_t)shape.size();
  for (size_t i = 0; i < shape.size(); ++i) desc->shape[i] = shape[i];
  return BYOC_OK;
}

byoc_status byoc_subgraph_stats(const byoc_subgraph* g, int64_t* macs, int64_t* weight_bytes,
                                int64_t* arena_bytes) {
  g_last_error.clear();
  if (!g || !g->engine) return fail(BYOC_ERR_INVALID_ARG, "subgraph handle is NULL");
  if (macs) *macs = g->engine->graph.macs;
  if (weight_bytes) *weight_bytes = g->engine->weight_bytes;
  if (arena_bytes) *arena_bytes = g->engine->arena_bytes;
  return BYOC_OK;
}

byoc_status byoc_subgraph_num_launches(const byoc_subgraph* g, int32_t* n) {
  g_last_error.clear();
  if (!g || !g->engine || !n) return fail(BYOC_ERR_INVALID_ARG, "NULL argument");
  *n = (int32_t)g->engine->launches.size();
  return BYOC_OK;
}

byoc_status byoc_subgraph_launch_info(const byoc_subgraph* g, int32_t i, byoc_launch_info* info) {
  g_last_error.clear();
  if (!g || !g->engine || !info) return fail(BYOC_ERR_INVALID_ARG, "NULL argument");
  if (i < 0 || i >= (int32_t)g->engine->launches.size())
    return fail(BYOC_ERR_INVALID_ARG, "launch index out of range");
  *info = g->engine->launches[i].info;
  return BYOC_OK;
}

byoc_status byoc_subgraph_set_options(byoc_subgraph* g, int32_t flags) {
  g_last_error.clear();
  if (!g || !g->engine) return fail(BYOC_ERR_INVALID_ARG, "subgraph handle is NULL");
  byoc::Status st = byoc::engine_set_options(g->engine, flags);
  return st.ok() ? BYOC_OK : fail(st);
}

byoc_status byoc_subgraph_profile_begin(byoc_subgraph* g, int32_t max_runs) {
  g_last_error.clear();
  if (!g || !g->engine) return fail(BYOC_ERR_INVALID_ARG, "subgraph handle is NULL");
  byoc::Status st = byoc::engine_profile_begin(g->engine, max_runs);
  return st.ok() ? BYOC_OK : fail(st);
}

byoc_status byoc_subgraph_profile_end(byoc_subgraph* g, float* ms, int32_t n, int32_t* runs) {
  g_last_error.clear();
  if (!g || !g->engine) return fail(BYOC_ERR_INVALID_ARG, "subgraph handle is NULL");
  byoc::Status st = byoc::engine_profile_end(g->engine, ms, n, runs);
  return st.ok() ? BYOC_OK : fail(st);
}

}  // extern "C"
