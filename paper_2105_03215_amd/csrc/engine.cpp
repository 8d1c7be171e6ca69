// Engine creation (planning, constant packing, arena layout) and runs.
#include "engine.h"
#include "static_scratch.h"

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>

namespace byoc {
namespace {

int64_t rup(int64_t a, int64_t b) { return (a + b - 1) / b * b; }
int64_t numel(const std::vector<int64_t>& s) {
  int64_t n = 1;
  for (int64_t d : s) n *= d;
  return n;
}

#define HIP_TRY(expr, what)                                                                   \
  do {                                                                                        \
    hipError_t e_ = (expr);                                                                   \
    if (e_ != hipSuccess)                                                                     \
      return Status::Err(e_ == hipErrorOutOfMemory ? BYOC_ERR_OOM : BYOC_ERR_DEVICE,          \
                         std::string(what) + ": " + hipGetErrorString(e_));                   \
  } while (0)

constexpr int kRowPad = 256;  // packed weight rows are padded to this (>= any tile BN)
constexpr int kKPad = 64;     // packed reduction length is padded to this (the stage depth)
constexpr int kHaloStages = 3;  // halo kernel weight ring: 3 stages of one kernel row (built-in choice)

struct PackJob {
  enum Kind { ConvW, DwW, DwW32, Vec, Copy, StemW, Host } kind;  // Host: copy blob n, built on the host
  int cidx = -1;       // constant index
  int64_t dst = 0;     // byte offset in the weights region
  int K = 0, Cg = 0, R = 0, S = 0, Cp = 0, Kgp = 0, rows = 0;
  int n = 0, n_out = 0;
};

// float32 form of a real rescaling factor of an int8 graph (rounded from
// float64); false unless finite, positive and below 2^20.
bool rescale_factor(double m, float* out) {
  const float f = (float)m;
  if (!(std::isfinite(f) && f > 0.0f && f < 1048576.0f)) return false;
  *out = f;
  return true;
}

// Chooses the workgroup tile (and split-K factor) of an implicit GEMM.  The
// kernel is latency bound per stage, so the model favours the largest tile
// that still yields about two workgroups per CU, and shares a long
// reduction between several wave groups of one workgroup when the output
// has too few tiles (split-K over workgroups, reduced deterministically by
// a second kernel, only when asked for).
void choose_conv_tile(int64_t M, int Kp, int Kg, ConvTile* t, int* splits, int* kps) {
  // Measured on MI355X over the ResNet-50 layers: 64x64 tiles (16x16x32
  // MFMA) win at most batch-32 shapes - larger tiles leave fewer workgroups
  // per CU to overlap each one's load/compute/epilogue phases - and split-K
  // only pays when the output has very few tiles.  Layers with few tiles and
  // a long reduction are latency bound: there two reduction groups per
  // workgroup (HBM->LDS pipeline) double the loads in flight.
  t->bm = M >= 48 ? 64 : 32;
  t->bn = 64;
  t->mf = 16;
  t->stages = 0;
  t->threads = 256;
  t->kgroups = 1;
  const int nk = (int)((Kg + kKPad - 1) / kKPad);
  const int64_t tiles = ((M + t->bm - 1) / t->bm) * ((Kp + t->bn - 1) / t->bn);
  *splits = 1;
  *kps = nk;
  if (tiles < 64 && nk >= 8) {
    int s = (int)std::min<int64_t>(nk / 4, (128 + tiles - 1) / tiles);
    s = std::max(1, std::min(s, 16));
    // Measured on MI355X (ResNet-18 block and ResNet-50 at batch 1): where
    // split-K would split only two ways, four reduction groups of 4 waves
    // sharing each tile's stages inside one workgroup (sums added in the
    // epilogue) beat the split and its reduce launch (a 3x3 64-channel
    // layer at 56x56: 8.4 against 12.5 us); where it splits four or more
    // ways, its extra workgroups win.  BYOC_CONV_KG4_MAXSPLIT=<n> moves the
    // threshold (0: always split-K).
    int kg4_max = 2;
    if (const char* e = std::getenv("BYOC_CONV_KG4_MAXSPLIT")) kg4_max = std::atoi(e);
    if (s > 1 && s <= kg4_max) {
      t->stages = 2;
      t->threads = 1024;
      t->kgroups = 4;
      return;
    }
    if (s > 1) {
      *kps = (nk + s - 1) / s;
      *splits = (nk + *kps - 1) / *kps;
      return;
    }
  }
  if (tiles <= 256 && nk >= 8) {
    t->stages = 3;
    t->threads = 512;
    t->kgroups = 2;
  }
}

// Tuning override (environment, read at engine creation):
// BYOC_CONV_TILE=<bm>x<bn>[x<mfma 16|32>] (register-staged) or d<bm>x<bn>s<stages>
// (HBM->LDS pipeline) forces a compiled tile, BYOC_CONV_SPLIT=<n> a
// split-K factor, for every conv/dense composite of the engine.
void apply_tile_override(int Kg, ConvTile* t, int* splits, int* kps) {
  const char* split_env = std::getenv("BYOC_CONV_SPLIT");
  if (split_env && !std::getenv("BYOC_CONV_TILE") && t->kgroups > 1) {
    // a forced split-K runs on the register-staged kernel
    t->stages = 0;
    t->threads = 256;
    t->kgroups = 1;
  }
  if (const char* e = std::getenv("BYOC_CONV_TILE")) {
    int bm = 0, bn = 0, mf = 16;
    int ns = 0;
    if (e[0] == 'h') {
      // h<bm>x<bn>s<stages>: halo kernel (3x3 stride-1 convs only; others keep their tile)
      if (std::sscanf(e + 1, "%dx%ds%d", &bm, &bn, &ns) == 3) {
        t->bm = bm;
        t->bn = bn;
        t->mf = 16;
        t->stages = ns;
        t->threads = 512;
        t->kgroups = 1;
        t->halo = 2;  // requested; resolved against the shape by the planner
      }
    } else if (e[0] == 'd') {
      // d<bm>x<bn>s<stages>[t<threads>[k<groups>]]: direct HBM->LDS pipeline
      int nt = 256, kgr = 1;
      if (std::sscanf(e + 1, "%dx%ds%dt%dk%d", &bm, &bn, &ns, &nt, &kgr) >= 3 &&
          conv_dma_tile_supported(bm, bn, ns, nt, kgr)) {
        t->bm = bm;
        t->bn = bn;
        t->mf = 16;
        t->stages = ns;
        t->threads = nt;
        t->kgroups = kgr;
      }
    } else {
      const int got = std::sscanf(e, "%dx%dx%d", &bm, &bn, &mf);
      if (got >= 2 && conv_mfma_tile_supported(bm, bn, mf)) {
        t->bm = bm;
        t->bn = bn;
        t->mf = mf;
        t->stages = 0;
      }
    }
  }
  if (t->kgroups > 1) {  // reduction groups replace split-K
    *splits = 1;
    *kps = (Kg + kKPad - 1) / kKPad;
    return;
  }
  if (const char* e = split_env) {
    const int nk = (Kg + kKPad - 1) / kKPad;
    const int sp = std::max(1, std::min(std::atoi(e), nk));
    *kps = (nk + sp - 1) / sp;
    *splits = (nk + *kps - 1) / *kps;
  }
}

// XCD placement of conv_dma tiles: the (8 / py) x py split of the tile grid
// that minimises one XCD's working set (its share of the input activations
// plus its share of the packed weights), so that each XCD's L2 serves the
// re-reads of its tiles.  BYOC_CONV_XCD=<py> (0 = linear order) overrides.
int choose_xcd_split(const ConvParams& p, const ConvTile& t) {
  if (const char* e = std::getenv("BYOC_CONV_XCD")) {
    const int v = std::atoi(e);
    if (v == 0 || v == 1 || v == 2 || v == 4 || v == 8) return v;
  }
  const int64_t ntm = (p.M + t.bm - 1) / t.bm, ntn = (p.Kp + t.bn - 1) / t.bn;
  const double a = (double)p.x_bytes, w = (double)p.Kp * p.Kg * 2.0;
  int best = 0;
  double best_ws = 0;
  for (int py : {1, 2, 4, 8}) {
    const int px = 8 / py;
    if (py > ntn || px > ntm) continue;
    const double ws = a / px + w / py;
    if (best == 0 || ws < best_ws) {
      best = py;
      best_ws = ws;
    }
  }
  return best;
}

void name_conv_i8(Launch& L) {
  if (L.tile.halo)
    std::snprintf(L.info.name, sizeof(L.info.name), "conv_i8_halo_%dx%d_s%d_lp%d_pb%d", L.tile.bm, L.tile.bn,
                  L.tile.stages, L.tile.lp, L.tile.npb);
  else
    std::snprintf(L.info.name, sizeof(L.info.name), L.tile.kgroups > 1 ? "conv_i8_%dx%d_s%d_w%d_k%d" : "conv_i8_%dx%d_s%d_w%d",
                  L.tile.bm, L.tile.bn, L.tile.stages, L.tile.threads / 64, L.tile.kgroups);
}

void name_conv(Launch& L) {
  if (L.tile.halo)
    std::snprintf(L.info.name, sizeof(L.info.name), "conv_halo_%dx%d_s%d_lp%d_pb%d", L.tile.bm, L.tile.bn,
                  L.tile.stages, L.tile.lp, L.tile.npb);
  else if (L.tile.stages > 0)
    std::snprintf(L.info.name, sizeof(L.info.name), "conv_dma_%dx%d_s%d_w%d_k%d_split%d", L.tile.bm, L.tile.bn,
                  L.tile.stages, L.tile.threads / 64, L.tile.kgroups, L.conv.splits);
  else
    std::snprintf(L.info.name, sizeof(L.info.name), "conv_mfma_%dx%d_mf%d_split%d", L.tile.bm, L.tile.bn,
                  L.tile.mf, L.conv.splits);
}

struct Planner {
  Engine* e;
  Graph& g;
  bool bf16;
  std::vector<Ref> loc;
  std::vector<int> cp;  // channel stride of each value's internal form
  std::vector<PackJob> jobs;
  int64_t wbytes = 0;
  Status err;
  // fused stems: conv node -> its max-pool node, max-pool node -> conv node
  std::vector<int> stem_pool, stem_conv;
  std::vector<int> post_add, post_conv;  // conv -> the add folded into it, and back
  // zero-copy concatenation: value -> the concatenation it is written into
  // (-1: none) and its first channel there
  std::vector<int> alias_of, alias_off;
  // int8 graphs: input value -> the conv node that reads it as im2col rows (-1: none)
  std::vector<int> im2col_of;
  // fused bottleneck blocks: 1x1 expand node -> its 3x3 node (-1: none) and
  // its projection node (-1: none), and the nodes planned with it
  std::vector<int> block_mid, block_proj;
  std::vector<bool> in_block;
  // fused inverted-residual blocks: 1x1 project node -> its depthwise node
  // (-1: none) and its expand node (-1: none), and the nodes planned with it
  std::vector<int> ir_dw, ir_exp;
  std::vector<bool> in_ir;

  bool i8;                                  // partially quantized (int8) graph
  const byoc_const* consts = nullptr;       // host constants (int8 weights are quantized on the host)
  std::vector<std::vector<uint8_t>> blobs;  // host-built constant blocks (PackJob::Host)

  Planner(Engine* e_, Graph& g_) : e(e_), g(g_), bf16(g_.compute == DType::BF16), i8(g_.compute == DType::I8) {
    loc.resize(g.values.size());
    cp.assign(g.values.size(), 0);
  }

  int64_t internal_bytes(int v) const {
    const auto& s = g.values[v].shape;
    if (i8) return (s.size() == 4 ? s[0] * s[2] * s[3] : s[0]) * rup(s[1], 16);
    if (!bf16) return numel(s) * 4;
    const int64_t c = rup(s[1], 8);
    return (s.size() == 4 ? s[0] * s[2] * s[3] : s[0]) * c * 2;
  }
  Ref arena(int64_t bytes) {
    ArenaBuf b;
    b.bytes = rup(bytes, 256);
    b.first = INT_MAX;
    b.last = -1;
    e->bufs.push_back(b);
    Ref r;
    r.kind = Ref::Arena;
    r.idx = (int)e->bufs.size() - 1;
    return r;
  }
  Ref wslot(int64_t bytes) {
    Ref r;
    r.kind = Ref::Weights;
    r.off = wbytes;
    wbytes += rup(bytes, 256);
    return r;
  }
  static Ref io(Ref::Kind k, int i) {
    Ref r;
    r.kind = k;
    r.idx = i;
    return r;
  }
  void name(Launch& L, const char* s) { std::snprintf(L.info.name, sizeof(L.info.name), "%s", s); }

  int64_t ext_bytes(int v, DType dt) const {
    return numel(g.values[v].shape) * (dt == DType::BF16 ? 2 : 4);
  }
  int64_t act_bytes(int v) const { return numel(g.values[v].shape) * (i8 ? 1 : (bf16 ? 2 : 4)); }
  Ref host_blob(std::vector<uint8_t>&& b) {
    Ref r = wslot((int64_t)b.size());
    PackJob j{PackJob::Host};
    j.dst = r.off;
    j.n = (int)blobs.size();
    jobs.push_back(j);
    blobs.push_back(std::move(b));
    return r;
  }

  Status plan();
  Status plan_i8();
  void plan_node(int ni);
  void plan_node_i8(int ni);
  bool quantize_conv_i8(const Node& n, int Cp, int Kgp, int rows, bool im2col, bool border,
                        std::vector<uint8_t>& packed, std::vector<int32_t>& qch, std::vector<int32_t>& wtap,
                        std::string* err_msg, int row_ld = 0);
  void plan_stem_i8(int conv_ni, int pool_ni);
  void find_post_adds();
  void find_stems();
  void find_concat_aliases();
  void find_blocks();
  void plan_block(int ci);
  void find_ir_blocks();
  void plan_ir(int ci);
  void plan_block_i8(int ci);
  Ref slice(int vcat, int channel) const {  // channel slice of a concatenation's buffer
    Ref r = loc[vcat];
    r.off += (int64_t)channel * 2;
    return r;
  }
  void plan_stem(int conv_ni, int pool_ni);
};

// A graph input in NCHW with at most 4 channels feeding only a conv whose
// output feeds only a max pool is planned as one fused stem kernel: the
// input is read in place (no layout transform) and the full-resolution conv
// output never exists.
void Planner::find_stems() {
  stem_pool.assign(g.nodes.size(), -1);
  stem_conv.assign(g.nodes.size(), -1);
  const char* env = std::getenv("BYOC_FUSE_STEM");  // =0: never fuse
  if (!(bf16 || i8) || (env && env[0] == '0')) return;
  auto uses = [&](int v, int* user) {
    int count = 0;
    for (size_t ni = 0; ni < g.nodes.size(); ++ni) {
      const Node& n = g.nodes[ni];
      for (int u : {n.data, n.weight, n.bias, n.residual, n.other})
        if (u == v) {
          ++count;
          *user = (int)ni;
        }
    }
    for (const IoDesc& o : g.outputs)
      if (o.value == v) count += 2;
    return count;
  };
  for (const IoDesc& in : g.inputs) {
    const auto& xs = g.values[in.value].shape;
    if (xs.size() != 4 || in.layout != BYOC_NCHW) continue;
    int ci = -1, pi = -1;
    if (uses(in.value, &ci) != 1) continue;
    const Node& c = g.nodes[ci];
    if (c.op != OpKind::Conv || c.data != in.value || c.depthwise || c.groups != 1 || c.residual >= 0) continue;
    if (uses(c.out, &pi) != 1) continue;
    const Node& pn = g.nodes[pi];
    if (pn.op != OpKind::MaxPool || pn.data != c.out) continue;
    const auto& ws = g.values[c.weight].shape;
    if (!stem_supported((int)xs[1], (int)ws[0], (int)ws[2], (int)ws[3], c.stride[0], c.stride[1], pn.pool[0],
                        pn.pool[1], pn.stride[0], pn.stride[1]))
      continue;
    // codes: a clamp activation, and the pool keeps the conv's (scale, zero point)
    if (i8 && (c.act == Act::Gelu || c.act == Act::Leaky || g.values[pn.out].qscale != g.values[c.out].qscale ||
               g.values[pn.out].qzero != g.values[c.out].qzero))
      continue;
    stem_pool[ci] = pi;
    stem_conv[pi] = ci;
  }
}

void Planner::plan_stem(int ci, int pi) {
  const Node& c = g.nodes[ci];
  const Node& pn = g.nodes[pi];
  const auto& xs = g.values[c.data].shape;
  const auto& cs = g.values[c.out].shape;
  const auto& ps = g.values[pn.out].shape;
  const auto& ws = g.values[c.weight].shape;
  const int in_idx = g.values[c.data].index;
  Launch L;
  L.op = Launch::StemConvPool;
  L.info.kind = BYOC_K_CONV_MFMA;
  L.info.node = ci;
  L.x = loc[c.data];
  L.y = loc[pn.out];
  StemParams& p = L.stem;
  p.x_bf16 = g.inputs[in_idx].dtype == DType::BF16;
  p.N = (int)xs[0], p.C = (int)xs[1], p.H = (int)xs[2], p.W = (int)xs[3];
  p.R = (int)ws[2], p.S = (int)ws[3], p.sh = c.stride[0], p.sw = c.stride[1], p.pt = c.pad[0], p.pl = c.pad[1];
  p.P = (int)cs[2], p.Q = (int)cs[3];
  p.kph = pn.pool[0], p.kpw = pn.pool[1], p.sph = pn.stride[0], p.spw = pn.stride[1];
  p.ppt = pn.pad[0], p.ppl = pn.pad[1];
  p.PO = (int)ps[2], p.QO = (int)ps[3];
  p.act = (int)c.act;
  p.alpha = c.alpha;
  p.wld = stem_weight_ld(p.R);
  // BYOC_STEM_GRID=<n>: at most n persistent workgroups (tests drive several
  // tiles through one workgroup on small inputs with it)
  if (const char* ev = std::getenv("BYOC_STEM_GRID")) p.grid_cap = std::max(0, std::atoi(ev));
  const int wc = g.values[c.weight].index;
  const int bc = c.bias >= 0 ? g.values[c.bias].index : -1;
  L.w = wslot((int64_t)64 * p.wld * 2);
  PackJob j{PackJob::StemW, wc, L.w.off, 64, p.C, p.R, p.S, 0, 0, 0, p.wld, 0};
  jobs.push_back(j);
  L.bias = wslot(64 * 4);
  jobs.push_back({PackJob::Vec, bc, L.bias.off, 0, 0, 0, 0, 0, 0, 0, bc >= 0 ? 64 : 0, 64});
  L.info.flops = 2 * c.macs;
  L.info.bytes = ext_bytes(c.data, g.inputs[in_idx].dtype) + numel(ws) * 2 + 64 * 4 + act_bytes(pn.out);
  name(L, "stem_conv_maxpool");
  e->launches.push_back(L);
}

// The int8 stem: the input's codes formed in the kernel (the boundary
// quantize of that input is not planned), weights quantized on the host as
// the int8 conv has them, in the stem's cell layout.
void Planner::plan_stem_i8(int ci, int pi) {
  const Node& c = g.nodes[ci];
  const Node& pn = g.nodes[pi];
  const Value& xv = g.values[c.data];
  const Value& yv = g.values[c.out];
  const auto& xs = xv.shape;
  const auto& cs = yv.shape;
  const auto& ps = g.values[pn.out].shape;
  const auto& ws = g.values[c.weight].shape;
  const int in_idx = xv.index;
  Launch L;
  L.op = Launch::StemConvPool;
  L.info.kind = BYOC_K_CONV_I8;
  L.info.node = ci;
  L.x = loc[c.data];
  L.y = loc[pn.out];
  StemParams& p = L.stem;
  p.x_bf16 = g.inputs[in_idx].dtype == DType::BF16;
  p.N = (int)xs[0], p.C = (int)xs[1], p.H = (int)xs[2], p.W = (int)xs[3];
  p.R = (int)ws[2], p.S = (int)ws[3], p.sh = c.stride[0], p.sw = c.stride[1], p.pt = c.pad[0], p.pl = c.pad[1];
  p.P = (int)cs[2], p.Q = (int)cs[3];
  p.kph = pn.pool[0], p.kpw = pn.pool[1], p.sph = pn.stride[0], p.spw = pn.stride[1];
  p.ppt = pn.pad[0], p.ppl = pn.pad[1];
  p.PO = (int)ps[2], p.QO = (int)ps[3];
  p.act = (int)c.act;
  p.i8 = 1;
  p.inv_scale = (float)(1.0 / xv.qscale);  // as the boundary quantize has it
  p.zx = xv.qzero;
  p.zy = yv.qzero;
  p.lo = -128, p.hi = 127;
  if (c.act == Act::Relu || c.act == Act::Relu6) p.lo = yv.qzero;
  if (c.act == Act::Relu6) {
    const double h = yv.qzero + std::nearbyint(6.0 / yv.qscale);
    p.hi = h < 127.0 ? (int)h : 127;
  }
  p.wld = stem_weight_ld_i8(p.R);
  if (const char* ev = std::getenv("BYOC_STEM_GRID")) p.grid_cap = std::max(0, std::atoi(ev));
  std::vector<uint8_t> packed;
  std::vector<int32_t> qch, wtap;
  std::string why;
  if (!quantize_conv_i8(c, 4, p.wld, 64, true, false, packed, qch, wtap, &why, 32)) {
    err = Status::Err(BYOC_ERR_UNSUPPORTED, "node " + std::to_string(ci) + " (" + c.composite + "): " + why);
    return;
  }
  L.w = host_blob(std::move(packed));
  std::vector<uint8_t> qb(qch.size() * 4);
  std::memcpy(qb.data(), qch.data(), qb.size());
  L.bias = host_blob(std::move(qb));
  L.info.flops = 2 * c.macs;
  L.info.bytes = ext_bytes(c.data, g.inputs[in_idx].dtype) + numel(ws) + 64 * 8 + act_bytes(pn.out);
  name(L, "stem_conv_maxpool_i8");
  e->launches.push_back(L);
}

// A concatenation's input produced by a conv, max pool or windowed average
// pool that nothing else reads is written by its producer straight into its
// channel slice of the concatenation's buffer (output pixel stride = the
// concatenation's channels); other inputs are copied in.
void Planner::find_concat_aliases() {
  alias_of.assign(g.values.size(), -1);
  alias_off.assign(g.values.size(), 0);
  std::vector<int> uses(g.values.size(), 0);
  for (const Node& n : g.nodes) {
    for (int a : {n.data, n.residual, n.other})
      if (a >= 0) ++uses[a];
    if (n.op == OpKind::Concat)
      for (size_t k = 1; k < n.cat.size(); ++k) ++uses[n.cat[k]];
  }
  for (const IoDesc& o : g.outputs) ++uses[o.value];
  for (size_t ni = 0; ni < g.nodes.size(); ++ni) {
    const Node& c = g.nodes[ni];
    if (c.op != OpKind::Concat) continue;
    int off = 0;
    for (int a : c.cat) {
      const Value& v = g.values[a];
      if (v.source == Value::Node && uses[a] == 1 && alias_of[a] < 0) {
        const Node& p = g.nodes[v.index];
        const bool kind = (p.op == OpKind::Conv && !p.depthwise) || p.op == OpKind::MaxPool ||
                          p.op == OpKind::AvgPoolWin;
        if (kind && stem_pool[v.index] < 0 && stem_conv[v.index] < 0) {
          alias_of[a] = c.out;
          alias_off[a] = off;
        }
      }
      off += (int)v.shape[1];
    }
  }
}

// A bf16 add reading a conv's activated output that nothing else reads (the
// residual of DarkNet's blocks comes after the leaky ReLU) folds into that
// conv: the conv is planned at the add, writes the add's output and adds the
// other operand to its bf16-rounded activation, which is the add's own
// arithmetic.  BYOC_FUSE_POST_ADD=0 keeps the two launches.
void Planner::find_post_adds() {
  post_add.assign(g.nodes.size(), -1);
  post_conv.assign(g.nodes.size(), -1);
  const char* env = std::getenv("BYOC_FUSE_POST_ADD");
  if (!(bf16 || i8) || (env && env[0] == '0')) return;
  std::vector<int> uses(g.values.size(), 0);
  for (const Node& n : g.nodes) {
    for (int a : {n.data, n.residual, n.other})
      if (a >= 0) ++uses[a];
    if (n.op == OpKind::Concat)
      for (size_t k = 1; k < n.cat.size(); ++k) ++uses[n.cat[k]];
  }
  for (const IoDesc& o : g.outputs) ++uses[o.value];
  for (size_t ai = 0; ai < g.nodes.size(); ++ai) {
    const Node& a = g.nodes[ai];
    if (a.op != OpKind::Add || a.act != Act::None) continue;
    for (int v : {a.data, a.other}) {
      const Value& cv = g.values[v];
      if (cv.source != Value::Node || uses[v] != 1 || cv.shape.size() != 4) continue;
      if (!alias_of.empty() && alias_of[v] >= 0) continue;
      const int ci = cv.index;
      const Node& c = g.nodes[ci];
      if (c.op != OpKind::Conv || c.depthwise || c.residual >= 0 || c.act == Act::Gelu) continue;
      if (post_add[ci] >= 0) continue;
      if (!stem_pool.empty() && (stem_pool[ci] >= 0 || stem_conv[ci] >= 0)) continue;
      if (i8 && im2col_of[c.data] == ci) continue;     // the stem form of the int8 conv
      if (!i8 && cv.shape[2] * cv.shape[3] == 1) continue;  // the dense-rows form keeps its own epilogue
      post_add[ci] = (int)ai;
      post_conv[ai] = ci;
      break;
    }
  }
}

// Bottleneck blocks: x -> 1x1 conv (+bias, act) -> 3x3 stride-1 pad-1 conv
// (+bias, act) -> 1x1 conv + bias + r (act) with r = x or r = a 1x1 conv of x
// without activation (the projection shortcut), each intermediate read only
// by the next conv, of a kind (mid width, channels of x, channels of the
// output) the fused kernel is compiled for, run as one launch (the
// intermediates stay in LDS)
// on bf16 activations always: with the small-tile variant (4 x 7 pixels, 4
// waves) offered to the autotune, measured on MI355X over ResNet-50 v1,
// fusing every stage-1 and stage-2 block made batch 1 12% faster (0.370 ->
// 0.324 ms), batches 2-8 4-13% faster and batches 16 and 32 faster than
// unfused.  On int8 codes (no small-tile variant) when the finest tiling
// gives at least one workgroup per CU (256).  BYOC_FUSE_BLOCK=0 keeps the
// three launches everywhere, =1 fuses every supported block.
void Planner::find_blocks() {
  block_mid.assign(g.nodes.size(), -1);
  block_proj.assign(g.nodes.size(), -1);
  in_block.assign(g.nodes.size(), false);
  const char* env = std::getenv("BYOC_FUSE_BLOCK");
  if (!(bf16 || i8) || (env && env[0] == '0')) return;
  const bool always = env && env[0] == '1';
  std::vector<int> uses(g.values.size(), 0);
  for (const Node& n : g.nodes) {
    for (int a : {n.data, n.residual, n.other})
      if (a >= 0) ++uses[a];
    if (n.op == OpKind::Concat)
      for (size_t k = 1; k < n.cat.size(); ++k) ++uses[n.cat[k]];
  }
  for (const IoDesc& o : g.outputs) uses[o.value] += 2;
  auto plain_conv = [&](const Node& n, int r, int pad, int stride) {
    // (the fused kernel applies none / ReLU / ReLU6 only)
    if (n.op != OpKind::Conv || n.depthwise || n.groups != 1 || n.act == Act::Gelu || n.act == Act::Leaky)
      return false;
    const auto& ws = g.values[n.weight].shape;
    return ws[2] == r && ws[3] == r && n.stride[0] == stride && n.stride[1] == stride && n.pad[0] == pad &&
           n.pad[1] == pad && n.pad[2] == pad && n.pad[3] == pad;
  };
  auto fused_elsewhere = [&](int ni) {
    return post_add[ni] >= 0 || post_conv[ni] >= 0 || stem_pool[ni] >= 0 || stem_conv[ni] >= 0;
  };
  for (size_t ci = 0; ci < g.nodes.size(); ++ci) {
    const Node& c = g.nodes[ci];
    if (!plain_conv(c, 1, 0, 1) || c.residual < 0 || fused_elsewhere((int)ci) || alias_of[c.out] >= 0) continue;
    const int m2 = c.data;
    // the residual: x itself, or the output of a projection conv of x (stride
    // 1 or 2, the stride of the block's first 1x1 then) read only here
    int x = c.residual, pi = -1, S = 1;
    const Value& rv = g.values[c.residual];
    if (rv.source == Value::Node) {
      const Node& pn = g.nodes[rv.index];
      for (int st : {1, 2})
        if (plain_conv(pn, 1, 0, st) && pn.residual < 0 && pn.act == Act::None && uses[c.residual] == 1 &&
            !fused_elsewhere(rv.index) && alias_of[c.residual] < 0) {
          pi = rv.index;
          x = pn.data;
          S = st;
        }
    }
    const Value& v2 = g.values[m2];
    if (v2.source != Value::Node || uses[m2] != 1) continue;
    const int bi = v2.index;
    const Node& b = g.nodes[bi];
    if (!plain_conv(b, 3, 1, 1) || b.residual >= 0 || fused_elsewhere(bi) || alias_of[m2] >= 0) continue;
    const int m1 = b.data;
    const Value& v1 = g.values[m1];
    if (v1.source != Value::Node || uses[m1] != 1) continue;
    const int ai = v1.index;
    const Node& a = g.nodes[ai];
    if (!plain_conv(a, 1, 0, S) || a.residual >= 0 || a.data != x || fused_elsewhere(ai) || alias_of[m1] >= 0)
      continue;
    const auto& xs = g.values[x].shape;
    const auto& s1 = g.values[m1].shape;
    const auto& ys = g.values[c.out].shape;
    if (xs.size() != 4 || s1.size() != 4 || ys.size() != 4 || ys[0] != xs[0] || ys[2] != s1[2] ||
        ys[3] != s1[3])
      continue;
    const int CIN = (int)xs[1], F = (int)s1[1], COUT = (int)ys[1];
    if ((pi < 0) != (COUT == CIN && S == 1) || bottleneck_variants(i8, F, CIN, COUT, S) <= 0) continue;
    // codes: the fused epilogue sums the rescaled terms unclamped, exact while
    // the residual's term stays below 2^19 (255 * its factor)
    if (i8 && !(g.values[c.residual].qscale / g.values[c.out].qscale < 2048.0)) continue;
    int most = 0;
    for (int v = 0; v < bottleneck_variants(i8, F, CIN, COUT, S); ++v)
      most = std::max(most, bottleneck_tiles(i8, F, CIN, COUT, S, v, (int)ys[0], (int)ys[2], (int)ys[3]));
    if (!always && i8 && most < 256) continue;
    if (xs[0] * xs[2] * xs[3] * std::max(CIN, COUT) * 2 >= (int64_t(1) << 31)) continue;
    block_mid[ci] = bi;
    block_proj[ci] = pi;
    in_block[ai] = in_block[bi] = true;
    if (pi >= 0) in_block[pi] = true;
  }
}

void Planner::plan_block(int ci) {
  const Node& c = g.nodes[ci];
  const Node& b = g.nodes[block_mid[ci]];
  const Node& a = g.nodes[g.values[b.data].index];
  const int x = a.data;
  const auto& xs = g.values[x].shape;
  Launch L;
  L.op = Launch::Bottleneck;
  L.info.kind = BYOC_K_CONV_MFMA;
  L.info.node = ci;
  L.x = loc[x];
  L.res = loc[x];
  L.y = loc[c.out];
  L.bnC = (int)xs[1];
  L.bnF = (int)g.values[a.out].shape[1];
  L.bnCout = (int)g.values[c.out].shape[1];
  L.bnS = a.stride[0];
  BottleneckParams& p = L.bn;
  const auto& ys = g.values[c.out].shape;
  p.N = (int)xs[0], p.H = (int)xs[2], p.W = (int)xs[3], p.P = (int)ys[2], p.Q = (int)ys[3];
  int64_t wbytes = 0;
  // packed weights and padded bias of one conv, as the implicit-GEMM kernel has them
  auto pack = [&](const Node& n, Ref* w, Ref* bias, int* ld, int* w_bytes, int* b_bytes) {
    const auto& ws = g.values[n.weight].shape;
    const int K = (int)ws[0], Cg = (int)ws[1], R = (int)ws[2], S = (int)ws[3];
    const int Cp = cp[n.data];
    const int rows = (int)rup(K, kRowPad);
    const int Kgp = (int)rup((int64_t)R * S * Cp, kKPad);
    const int wc = g.values[n.weight].index;
    const int bc = n.bias >= 0 ? g.values[n.bias].index : -1;
    *w = wslot((int64_t)rows * Kgp * 2);
    jobs.push_back({PackJob::ConvW, wc, w->off, K, Cg, R, S, Cp, Kgp, rows, 0, 0});
    *bias = wslot((int64_t)rows * 4);
    jobs.push_back({PackJob::Vec, bc, bias->off, 0, 0, 0, 0, 0, 0, 0, bc >= 0 ? K : 0, rows});
    *ld = Kgp;
    *w_bytes = rows * Kgp * 2;
    *b_bytes = rows * 4;
    wbytes += numel(ws) * 2 + (bc >= 0 ? K * 4 : 0);
  };
  pack(a, &L.w, &L.bias, &p.ld1, &p.w1_bytes, &p.b1_bytes);
  pack(b, &L.w2, &L.b2, &p.ld2, &p.w2_bytes, &p.b2_bytes);
  pack(c, &L.w3, &L.b3, &p.ld3, &p.w3_bytes, &p.b3_bytes);
  int64_t pmacs = 0;
  if (block_proj[ci] >= 0) {
    const Node& pn = g.nodes[block_proj[ci]];
    pack(pn, &L.wp, &L.bp, &p.ldp, &p.wp_bytes, &p.bp_bytes);
    pmacs = pn.macs;
  }
  p.x_bytes = (int)act_bytes(x);
  p.y_bytes = (int)act_bytes(c.out);
  p.act1 = (int)a.act, p.act2 = (int)b.act, p.act3 = (int)c.act;
  p.alpha1 = a.alpha, p.alpha2 = b.alpha, p.alpha3 = c.alpha;
  L.info.flops = 2 * (a.macs + b.macs + c.macs + pmacs);
  L.info.bytes = act_bytes(x) + act_bytes(c.out) + wbytes;
  // built-in variant 0; BYOC_BLOCK_VARIANT=<v> forces another
  int v = 0;
  if (const char* bv = std::getenv("BYOC_BLOCK_VARIANT")) v = std::atoi(bv);
  if (v < 0 || v >= bottleneck_variants(false, L.bnF, L.bnC, L.bnCout, L.bnS)) v = 0;
  L.tile = ConvTile{};
  L.tile.bnv = v;
  L.tile_default = L.tile;
  name(L, bottleneck_variant_name(false, L.bnF, L.bnC, L.bnCout, L.bnS, v));
  e->launches.push_back(L);
}

// MobileNetV2 inverted-residual blocks: [x -> 1x1 conv (+bias, act) ->]
// depthwise 3x3 pad 1 stride 1 or 2 (+bias, act) -> 1x1 conv (+bias, act)
// [+ x], each intermediate read only by the next composite, of channel
// counts the fused kernel is compiled for, run as one launch at any batch:
// measured on MI355X over MobileNetV2, fusing every block with at most 64
// input channels made batch 1 17% faster (0.239 -> 0.199 ms), batches 2-8
// 8-13% faster and batch 16 faster than fusing only the blocks with 256 or
// more tiles.  The wider blocks (96 and 160 input channels, expanded to
// 576 and 960) stay separate unless BYOC_FUSE_IR=1: their workgroups walk
// 9 or 15 slices of the expanded width one after the other (18-39 us per
// block at batch 1 and 16 against 14-19 us for the three launches).
// BYOC_FUSE_IR=0 keeps the separate launches everywhere.
void Planner::find_ir_blocks() {
  ir_dw.assign(g.nodes.size(), -1);
  ir_exp.assign(g.nodes.size(), -1);
  in_ir.assign(g.nodes.size(), false);
  const char* env = std::getenv("BYOC_FUSE_IR");
  if (!bf16 || (env && env[0] == '0')) return;
  const bool always = env && env[0] == '1';
  std::vector<int> uses(g.values.size(), 0);
  for (const Node& n : g.nodes) {
    for (int a : {n.data, n.residual, n.other})
      if (a >= 0) ++uses[a];
    if (n.op == OpKind::Concat)
      for (size_t k = 1; k < n.cat.size(); ++k) ++uses[n.cat[k]];
  }
  for (const IoDesc& o : g.outputs) uses[o.value] += 2;
  auto clamp_act = [](const Node& n) { return n.act != Act::Gelu && n.act != Act::Leaky; };
  auto conv1x1 = [&](const Node& n) {
    if (n.op != OpKind::Conv || n.depthwise || n.groups != 1 || !clamp_act(n)) return false;
    const auto& ws = g.values[n.weight].shape;
    return ws[2] == 1 && ws[3] == 1 && n.stride[0] == 1 && n.stride[1] == 1 && n.pad[0] == 0 && n.pad[1] == 0 &&
           n.pad[2] == 0 && n.pad[3] == 0;
  };
  auto elsewhere = [&](int ni) {
    return post_add[ni] >= 0 || post_conv[ni] >= 0 || stem_pool[ni] >= 0 || stem_conv[ni] >= 0 || in_block[ni] ||
           block_mid[ni] >= 0 || alias_of[g.nodes[ni].out] >= 0;
  };
  for (size_t ci = 0; ci < g.nodes.size(); ++ci) {
    const Node& c = g.nodes[ci];
    if (!conv1x1(c) || elsewhere((int)ci)) continue;
    const Value& vd = g.values[c.data];
    if (vd.source != Value::Node || uses[c.data] != 1) continue;
    const int di = vd.index;
    const Node& d = g.nodes[di];
    if (d.op != OpKind::Conv || !d.depthwise || !clamp_act(d) || d.residual >= 0 || elsewhere(di)) continue;
    const auto& dws = g.values[d.weight].shape;
    const int S = d.stride[0];
    if (dws[2] != 3 || dws[3] != 3 || d.stride[1] != S || (S != 1 && S != 2) || d.pad[0] != 1 || d.pad[1] != 1 ||
        d.pad[2] != 1 || d.pad[3] != 1)
      continue;
    // the expand conv, when the depthwise input is a 1x1 conv read only here
    int ai = -1, x = d.data;
    const Value& ve = g.values[d.data];
    if (ve.source == Value::Node && uses[d.data] == 1) {
      const int e = ve.index;
      const Node& a = g.nodes[e];
      if (conv1x1(a) && a.residual < 0 && !elsewhere(e)) {
        ai = e;
        x = a.data;
      }
    }
    const auto& xs = g.values[x].shape;
    const auto& es = g.values[d.data].shape;
    const auto& ys = g.values[c.out].shape;
    if (xs.size() != 4 || es.size() != 4 || ys.size() != 4) continue;
    const int CIN = (int)xs[1], F = (int)es[1], COUT = (int)ys[1];
    if (ai < 0 && F != CIN) continue;
    if (ai >= 0 && F == CIN) continue;  // (the kind is told apart by F != CIN)
    if (c.residual >= 0 && (c.residual != x || S != 1 || CIN != COUT)) continue;
    const int nv = ir_block_variants(CIN, F, COUT, S);
    if (nv <= 0 || (!always && CIN > 64)) continue;
    if (xs[0] * xs[2] * xs[3] * std::max(std::max(CIN, F), COUT) * 2 >= (int64_t(1) << 31)) continue;
    ir_dw[ci] = di;
    ir_exp[ci] = ai;
    in_ir[di] = true;
    if (ai >= 0) in_ir[ai] = true;
  }
}

void Planner::plan_ir(int ci) {
  const Node& c = g.nodes[ci];
  const Node& d = g.nodes[ir_dw[ci]];
  const int ai = ir_exp[ci];
  const int x = ai >= 0 ? g.nodes[ai].data : d.data;
  const auto& xs = g.values[x].shape;
  const auto& ys = g.values[c.out].shape;
  Launch L;
  L.op = Launch::IrBlock;
  L.info.kind = BYOC_K_CONV_MFMA;
  L.info.node = ci;
  L.x = loc[x];
  L.res = loc[x];
  L.y = loc[c.out];
  IrParams& p = L.ir;
  p.N = (int)xs[0], p.H = (int)xs[2], p.W = (int)xs[3], p.P = (int)ys[2], p.Q = (int)ys[3], p.S = d.stride[0];
  p.CIN = cp[x], p.F = cp[d.data], p.COUT = cp[c.out];
  int64_t wbytes = 0;
  // a 1x1 conv's packed weights and padded bias, as the implicit-GEMM kernel has them
  auto pack = [&](const Node& n, Ref* w, Ref* bias, int* ld, int* w_bytes, int* b_bytes) {
    const auto& ws = g.values[n.weight].shape;
    const int K = (int)ws[0], Cg = (int)ws[1];
    const int Cp = cp[n.data];
    const int rows = (int)rup(K, kRowPad);
    const int Kgp = (int)rup(Cp, kKPad);
    const int wc = g.values[n.weight].index;
    const int bc = n.bias >= 0 ? g.values[n.bias].index : -1;
    *w = wslot((int64_t)rows * Kgp * 2);
    jobs.push_back({PackJob::ConvW, wc, w->off, K, Cg, 1, 1, Cp, Kgp, rows, 0, 0});
    *bias = wslot((int64_t)rows * 4);
    jobs.push_back({PackJob::Vec, bc, bias->off, 0, 0, 0, 0, 0, 0, 0, bc >= 0 ? K : 0, rows});
    *ld = Kgp;
    *w_bytes = rows * Kgp * 2;
    *b_bytes = rows * 4;
    wbytes += numel(ws) * 2 + (bc >= 0 ? K * 4 : 0);
  };
  if (ai >= 0) {
    const Node& a = g.nodes[ai];
    pack(a, &L.w, &L.bias, &p.ldE, &p.we_bytes, &p.be_bytes);
    p.act_e = (int)a.act, p.alpha_e = a.alpha;
  }
  {  // the depthwise weights [9][F] (float32 values of the bf16 taps) and bias
    const int Cp = cp[d.data];
    const int K = (int)g.values[d.weight].shape[0];
    const int wc = g.values[d.weight].index;
    const int bc = d.bias >= 0 ? g.values[d.bias].index : -1;
    L.w2 = wslot((int64_t)9 * Cp * 4);
    jobs.push_back({PackJob::DwW32, wc, L.w2.off, K, 1, 3, 3, Cp, 0, 0, 0, 0});
    L.b2 = wslot(Cp * 4);
    jobs.push_back({PackJob::Vec, bc, L.b2.off, 0, 0, 0, 0, 0, 0, 0, bc >= 0 ? K : 0, Cp});
    p.wd_bytes = 9 * Cp * 4;
    p.bd_bytes = Cp * 4;
    p.act_d = (int)d.act, p.alpha_d = d.alpha;
    wbytes += numel(g.values[d.weight].shape) * 2 + (bc >= 0 ? K * 4 : 0);
  }
  pack(c, &L.w3, &L.b3, &p.ldP, &p.wp_bytes, &p.bp_bytes);
  p.act_p = (int)c.act, p.alpha_p = c.alpha;
  p.res = c.residual >= 0;
  p.x_bytes = (int)act_bytes(x);
  p.y_bytes = (int)act_bytes(c.out);
  L.info.flops = 2 * ((ai >= 0 ? g.nodes[ai].macs : 0) + d.macs + c.macs);
  L.info.bytes = act_bytes(x) + act_bytes(c.out) + wbytes;
  // built-in variant: the first with at least 256 tiles (else the finest);
  // BYOC_IR_VARIANT=<v> forces one
  const int nv = ir_block_variants(p.CIN, p.F, p.COUT, p.S);
  int v = nv - 1;
  for (int k = nv - 1; k >= 0; --k)
    if (ir_block_tiles(p.CIN, p.F, p.COUT, p.S, k, p.N, p.P, p.Q) >= 256) v = k;
  if (const char* ev = std::getenv("BYOC_IR_VARIANT")) v = std::atoi(ev);
  if (v < 0 || v >= nv) v = 0;
  L.tile = ConvTile{};
  L.tile.bnv = v;
  L.tile_default = L.tile;
  name(L, ir_block_name(p.CIN, p.F, p.COUT, p.S, v));
  e->launches.push_back(L);
}

// The int8 form of a fused block: the three (four) convs quantized on the
// host as the int8 conv kernel has them; each composite's output zero point
// and activation clamp, and the residual's rescaling into y's scale.
void Planner::plan_block_i8(int ci) {
  const Node& c = g.nodes[ci];
  const Node& b = g.nodes[block_mid[ci]];
  const Node& a = g.nodes[g.values[b.data].index];
  const int x = a.data;
  const auto& xs = g.values[x].shape;
  const std::string where = "node " + std::to_string(ci) + " (" + c.composite + ")";
  Launch L;
  L.op = Launch::Bottleneck;
  L.info.kind = BYOC_K_CONV_I8;
  L.info.node = ci;
  L.x = loc[x];
  L.res = loc[x];
  L.y = loc[c.out];
  L.bnI8 = true;
  L.bnC = (int)xs[1];
  L.bnF = (int)g.values[a.out].shape[1];
  L.bnCout = (int)g.values[c.out].shape[1];
  L.bnS = a.stride[0];
  BottleneckParams& p = L.bn;
  const auto& ys = g.values[c.out].shape;
  p.N = (int)xs[0], p.H = (int)xs[2], p.W = (int)xs[3], p.P = (int)ys[2], p.Q = (int)ys[3];
  // output zero point and activation clamp in codes (as the int8 conv has them)
  auto clamp_of = [&](const Node& n, int slot) {
    const Value& yv = g.values[n.out];
    int lo = -128, hi = 127;
    if (n.act == Act::Relu || n.act == Act::Relu6) lo = yv.qzero;
    if (n.act == Act::Relu6) {
      const double h = yv.qzero + std::nearbyint(6.0 / yv.qscale);
      hi = h < 127.0 ? (int)h : 127;
    }
    p.qz[slot] = yv.qzero, p.qlo[slot] = lo, p.qhi[slot] = hi;
  };
  int64_t wbytes = 0;
  auto pack = [&](const Node& n, Ref* w, Ref* bias, int* ld, int* w_bytes, int* b_bytes) {
    const auto& ws = g.values[n.weight].shape;
    const int K = (int)ws[0], R = (int)ws[2], S = (int)ws[3];
    const int Cp = cp[n.data];
    const int rows = (int)rup(K, kRowPad);
    const int Kgp = (int)rup((int64_t)R * S * Cp, 128);
    if ((int64_t)R * S * ws[1] * 255 * 127 >= (int64_t(1) << 30)) {
      err = Status::Err(BYOC_ERR_UNSUPPORTED, where + ": reduction too long for int32 accumulation");
      return;
    }
    std::vector<uint8_t> packed;
    std::vector<int32_t> qch, wtap;
    std::string why;
    if (!quantize_conv_i8(n, Cp, Kgp, rows, false, false, packed, qch, wtap, &why)) {
      err = Status::Err(BYOC_ERR_UNSUPPORTED, where + ": " + why);
      return;
    }
    *w = host_blob(std::move(packed));
    std::vector<uint8_t> qb(qch.size() * 4);
    std::memcpy(qb.data(), qch.data(), qb.size());
    *bias = host_blob(std::move(qb));
    *ld = Kgp;
    *w_bytes = rows * Kgp;
    *b_bytes = rows * 8;
    wbytes += numel(ws) + K * 8;
  };
  pack(a, &L.w, &L.bias, &p.ld1, &p.w1_bytes, &p.b1_bytes);
  pack(b, &L.w2, &L.b2, &p.ld2, &p.w2_bytes, &p.b2_bytes);
  pack(c, &L.w3, &L.b3, &p.ld3, &p.w3_bytes, &p.b3_bytes);
  clamp_of(a, 0);
  clamp_of(b, 1);
  clamp_of(c, 2);
  int64_t pmacs = 0;
  if (block_proj[ci] >= 0) {
    const Node& pn = g.nodes[block_proj[ci]];
    pack(pn, &L.wp, &L.bp, &p.ldp, &p.wp_bytes, &p.bp_bytes);
    clamp_of(pn, 3);
    pmacs = pn.macs;
  }
  if (!err.ok()) return;
  const Value& rv = g.values[c.residual];  // x, or the projection's output
  p.zr = rv.qzero;
  if (!rescale_factor(rv.qscale / g.values[c.out].qscale, &p.mr) || !(p.mr < 2048.f)) {
    err = Status::Err(BYOC_ERR_UNSUPPORTED, where + ": residual rescaling factor outside (0, 2048)");
    return;
  }
  p.x_bytes = (int)act_bytes(x);
  p.y_bytes = (int)act_bytes(c.out);
  L.info.flops = 2 * (a.macs + b.macs + c.macs + pmacs);
  L.info.bytes = act_bytes(x) + act_bytes(c.out) + wbytes;
  // built-in variant 0; BYOC_BLOCK_VARIANT=<v> forces another
  int v = 0;
  if (const char* bv = std::getenv("BYOC_BLOCK_VARIANT")) v = std::atoi(bv);
  if (v < 0 || v >= bottleneck_variants(true, L.bnF, L.bnC, L.bnCout, L.bnS)) v = 0;
  L.tile = ConvTile{};
  L.tile.bnv = v;
  L.tile_default = L.tile;
  name(L, bottleneck_variant_name(true, L.bnF, L.bnC, L.bnCout, L.bnS, v));
  e->launches.push_back(L);
}

Status Planner::plan() {
  if (i8) return plan_i8();
  find_stems();
  find_concat_aliases();
  find_post_adds();
  find_blocks();
  find_ir_blocks();
  // concatenation outputs are allocated first: their producers write into them
  for (const Node& n : g.nodes)
    if (n.op == OpKind::Concat) {
      cp[n.out] = (int)rup(g.values[n.out].shape[1], 8);
      loc[n.out] = arena(internal_bytes(n.out));
    }
  // ---- inputs: direct use or boundary transform ----------------------------
  for (size_t i = 0; i < g.inputs.size(); ++i) {
    const IoDesc& in = g.inputs[i];
    const int v = in.value;
    const auto& s = g.values[v].shape;
    cp[v] = bf16 ? (int)rup(s[1], 8) : (int)s[1];
    bool fused_stem = false;
    for (size_t ni = 0; ni < g.nodes.size(); ++ni)
      if (stem_pool[ni] >= 0 && g.nodes[ni].data == v) fused_stem = true;
    if (fused_stem) {  // read in place by the fused stem kernel
      loc[v] = io(Ref::Input, (int)i);
      continue;
    }
    const bool direct = bf16 ? (s.size() == 2 && in.dtype == DType::BF16 && s[1] % 8 == 0)
                             : (in.dtype == DType::F32);
    if (direct) {
      loc[v] = io(Ref::Input, (int)i);
      continue;
    }
    loc[v] = arena(internal_bytes(v));
    Launch L;
    L.info.kind = BYOC_K_TRANSFORM;
    L.info.node = -1;
    L.x = io(Ref::Input, (int)i);
    L.y = loc[v];
    L.src_bf16 = in.dtype == DType::BF16;
    L.info.bytes = ext_bytes(v, in.dtype) + act_bytes(v);
    if (!bf16) {
      L.op = Launch::Cast;
      L.dst_bf16 = false;
      L.n = numel(s);
      name(L, "cast_in");
    } else if (s.size() == 4) {
      L.op = Launch::NchwToNhwc;
      L.N = (int)s[0], L.C = (int)s[1], L.H = (int)s[2], L.W = (int)s[3], L.Cp = cp[v];
      name(L, "nchw_to_nhwc");
    } else {
      L.op = Launch::RowsToPadded;
      L.M = (int)s[0], L.K = (int)s[1], L.Kp = cp[v];
      name(L, "rows_to_padded");
    }
    e->launches.push_back(L);
  }
  // ---- nodes ---------------------------------------------------------------
  std::vector<bool> direct_out(g.outputs.size(), false);
  for (size_t ni = 0; ni < g.nodes.size(); ++ni) {
    const Node& n = g.nodes[ni];
    const int v = n.out;
    const auto& s = g.values[v].shape;
    cp[v] = bf16 ? (int)rup(s[1], 8) : (int)s[1];
    bool placed = false;
    for (size_t j = 0; j < g.outputs.size() && !placed; ++j) {
      const IoDesc& o = g.outputs[j];
      if (o.value != v || direct_out[j]) continue;
      const bool ok = bf16 ? (s.size() == 2 && o.dtype == DType::BF16 && s[1] % 8 == 0)
                           : (o.dtype == DType::F32);
      if (ok) {
        loc[v] = io(Ref::Output, (int)j);
        direct_out[j] = true;
        placed = true;
      }
    }
    if (stem_pool[ni] >= 0 || post_add[ni] >= 0 || in_block[ni] || in_ir[ni]) {  // planned with the node that consumes it
      loc[v] = Ref();
      continue;
    }
    if (n.op == OpKind::Concat) placed = true;  // allocated above
    if (!placed && alias_of[v] >= 0) {
      loc[v] = slice(alias_of[v], alias_off[v]);
      placed = true;
    }
    if (!placed) loc[v] = arena(internal_bytes(v));
    if (stem_conv[ni] >= 0)
      plan_stem(stem_conv[ni], (int)ni);
    else if (block_mid[ni] >= 0)
      plan_block((int)ni);
    else if (ir_dw[ni] >= 0)
      plan_ir((int)ni);
    else if (post_conv[ni] >= 0)
      plan_node(post_conv[ni]);
    else
      plan_node((int)ni);
    if (!err.ok()) return err;
  }
  // ---- outputs not written in place: boundary transforms ---------------------
  for (size_t j = 0; j < g.outputs.size(); ++j) {
    if (direct_out[j]) continue;
    const IoDesc& o = g.outputs[j];
    const int v = o.value;
    const auto& s = g.values[v].shape;
    Launch L;
    L.info.kind = BYOC_K_TRANSFORM;
    L.info.node = -1;
    L.x = loc[v];
    L.y = io(Ref::Output, (int)j);
    L.dst_bf16 = o.dtype == DType::BF16;
    L.info.bytes = act_bytes(v) + ext_bytes(v, o.dtype);
    const bool src_is_input = g.values[v].source == Value::Input && loc[v].kind == Ref::Input;
    if (!bf16) {
      L.op = Launch::Cast;
      L.src_bf16 = src_is_input ? g.inputs[g.values[v].index].dtype == DType::BF16 : false;
      L.n = numel(s);
      name(L, "cast_out");
    } else if (s.size() == 4) {
      L.op = Launch::NhwcToNchw;
      L.N = (int)s[0], L.C = (int)s[1], L.H = (int)s[2], L.W = (int)s[3], L.Cp = cp[v];
      name(L, "nhwc_to_nchw");
    } else {
      L.op = Launch::PaddedToRows;
      L.M = (int)s[0], L.K = (int)s[1], L.Kp = cp[v];
      name(L, "padded_to_rows");
    }
    e->launches.push_back(L);
  }
  return Status::Ok();
}

void Planner::plan_node(int ni) {
  const Node& n = g.nodes[ni];
  const auto& xs = g.values[n.data].shape;
  const auto& ys = g.values[n.out].shape;
  Launch L;
  L.info.node = ni;
  L.x = loc[n.data];
  L.y = loc[n.out];
  L.act = (int)n.act;
  L.alpha = n.alpha;
  if (n.residual >= 0) L.res = loc[n.residual];
  const int pa = post_add.empty() ? -1 : post_add[ni];  // add folded in after the activation
  if (pa >= 0) {
    const Node& a = g.nodes[pa];
    L.y = loc[a.out];
    L.res = loc[a.data == n.out ? a.other : a.data];
  }
  const int64_t ebytes = bf16 ? 2 : 4;

  if (n.op == OpKind::Conv || n.op == OpKind::Dense) {
    const auto& ws = g.values[n.weight].shape;
    const bool dense = n.op == OpKind::Dense;
    const int K = (int)ws[0];
    const int Cg = dense ? (int)ws[1] : (int)ws[1];
    const int R = dense ? 1 : (int)ws[2];
    const int S = dense ? 1 : (int)ws[3];
    const int N = (int)xs[0];
    const int C = (int)xs[1];
    const int H = dense ? 1 : (int)xs[2];
    const int W = dense ? 1 : (int)xs[3];
    const int P = dense ? 1 : (int)ys[2];
    const int Q = dense ? 1 : (int)ys[3];
    const int wc = g.values[n.weight].index;
    const int bc = n.bias >= 0 ? g.values[n.bias].index : -1;
    L.info.flops = 2 * n.macs;
    L.info.bytes = act_bytes(n.data) + numel(ws) * ebytes + (bc >= 0 ? K * 4 : 0) +
                   act_bytes(n.out) * (n.residual >= 0 || pa >= 0 ? 2 : 1);
    if (!bf16) {
      L.op = Launch::ConvF32;
      L.info.kind = BYOC_K_CONV_F32;
      ConvF32Params& p = L.cf;
      p.N = N, p.C = C, p.H = H, p.W = W, p.K = K, p.P = P, p.Q = Q, p.R = R, p.S = S;
      p.sh = n.stride[0], p.sw = n.stride[1], p.pt = n.pad[0], p.pl = n.pad[1];
      p.groups = n.groups, p.act = (int)n.act;
      p.alpha = n.alpha;
      L.w = wslot(numel(ws) * 4);
      jobs.push_back({PackJob::Copy, wc, L.w.off, 0, 0, 0, 0, 0, 0, 0, (int)numel(ws), (int)numel(ws)});
      if (bc >= 0) {
        L.bias = wslot(K * 4);
        jobs.push_back({PackJob::Vec, bc, L.bias.off, 0, 0, 0, 0, 0, 0, 0, K, K});
      }
      name(L, n.depthwise ? "conv_f32_depthwise" : "conv_f32_direct");
      e->launches.push_back(L);
      return;
    }
    const int Cp = cp[n.data];
    const int Kp = cp[n.out];
    if (n.depthwise) {
      L.op = Launch::Depthwise;
      L.info.kind = BYOC_K_DEPTHWISE;
      DwParams& p = L.dw;
      p.N = N, p.H = H, p.W = W, p.Cp = Cp, p.P = P, p.Q = Q, p.R = R, p.S = S;
      p.sh = n.stride[0], p.sw = n.stride[1], p.pt = n.pad[0], p.pl = n.pad[1], p.act = (int)n.act;
      p.alpha = n.alpha;
      L.w = wslot((int64_t)R * S * Cp * 2);
      jobs.push_back({PackJob::DwW, wc, L.w.off, K, 1, R, S, Cp, 0, 0, 0, 0});
      L.bias = wslot(Cp * 4);
      jobs.push_back({PackJob::Vec, bc, L.bias.off, 0, 0, 0, 0, 0, 0, 0, K, Cp});
      name(L, "depthwise_nhwc");
      e->launches.push_back(L);
      return;
    }
    ConvParams& p = L.conv;
    p.N = N, p.H = H, p.W = W, p.Cp = Cp, p.P = P, p.Q = Q, p.R = R, p.S = S;
    p.sh = n.stride[0], p.sw = n.stride[1], p.pt = n.pad[0], p.pl = n.pad[1];
    p.M = N * P * Q;
    p.Kp = Kp;
    p.Kg = R * S * Cp;
    p.Kgp = (int)rup(p.Kg, kKPad);
    p.ldy = alias_of[n.out] >= 0 ? cp[alias_of[n.out]] : Kp;
    p.ldr = Kp;
    p.act = (int)n.act;
    p.alpha = n.alpha;
    p.res_post = pa >= 0;
    const int rows = (int)rup(Kp, kRowPad);
    const int64_t xb = (int64_t)N * H * W * Cp * 2, wb = (int64_t)rows * p.Kgp * 2;
    if (xb >= (int64_t(1) << 31) || wb >= (int64_t(1) << 31)) {
      err = Status::Err(BYOC_ERR_UNSUPPORTED, "node " + std::to_string(ni) + " (" + n.composite +
                                                  "): input or packed weights of 2 GiB or more");
      return;
    }
    const int64_t rb = (int64_t)p.M * Kp * 2;
    if (rb >= (int64_t(1) << 31)) {
      err = Status::Err(BYOC_ERR_UNSUPPORTED, "node " + std::to_string(ni) + " (" + n.composite +
                                                  "): output of 2 GiB or more");
      return;
    }
    p.x_bytes = (int)xb;
    p.w_bytes = (int)wb;
    p.res_bytes = (int)rb;
    // index math divides by P*Q, Q, Cp and S with 40-bit reciprocals (exact
    // while dividend * divisor < 2^40)
    if ((int64_t)p.M * P * Q >= (int64_t(1) << 40) || (int64_t)p.Kg * Cp >= (int64_t(1) << 40)) {
      err = Status::Err(BYOC_ERR_UNSUPPORTED, "node " + std::to_string(ni) + " (" + n.composite +
                                                  "): too many output pixels for the index arithmetic");
      return;
    }
    p.mg_pq = magic40(P * Q);
    p.mg_q = magic40(Q);
    p.mg_cp = magic40(Cp);
    p.mg_s = magic40(S);
    L.w = wslot((int64_t)rows * p.Kgp * 2);
    jobs.push_back({PackJob::ConvW, wc, L.w.off, K, Cg, R, S, Cp, p.Kgp, rows, 0, 0});
    L.bias = wslot((int64_t)rows * 4);
    jobs.push_back({PackJob::Vec, bc, L.bias.off, 0, 0, 0, 0, 0, 0, 0, bc >= 0 ? K : 0, rows});
    // few rows of a plain matrix product (a classifier at small batch):
    // the dense-rows kernel, one workgroup per 16 output channels with the
    // reduction split over its waves; BYOC_DENSE_ROWS=0 (or a forced conv
    // tile) keeps the conv kernels
    const bool rows_gemm = R == 1 && S == 1 && H == 1 && W == 1 && P == 1 && Q == 1;
    const char* dr_env = std::getenv("BYOC_DENSE_ROWS");
    if (rows_gemm && p.M <= 64 && !std::getenv("BYOC_CONV_TILE") && !(dr_env && dr_env[0] == '0')) {
      p.splits = 1;
      p.k_tiles_per_split = p.Kgp / kKPad;
      if (dense_rows_supported(p)) {
        L.op = Launch::DenseRows;
        L.info.kind = BYOC_K_CONV_MFMA;
        char nm[32];
        std::snprintf(nm, sizeof(nm), "dense_rows_m%d", p.M);
        name(L, nm);
        e->launches.push_back(L);
        return;
      }
    }
    int splits, kps;
    choose_conv_tile(p.M, Kp, p.Kg, &L.tile, &splits, &kps);
    apply_tile_override(p.Kg, &L.tile, &splits, &kps);
    p.splits = splits;
    p.k_tiles_per_split = kps;
    {
      // 3x3 stride-1 convs with at least 256 input channels and enough
      // 128x64 tiles to fill most CUs run on the halo kernel (input window
      // staged in LDS once per 64-channel slice).  Measured on MI355X over
      // the ResNet-50 layers at batch 32: it wins on 256 channels at 14x14
      // (196 tiles) and loses where the patch is large against the work
      // (64 channels at 56x56), where the implicit-GEMM kernel's 128x128
      // tiles win (128 channels at 28x28) and where 128x64 tiles leave most
      // CUs idle (512 channels at 7x7, 104 tiles).  Where 128x64 tiles are
      // too few but 64x64 tiles are enough (512 channels at 7x7: 200 tiles)
      // it runs on 64x64 tiles.  BYOC_CONV_HALO=1 takes it wherever the
      // shape allows, =0 never; a forced tile decides alone.
      const bool forced = L.tile.halo == 2;
      const char* he = std::getenv("BYOC_CONV_HALO");
      const int64_t halo_tiles = ((p.M + 127) / 128) * ((Kp + 63) / 64);
      const int64_t halo64_tiles = ((p.M + 63) / 64) * ((Kp + 63) / 64);
      const bool by_rule = Cp >= 256 && halo_tiles >= 160;
      const bool by_rule64 = Cp >= 256 && !by_rule && halo64_tiles >= 160;
      const bool want =
          forced || (!std::getenv("BYOC_CONV_TILE") && (he ? he[0] == '1' : by_rule || by_rule64));
      const int ns = forced ? L.tile.stages : kHaloStages;
      const int hbm = forced ? L.tile.bm : by_rule64 ? 64 : 128;
      int lp = 0, npb = 0;
      if (forced) {  // a forced halo tile also forgoes split-K
        ConvParams q = p;
        q.splits = 1;
        if (L.tile.bn == 64 && conv_halo_plan(q, hbm, 64, ns, &lp, &npb)) {
          splits = 1;
          kps = (int)((p.Kg + kKPad - 1) / kKPad);
          p.splits = splits;
          p.k_tiles_per_split = kps;
        }
      }
      if (want && splits == 1 && conv_halo_plan(p, hbm, 64, ns, &lp, &npb)) {
        L.tile = ConvTile{};
        L.tile.bm = hbm;
        L.tile.bn = 64;
        L.tile.stages = ns;
        L.tile.threads = 512;
        L.tile.halo = 1;
        L.tile.lp = lp;
        L.tile.npb = npb;
      } else if (forced) {
        L.tile = ConvTile{};
        choose_conv_tile(p.M, Kp, p.Kg, &L.tile, &splits, &kps);
        p.splits = splits;
        p.k_tiles_per_split = kps;
      }
    }
    p.xcd_py = L.tile.stages > 0 ? choose_xcd_split(p, L.tile) : 0;
    L.tile_default = L.tile;
    L.op = Launch::ConvMfma;
    L.info.kind = BYOC_K_CONV_MFMA;
    name_conv(L);
    if (splits > 1) {
      L.partial = arena((int64_t)splits * p.M * Kp * 4);
      Launch Rd = L;
      Rd.op = Launch::SplitReduce;
      Rd.info.kind = BYOC_K_REDUCE;
      Rd.info.flops = 0;
      Rd.info.bytes = 0;
      name(Rd, "splitk_reduce");
      L.y = Ref();
      L.res = Ref();
      Ref keep_bias = L.bias;
      L.bias = Ref();
      e->launches.push_back(L);
      Rd.bias = keep_bias;
      Rd.x = Ref();
      Rd.w = Ref();
      e->launches.push_back(Rd);
    } else {
      e->launches.push_back(L);
    }
    return;
  }
  if (n.op == OpKind::Concat) {  // copies of the inputs not written in place
    const auto& cs = g.values[n.out].shape;
    int off = 0;
    for (int a : n.cat) {
      const int ca = (int)g.values[a].shape[1];
      if (alias_of[a] != n.out) {
        Launch C;
        C.op = Launch::CopyChannels;
        C.info.kind = BYOC_K_ADD;
        C.info.node = ni;
        C.x = loc[a];
        C.y = slice(n.out, off);
        C.M = (int)(cs[0] * cs[2] * cs[3]);
        C.C = ca;
        C.Cp = cp[a];
        C.Kp = cp[n.out];
        C.info.bytes = 2 * act_bytes(a);
        name(C, "concat_copy");
        e->launches.push_back(C);
      }
      off += ca;
    }
    return;
  }
  if (n.op == OpKind::MaxPool || n.op == OpKind::AvgPool || n.op == OpKind::AvgPoolWin) {
    PoolParams& p = L.pool;
    p.N = (int)xs[0], p.C = (int)xs[1], p.H = (int)xs[2], p.W = (int)xs[3], p.Cp = cp[n.data];
    p.R = n.pool[0], p.S = n.pool[1], p.sh = n.stride[0], p.sw = n.stride[1];
    p.pt = n.pad[0], p.pl = n.pad[1];
    p.P = n.op != OpKind::AvgPool ? (int)ys[2] : 1;
    p.Q = n.op != OpKind::AvgPool ? (int)ys[3] : 1;
    p.ldy = alias_of[n.out] >= 0 ? cp[alias_of[n.out]] : 0;
    L.info.bytes = act_bytes(n.data) + act_bytes(n.out);
    if (n.op == OpKind::AvgPoolWin) {
      L.op = Launch::AvgPoolWinBf16;
      L.info.kind = BYOC_K_AVGPOOL;
      L.count_include_pad = n.count_include_pad;
      name(L, "avgpool_win_nhwc");
    } else if (n.op == OpKind::MaxPool) {
      L.op = bf16 ? Launch::MaxPoolBf16 : Launch::MaxPoolF32;
      L.info.kind = BYOC_K_MAXPOOL;
      name(L, bf16 ? "maxpool_nhwc" : "maxpool_nchw_f32");
    } else {
      L.op = bf16 ? Launch::AvgPoolBf16 : Launch::AvgPoolF32;
      L.info.kind = BYOC_K_AVGPOOL;
      name(L, bf16 ? "avgpool_nhwc" : "avgpool_nchw_f32");
    }
    e->launches.push_back(L);
    return;
  }
  // Add
  L.op = bf16 ? Launch::AddBf16 : Launch::AddF32;
  L.info.kind = BYOC_K_ADD;
  L.other = loc[n.other];
  L.n = bf16 ? internal_bytes(n.out) / 2 : numel(ys);
  L.info.bytes = 3 * act_bytes(n.out);
  name(L, bf16 ? "add_bf16" : "add_f32");
  e->launches.push_back(L);
}

// ---- int8 graphs (partial quantization, Sec. 3.2, Fig. 4a) -----------------
// Inputs pass through a quantize node (fp32 arithmetic, NCHW -> NHWC codes
// with channels padded to 16), every composite runs on codes, outputs pass
// through a dequantize node.  Weights, biases and rescaling factors are
// quantized here on the host, in float64, and uploaded as built.
Status Planner::plan_i8() {
  auto dims = [&](int v, int* N, int* C, int* H, int* W) {
    const auto& s = g.values[v].shape;
    *N = (int)s[0];
    *C = (int)s[1];
    *H = s.size() == 4 ? (int)s[2] : 1;
    *W = s.size() == 4 ? (int)s[3] : 1;
  };
  // A few-channel image read only by one conv is quantized straight into that
  // conv's im2col rows (R*S taps of 4 channel codes per output pixel, padded
  // to 16): the conv becomes a 1x1 product over a reduction of R*S*4 instead
  // of R*S*16 (channels padded to 16), and out-of-image taps hold the zero
  // point, so the folded -Z_x * sum(w) of the bias is exact for every pixel.
  find_stems();
  std::vector<bool> stem_input(g.values.size(), false);  // read in place by a fused stem
  for (size_t ni = 0; ni < g.nodes.size(); ++ni)
    if (stem_pool[ni] >= 0) stem_input[g.nodes[ni].data] = true;
  im2col_of.assign(g.values.size(), -1);
  {
    std::vector<int> uses(g.values.size(), 0), reader(g.values.size(), -1);
    for (size_t ni = 0; ni < g.nodes.size(); ++ni) {
      const Node& n = g.nodes[ni];
      for (int a : {n.data, n.residual, n.other})
        if (a >= 0) ++uses[a], reader[a] = (int)ni;
    }
    for (const IoDesc& o : g.outputs) ++uses[o.value];
    for (const IoDesc& in : g.inputs) {
      const int v = in.value;
      const auto& s = g.values[v].shape;
      if (s.size() != 4 || s[1] > 4 || uses[v] != 1 || reader[v] < 0 || stem_input[v]) continue;
      const Node& n = g.nodes[reader[v]];
      if (n.op != OpKind::Conv || n.depthwise || n.data != v) continue;
      const auto& ws = g.values[n.weight].shape;
      const auto& ys = g.values[n.out].shape;
      const int64_t kc = rup(ws[2] * ws[3] * 4, 16);
      // (the staging kernel holds the R input rows of an output row in 48 KB of LDS)
      if (kc <= 512 && s[0] * ys[2] * ys[3] * kc < (int64_t(1) << 31) && ws[2] * s[3] * 4 <= 48 * 1024)
        im2col_of[v] = reader[v];
    }
  }
  for (size_t i = 0; i < g.inputs.size(); ++i) {
    const IoDesc& in = g.inputs[i];
    const int v = in.value;
    const Value& val = g.values[v];
    if (stem_input[v]) {
      loc[v] = io(Ref::Input, (int)i);
      continue;
    }
    if (im2col_of[v] >= 0) {
      const Node& n = g.nodes[im2col_of[v]];
      const auto& ws = g.values[n.weight].shape;
      const auto& ys = g.values[n.out].shape;
      Launch L;
      L.op = Launch::QuantizeIm2colI8;
      L.info.kind = BYOC_K_TRANSFORM;
      L.info.node = -1;
      L.x = io(Ref::Input, (int)i);
      L.src_bf16 = in.dtype == DType::BF16;
      PoolParams& q = L.pool;
      q.N = (int)val.shape[0], q.C = (int)val.shape[1], q.H = (int)val.shape[2], q.W = (int)val.shape[3];
      q.R = (int)ws[2], q.S = (int)ws[3], q.sh = n.stride[0], q.sw = n.stride[1], q.pt = n.pad[0], q.pl = n.pad[1];
      q.P = (int)ys[2], q.Q = (int)ys[3];
      q.Cp = (int)rup(q.R * q.S * 4, 16);
      cp[v] = q.Cp;
      loc[v] = arena((int64_t)q.N * q.P * q.Q * q.Cp);
      L.y = loc[v];
      L.qscale = (float)(1.0 / val.qscale);
      L.qzero = val.qzero;
      L.info.bytes = ext_bytes(v, in.dtype) + (int64_t)q.N * q.P * q.Q * q.Cp;
      name(L, "quantize_im2col_in");
      e->launches.push_back(L);
      continue;
    }
    cp[v] = (int)rup(val.shape[1], 16);
    loc[v] = arena(internal_bytes(v));
    Launch L;
    L.op = Launch::QuantizeI8;
    L.info.kind = BYOC_K_TRANSFORM;
    L.info.node = -1;
    L.x = io(Ref::Input, (int)i);
    L.y = loc[v];
    L.src_bf16 = in.dtype == DType::BF16;
    dims(v, &L.N, &L.C, &L.H, &L.W);
    L.Cp = cp[v];
    L.qscale = (float)(1.0 / val.qscale);
    L.qzero = val.qzero;
    L.info.bytes = ext_bytes(v, in.dtype) + act_bytes(v);
    name(L, "quantize_in");
    e->launches.push_back(L);
  }
  find_post_adds();
  alias_of.assign(g.values.size(), -1);  // (no concatenation aliases on codes)
  find_blocks();
  for (size_t ni = 0; ni < g.nodes.size(); ++ni) {
    const int v = g.nodes[ni].out;
    cp[v] = (int)rup(g.values[v].shape[1], 16);
    // planned at the add folded into it, with its block or with its stem's pool
    if (post_add[ni] >= 0 || in_block[ni] || stem_pool[ni] >= 0) {
      loc[v] = Ref();
      continue;
    }
    loc[v] = arena(internal_bytes(v));
    if (stem_conv[ni] >= 0)
      plan_stem_i8(stem_conv[ni], (int)ni);
    else if (block_mid[ni] >= 0)
      plan_block_i8((int)ni);
    else
      plan_node_i8(post_conv[ni] >= 0 ? post_conv[ni] : (int)ni);
    if (!err.ok()) return err;
  }
  for (size_t j = 0; j < g.outputs.size(); ++j) {
    const IoDesc& o = g.outputs[j];
    const int v = o.value;
    const Value& val = g.values[v];
    Launch L;
    L.op = Launch::DequantizeI8;
    L.info.kind = BYOC_K_TRANSFORM;
    L.info.node = -1;
    L.x = loc[v];
    L.y = io(Ref::Output, (int)j);
    L.dst_bf16 = o.dtype == DType::BF16;
    dims(v, &L.N, &L.C, &L.H, &L.W);
    L.Cp = cp[v];
    L.qscale = (float)val.qscale;
    L.qzero = val.qzero;
    L.info.bytes = act_bytes(v) + ext_bytes(v, o.dtype);
    name(L, "dequantize_out");
    e->launches.push_back(L);
  }
  return Status::Ok();
}

// Host quantization of a conv's (or dense's) weights - per output channel,
// symmetric, int8 - its bias (int32, with -Z_x times the channel's weight sum
// folded in) and the per-channel rescaling factors S_x S_w / S_y, as the int8
// implicit-GEMM kernel reads them: packed [rows][Kgp], column (r*S + s)*Cp + c
// (im2col rows: (r*S + s)*4 + c; row_ld > 0: r*row_ld + s*4 + c, the fused
// stem's cells); qch [rows][2] = {bias, factor bits}; with
// `border`, wtap [R*S][rows] the weight sums per tap (tap-major: the 8
// consecutive channels an epilogue thread finishes are 32 contiguous
// bytes of one tap).  False, with the reason
// in *err_msg, on a value outside the kernel's ranges.
bool Planner::quantize_conv_i8(const Node& n, int Cp, int Kgp, int rows, bool im2col, bool border,
                               std::vector<uint8_t>& packed, std::vector<int32_t>& qch, std::vector<int32_t>& wtap,
                               std::string* err_msg, int row_ld) {
  auto why = [&](const std::string& m) {
    *err_msg = m;
    return false;
  };
  const Value& xv = g.values[n.data];
  const Value& yv = g.values[n.out];
  const auto& ws = g.values[n.weight].shape;
  const bool dense = n.op == OpKind::Dense;
  const int K = (int)ws[0], Cg = (int)ws[1];
  const int R = dense ? 1 : (int)ws[2], S = dense ? 1 : (int)ws[3];
  const byoc_const& wcst = consts[g.values[n.weight].index];
  const bool wbf = wcst.dtype == BYOC_BF16;
  auto wget = [&](int64_t i) -> double {
    if (wbf) {
      const uint32_t b = (uint32_t)((const uint16_t*)wcst.data)[i] << 16;
      float f;
      std::memcpy(&f, &b, 4);
      return f;
    }
    return ((const float*)wcst.data)[i];
  };
  const byoc_const* bcst = n.bias >= 0 ? &consts[g.values[n.bias].index] : nullptr;
  auto bget = [&](int k) -> double {
    if (bcst->dtype == BYOC_BF16) {
      const uint32_t b = (uint32_t)((const uint16_t*)bcst->data)[k] << 16;
      float f;
      std::memcpy(&f, &b, 4);
      return f;
    }
    return ((const float*)bcst->data)[k];
  };
  const int RS = R * S;
  packed.assign((size_t)rows * Kgp, 0);
  qch.assign((size_t)rows * 2, 0);
  wtap.assign(border ? (size_t)rows * RS : 0, 0);
  const double sx = xv.qscale, sy = yv.qscale;
  for (int k = 0; k < K; ++k) {
    const int64_t base = (int64_t)k * Cg * RS;
    double amax = 0.0;
    for (int64_t i = 0; i < (int64_t)Cg * RS; ++i) amax = std::max(amax, std::fabs(wget(base + i)));
    const double sw = amax > 0.0 ? amax / 127.0 : 1.0;
    int64_t total = 0;
    for (int c = 0; c < Cg; ++c)
      for (int r = 0; r < R; ++r)
        for (int s2 = 0; s2 < S; ++s2) {
          double qv = std::nearbyint(wget(base + ((int64_t)c * R + r) * S + s2) / sw);
          qv = std::min(127.0, std::max(-127.0, qv));
          const int wq = (int)qv;
          const size_t col = row_ld > 0 ? (size_t)r * row_ld + s2 * 4 + c
                             : im2col ? (size_t)(r * S + s2) * 4 + c : (size_t)(r * S + s2) * Cp + c;
          packed[(size_t)k * Kgp + col] = (uint8_t)(int8_t)wq;
          total += wq;
          if (border) wtap[(size_t)(r * S + s2) * rows + k] += wq;
        }
    double bq = 0.0;
    if (bcst) {
      bq = std::nearbyint(bget(k) / (sx * sw));
      bq = std::min(2147483647.0, std::max(-2147483648.0, bq));
    }
    const int64_t beff = (int64_t)bq - (int64_t)xv.qzero * total;
    if (beff <= -(int64_t(1) << 30) || beff >= (int64_t(1) << 30))
      return why("quantized bias of channel " + std::to_string(k) + " outside +-2^30");
    float mk = 0.f;
    if (!rescale_factor((sx * sw) / sy, &mk))
      return why("rescaling factor of channel " + std::to_string(k) + " outside (0, 2^20)");
    qch[(size_t)k * 2 + 0] = (int32_t)beff;
    std::memcpy(&qch[(size_t)k * 2 + 1], &mk, 4);
  }
  return true;
}

void Planner::plan_node_i8(int ni) {
  const Node& n = g.nodes[ni];
  const Value& xv = g.values[n.data];
  const Value& yv = g.values[n.out];
  const auto& xs = xv.shape;
  const auto& ys = yv.shape;
  const std::string where = "node " + std::to_string(ni) + " (" + n.composite + ")";
  auto fail = [&](const std::string& m) { err = Status::Err(BYOC_ERR_UNSUPPORTED, where + ": " + m); };
  Launch L;
  L.info.node = ni;
  L.x = loc[n.data];
  L.y = loc[n.out];
  L.act = (int)n.act;
  // activation clamp in output codes (ReLU: v >= Z_y; ReLU6: v <= Z_y + rint(6 / S_y))
  int lo = -128, hi = 127;
  if (n.act == Act::Relu || n.act == Act::Relu6) lo = yv.qzero;
  if (n.act == Act::Relu6) {
    const double h = yv.qzero + std::nearbyint(6.0 / yv.qscale);
    hi = h < 127.0 ? (int)h : 127;
  }

  if (n.op == OpKind::Conv && n.depthwise) {
    // exact integer taps on the vector ALU; weights quantized per channel here
    const auto& ws = g.values[n.weight].shape;
    const int C = (int)ws[0], R = (int)ws[2], S = (int)ws[3];
    QDwParams& d = L.qd;
    d.N = (int)xs[0], d.H = (int)xs[2], d.W = (int)xs[3], d.Cp = cp[n.data], d.P = (int)ys[2], d.Q = (int)ys[3];
    d.R = R, d.S = S, d.sh = n.stride[0], d.sw = n.stride[1], d.pt = n.pad[0], d.pl = n.pad[1];
    if ((int64_t)R * S * 255 * 127 >= (int64_t(1) << 30)) return fail("window too large for int32 accumulation");
    const byoc_const& wcst = consts[g.values[n.weight].index];
    const byoc_const* bcst = n.bias >= 0 ? &consts[g.values[n.bias].index] : nullptr;
    auto fget = [](const byoc_const& cst, int64_t i) -> double {
      if (cst.dtype == BYOC_BF16) {
        const uint32_t b = (uint32_t)((const uint16_t*)cst.data)[i] << 16;
        float f;
        std::memcpy(&f, &b, 4);
        return f;
      }
      return ((const float*)cst.data)[i];
    };
    const int RS = R * S;
    std::vector<uint8_t> packed((size_t)RS * d.Cp, 0);
    std::vector<int32_t> qch((size_t)d.Cp * 2, 0);
    const double sx = xv.qscale, sy = yv.qscale;
    for (int k = 0; k < C; ++k) {
      double amax = 0.0;
      for (int t = 0; t < RS; ++t) amax = std::max(amax, std::fabs(fget(wcst, (int64_t)k * RS + t)));
      const double sw = amax > 0.0 ? amax / 127.0 : 1.0;
      for (int t = 0; t < RS; ++t) {
        const double qv = std::min(127.0, std::max(-127.0, std::nearbyint(fget(wcst, (int64_t)k * RS + t) / sw)));
        packed[(size_t)t * d.Cp + k] = (uint8_t)(int8_t)(int)qv;
      }
      double bq = 0.0;
      if (bcst) bq = std::min(2147483647.0, std::max(-2147483648.0, std::nearbyint(fget(*bcst, k) / (sx * sw))));
      if (bq <= -1073741824.0 || bq >= 1073741824.0)
        return fail("quantized bias of channel " + std::to_string(k) + " outside +-2^30");
      float mk = 0.f;
      if (!rescale_factor((sx * sw) / sy, &mk))
        return fail("rescaling factor of channel " + std::to_string(k) + " outside (0, 2^20)");
      qch[(size_t)k * 2] = (int32_t)bq;
      std::memcpy(&qch[(size_t)k * 2 + 1], &mk, 4);
    }
    L.w = host_blob(std::move(packed));
    std::vector<uint8_t> qb(qch.size() * 4);
    std::memcpy(qb.data(), qch.data(), qb.size());
    L.bias = host_blob(std::move(qb));
    d.zx = xv.qzero, d.zy = yv.qzero, d.lo = lo, d.hi = hi;
    d.leaky = n.act == Act::Leaky, d.slope = n.alpha;
    if (n.residual >= 0) {
      const Value& rv = g.values[n.residual];
      L.res = loc[n.residual];
      d.zr = rv.qzero;
      if (!rescale_factor(rv.qscale / sy, &d.mr)) return fail("residual rescaling factor outside (0, 2^20)");
    }
    L.op = Launch::DepthwiseI8;
    L.info.kind = BYOC_K_DEPTHWISE;
    L.info.flops = 2 * n.macs;
    L.info.bytes = numel(xs) + numel(ws) + numel(ys) * (n.residual >= 0 ? 2 : 1);
    name(L, "depthwise_nhwc_i8");
    e->launches.push_back(L);
    return;
  }
  if (n.op == OpKind::Conv || n.op == OpKind::Dense) {
    const bool dense = n.op == OpKind::Dense;
    const auto& ws = g.values[n.weight].shape;
    const int K = (int)ws[0], Cg = (int)ws[1];
    const int R = dense ? 1 : (int)ws[2], S = dense ? 1 : (int)ws[3];
    const int N = (int)xs[0], C = (int)xs[1];
    const int H = dense ? 1 : (int)xs[2], W = dense ? 1 : (int)xs[3];
    const int P = dense ? 1 : (int)ys[2], Q = dense ? 1 : (int)ys[3];
    const int Cp = cp[n.data], Kp = cp[n.out];
    // input as im2col rows: a 1x1 product over the P x Q image of R*S*C codes
    const bool im2col = !dense && im2col_of[n.data] == ni;
    QConvParams& q = L.qc;
    ConvParams& p = q.g;
    if (im2col) {
      p.N = N, p.H = P, p.W = Q, p.Cp = Cp, p.P = P, p.Q = Q, p.R = 1, p.S = 1;
      p.sh = 1, p.sw = 1, p.pt = 0, p.pl = 0;
    } else {
      p.N = N, p.H = H, p.W = W, p.Cp = Cp, p.P = P, p.Q = Q, p.R = R, p.S = S;
      p.sh = n.stride[0], p.sw = n.stride[1], p.pt = n.pad[0], p.pl = n.pad[1];
    }
    p.M = N * P * Q;
    p.Kp = Kp;
    p.Kg = p.R * p.S * Cp;
    p.Kgp = (int)rup(p.Kg, 128);
    p.ldy = Kp;
    p.ldr = Kp;
    p.act = (int)n.act;
    p.splits = 1;
    p.k_tiles_per_split = p.Kgp / 128;
    const int rows = (int)rup(Kp, kRowPad);
    const int64_t xb = (int64_t)N * p.H * p.W * Cp, wb = (int64_t)rows * p.Kgp, rb = (int64_t)p.M * Kp;
    if (xb >= (int64_t(1) << 31) || wb >= (int64_t(1) << 31) || rb >= (int64_t(1) << 31))
      return fail("an operand of 2 GiB or more");
    if ((int64_t)p.M * P * Q >= (int64_t(1) << 40) || (int64_t)p.Kg * Cp >= (int64_t(1) << 40))
      return fail("too many output pixels for the index arithmetic");
    // |sum of (x - Z_x) w| <= R S C 255 127 plus the folded bias (< 2^30) stays inside int32
    if ((int64_t)R * S * Cg * 255 * 127 >= (int64_t(1) << 30)) return fail("reduction too long for int32 accumulation");
    p.x_bytes = (int)xb;
    p.w_bytes = (int)wb;
    p.res_bytes = (int)rb;
    p.mg_pq = magic40(P * Q);
    p.mg_q = magic40(Q);
    p.mg_cp = magic40(Cp);
    p.mg_s = magic40(p.S);

    // host quantization of the weights (per output channel, symmetric),
    // the bias and the rescaling factors
    const bool border = !dense && !im2col && xv.qzero != 0 && (n.pad[0] | n.pad[1] | n.pad[2] | n.pad[3]) != 0;
    std::vector<uint8_t> packed;
    std::vector<int32_t> qch, wtap;
    std::string why;
    if (!quantize_conv_i8(n, Cp, p.Kgp, rows, im2col, border, packed, qch, wtap, &why)) return fail(why);
    const double sy = yv.qscale;
    L.w = host_blob(std::move(packed));
    std::vector<uint8_t> qb(qch.size() * 4);
    std::memcpy(qb.data(), qch.data(), qb.size());
    L.bias = host_blob(std::move(qb));
    if (border) {
      std::vector<uint8_t> tb(wtap.size() * 4);
      std::memcpy(tb.data(), wtap.data(), tb.size());
      L.other = host_blob(std::move(tb));
    }
    q.wtap_ld = rows;
    q.zx = xv.qzero;
    q.zy = yv.qzero;
    q.lo = lo;
    q.hi = hi;
    q.leaky = n.act == Act::Leaky;
    q.slope = n.alpha;
    if (n.residual >= 0) {
      const Value& rv = g.values[n.residual];
      L.res = loc[n.residual];
      q.zr = rv.qzero;
      if (!rescale_factor(rv.qscale / sy, &q.mr)) return fail("residual rescaling factor outside (0, 2^20)");
    }
    const int pa = post_add.empty() ? -1 : post_add[ni];
    if (pa >= 0) {  // the add that follows, folded in: it writes the add's output
      const Node& a = g.nodes[pa];
      const Value& ov = g.values[a.data == n.out ? a.other : a.data];
      const Value& av = g.values[a.out];
      L.y = loc[a.out];
      L.res = loc[a.data == n.out ? a.other : a.data];
      q.post = 1;
      q.pz = av.qzero;
      q.zr = ov.qzero;
      if (!rescale_factor(sy / av.qscale, &q.pm) || !rescale_factor(ov.qscale / av.qscale, &q.mr))
        return fail("rescaling factor of the folded add outside (0, 2^20)");
    }
    // tile: the largest with at least two workgroups per CU
    auto tiles = [&](int bm, int bn) { return ((int64_t)p.M + bm - 1) / bm * ((Kp + bn - 1) / bn); };
    ConvTile& t = L.tile;
    t = ConvTile{};
    t.stages = 3;
    if (tiles(128, 128) >= 512) t.bm = 128, t.bn = 128;
    else if (tiles(128, 64) >= 512) t.bm = 128, t.bn = 64;
    else if (p.M <= 32) t.bm = 32, t.bn = 64;
    else t.bm = 64, t.bn = 64;
    // BYOC_I8_TILE=<bm>x<bn>s<stages>[w<waves>[k<groups>]] forces a tile (any
    // tile gives the same codes)
    if (const char* te = std::getenv("BYOC_I8_TILE")) {
      int bm = 0, bn = 0, ns = 0, nw = 4, kgr = 1;
      if (std::sscanf(te, "%dx%ds%dw%dk%d", &bm, &bn, &ns, &nw, &kgr) >= 3 &&
          conv_i8_tile_supported(bm, bn, ns, 64 * nw, kgr))
        t.bm = bm, t.bn = bn, t.stages = ns, t.threads = 64 * nw, t.kgroups = kgr;
    }
    // 3x3 stride-1 convs with at least 256 input channels and enough 128x64
    // tiles run on the windowed kernel (input window staged in LDS once per
    // 128-channel slice; the same codes), the rule of the bf16 convs, on
    // 64x64 tiles where only those fill the chip; BYOC_CONV_HALO=1 takes it
    // wherever the shape allows, =0 never.
    {
      // BYOC_I8_TILE=h<stages>[b<pixels>] forces it with that weight ring
      // depth (and tile height, 128 or 64).
      const char* he = std::getenv("BYOC_CONV_HALO");
      const char* te = std::getenv("BYOC_I8_TILE");
      const int64_t halo_tiles = ((int64_t)(p.M + 127) / 128) * ((Kp + 63) / 64);
      const int64_t halo64_tiles = ((int64_t)(p.M + 63) / 64) * ((Kp + 63) / 64);
      const bool r128 = Cp >= 256 && halo_tiles >= 160;
      const bool r64 = Cp >= 256 && !r128 && halo64_tiles >= 160;
      int ns = kHaloStages, hbm = r64 ? 64 : 128;
      bool want = he ? he[0] == '1' : (r128 || r64);
      if (te) {
        hbm = 128;
        want = te[0] == 'h' && std::sscanf(te + 1, "%db%d", &ns, &hbm) >= 1;
      }
      int lp = 0, npb = 0;
      if (!im2col && want && conv_halo_plan(p, hbm, 64, ns, &lp, &npb, true)) {
        t = ConvTile{};
        t.bm = hbm, t.bn = 64, t.stages = ns, t.threads = 512;
        t.halo = 1, t.lp = lp, t.npb = npb;
      }
    }
    p.xcd_py = choose_xcd_split(p, t);
    L.tile_default = t;
    L.op = Launch::ConvI8;
    L.info.kind = BYOC_K_CONV_I8;
    L.info.flops = 2 * n.macs;
    L.info.bytes = numel(xs) + numel(ws) + numel(ys) * (n.residual >= 0 ? 2 : 1);
    name_conv_i8(L);
    e->launches.push_back(L);
    return;
  }
  if (n.op == OpKind::MaxPool || n.op == OpKind::AvgPool) {
    PoolParams& p = L.pool;
    p.N = (int)xs[0], p.C = (int)xs[1], p.H = (int)xs[2], p.W = (int)xs[3], p.Cp = cp[n.data];
    p.R = n.pool[0], p.S = n.pool[1], p.sh = n.stride[0], p.sw = n.stride[1];
    p.pt = n.pad[0], p.pl = n.pad[1];
    p.P = n.op == OpKind::MaxPool ? (int)ys[2] : 1;
    p.Q = n.op == OpKind::MaxPool ? (int)ys[3] : 1;
    L.info.bytes = act_bytes(n.data) + act_bytes(n.out);
    if (n.op == OpKind::MaxPool) {
      L.op = Launch::MaxPoolI8;
      L.info.kind = BYOC_K_MAXPOOL;
      name(L, "maxpool_nhwc_i8");
    } else {
      if ((int64_t)p.H * p.W * 256 >= (int64_t(1) << 31)) return fail("image too large for the int32 pool sum");
      L.op = Launch::AvgPoolI8;
      L.info.kind = BYOC_K_AVGPOOL;
      L.qzx = xv.qzero;
      L.qzy = yv.qzero;
      if (!rescale_factor(xv.qscale / (yv.qscale * p.H * p.W), &L.qm))
        return fail("rescaling factor outside (0, 2^20)");
      name(L, "avgpool_nhwc_i8");
    }
    e->launches.push_back(L);
    return;
  }
  // Add
  const Value& bv = g.values[n.other];
  QAddParams& a = L.qa;
  a.n = internal_bytes(n.out);
  a.za = xv.qzero;
  a.zb = bv.qzero;
  a.zy = yv.qzero;
  a.lo = lo;
  a.hi = hi;
  a.leaky = n.act == Act::Leaky;
  a.slope = n.alpha;
  if (!rescale_factor(xv.qscale / yv.qscale, &a.ma) || !rescale_factor(bv.qscale / yv.qscale, &a.mb))
    return fail("rescaling factor outside (0, 2^20)");
  L.op = Launch::AddI8;
  L.info.kind = BYOC_K_ADD;
  L.other = loc[n.other];
  L.info.bytes = 3 * act_bytes(n.out);
  name(L, "add_i8");
  e->launches.push_back(L);
}

// First-fit offset allocator over the arena with coalescing frees.
struct OffsetAlloc {
  std::vector<std::pair<int64_t, int64_t>> free_;  // (offset, size), sorted by offset
  int64_t hwm = 0;
  int64_t alloc(int64_t size) {
    for (size_t i = 0; i < free_.size(); ++i) {
      if (free_[i].second >= size) {
        int64_t off = free_[i].first;
        free_[i].first += size;
        free_[i].second -= size;
        if (free_[i].second == 0) free_.erase(free_.begin() + i);
        return off;
      }
    }
    // extend: merge with a trailing free block that ends at hwm
    if (!free_.empty() && free_.back().first + free_.back().second == hwm) {
      int64_t off = free_.back().first;
      hwm = off + size;
      free_.pop_back();
      return off;
    }
    int64_t off = hwm;
    hwm += size;
    return off;
  }
  void release(int64_t off, int64_t size) {
    auto it = std::lower_bound(free_.begin(), free_.end(), std::make_pair(off, (int64_t)0));
    it = free_.insert(it, {off, size});
    size_t i = it - free_.begin();
    if (i + 1 < free_.size() && free_[i].first + free_[i].second == free_[i + 1].first) {
      free_[i].second += free_[i + 1].second;
      free_.erase(free_.begin() + i + 1);
    }
    if (i > 0 && free_[i - 1].first + free_[i - 1].second == free_[i].first) {
      free_[i - 1].second += free_[i].second;
      free_.erase(free_.begin() + i);
    }
  }
};

void layout_arena(Engine* e) {
  auto touch = [&](const Ref& r, int li) {
    if (r.kind != Ref::Arena) return;
    ArenaBuf& b = e->bufs[r.idx];
    b.first = std::min(b.first, li);
    b.last = std::max(b.last, li);
  };
  for (size_t i = 0; i < e->launches.size(); ++i) {
    const Launch& L = e->launches[i];
    for (const Ref* r : {&L.x, &L.w, &L.bias, &L.res, &L.y, &L.partial, &L.other}) touch(*r, (int)i);
  }
  OffsetAlloc a;
  for (size_t i = 0; i < e->launches.size(); ++i) {
    for (auto& b : e->bufs)
      if (b.first == (int)i && b.off < 0) b.off = a.alloc(b.bytes);
    for (auto& b : e->bufs)
      if (b.last == (int)i && b.off >= 0) a.release(b.off, b.bytes);
  }
  for (auto& b : e->bufs)
    if (b.off < 0) b.off = a.alloc(b.bytes);  // unused buffer: give it space anyway
  e->arena_bytes = a.hwm;
}

struct RunCtx {
  const Engine* e;
  const void* const* in;
  void* const* out;
  hipStream_t s;
  char* arena = nullptr;  // base of the intermediates (nullptr: the engine's own arena)
  void* ptr(const Ref& r) const {
    switch (r.kind) {
      case Ref::Arena: return (arena ? arena : e->arena) + e->bufs[r.idx].off + r.off;
      case Ref::Input: return const_cast<void*>(in[r.idx]);
      case Ref::Output: return out[r.idx];
      case Ref::Weights: return e->weights + r.off;
      default: return nullptr;
    }
  }
};

hipError_t exec(const Launch& L, const RunCtx& c) {
  switch (L.op) {
    case Launch::ConvMfma:
    case Launch::SplitReduce: {
      ConvParams p = L.conv;
      p.x = (const bf16_t*)c.ptr(L.x);
      p.w = (const bf16_t*)c.ptr(L.w);
      p.bias = (const float*)c.ptr(L.bias);
      p.res = (const bf16_t*)c.ptr(L.res);
      p.y = (bf16_t*)c.ptr(L.y);
      p.partial = (float*)c.ptr(L.partial);
      if (L.op == Launch::SplitReduce) return launch_splitk_reduce(p, c.s);
      if (L.tile.halo) return launch_conv_halo(p, L.tile.bm, L.tile.bn, L.tile.stages, L.tile.lp, L.tile.npb, c.s);
      return L.tile.stages > 0
                 ? launch_conv_dma(p, L.tile.bm, L.tile.bn, L.tile.stages, L.tile.threads, L.tile.kgroups, c.s)
                               : launch_conv_mfma(p, L.tile, c.s);
    }
    case Launch::DenseRows: {
      ConvParams p = L.conv;
      p.x = (const bf16_t*)c.ptr(L.x);
      p.w = (const bf16_t*)c.ptr(L.w);
      p.bias = (const float*)c.ptr(L.bias);
      p.res = (const bf16_t*)c.ptr(L.res);
      p.y = (bf16_t*)c.ptr(L.y);
      p.partial = nullptr;
      return launch_dense_rows(p, c.s);
    }
    case Launch::ConvF32: {
      ConvF32Params p = L.cf;
      p.x = (const float*)c.ptr(L.x);
      p.w = (const float*)c.ptr(L.w);
      p.bias = (const float*)c.ptr(L.bias);
      p.res = (const float*)c.ptr(L.res);
      p.y = (float*)c.ptr(L.y);
      return launch_conv_f32(p, c.s);
    }
    case Launch::Depthwise: {
      DwParams p = L.dw;
      p.x = (const bf16_t*)c.ptr(L.x);
      p.w = (const bf16_t*)c.ptr(L.w);
      p.bias = (const float*)c.ptr(L.bias);
      p.res = (const bf16_t*)c.ptr(L.res);
      p.y = (bf16_t*)c.ptr(L.y);
      return launch_depthwise(p, c.s);
    }
    case Launch::AvgPoolWinBf16: {
      PoolParams p = L.pool;
      p.x = c.ptr(L.x);
      p.y = c.ptr(L.y);
      return launch_avgpool_win_nhwc_bf16(p, L.count_include_pad, c.s);
    }
    case Launch::CopyChannels:
      return launch_copy_channels_bf16((const bf16_t*)c.ptr(L.x), L.Cp, (bf16_t*)c.ptr(L.y), L.Kp, L.M, L.C, c.s);
    case Launch::MaxPoolBf16:
    case Launch::AvgPoolBf16:
    case Launch::MaxPoolF32:
    case Launch::AvgPoolF32: {
      PoolParams p = L.pool;
      p.x = c.ptr(L.x);
      p.y = c.ptr(L.y);
      if (L.op == Launch::MaxPoolBf16) return launch_maxpool_nhwc_bf16(p, c.s);
      if (L.op == Launch::AvgPoolBf16) return launch_avgpool_nhwc_bf16(p, c.s);
      if (L.op == Launch::MaxPoolF32) return launch_maxpool_nchw_f32(p, c.s);
      return launch_avgpool_nchw_f32(p, c.s);
    }
    case Launch::AddBf16:
      return launch_add_bf16((const bf16_t*)c.ptr(L.x), (const bf16_t*)c.ptr(L.other),
                             (bf16_t*)c.ptr(L.y), L.n, L.act, L.alpha, c.s);
    case Launch::AddF32:
      return launch_add_f32((const float*)c.ptr(L.x), (const float*)c.ptr(L.other),
                            (float*)c.ptr(L.y), L.n, L.act, L.alpha, c.s);
    case Launch::NchwToNhwc:
      return launch_nchw_to_nhwc(c.ptr(L.x), L.src_bf16, (bf16_t*)c.ptr(L.y), L.N, L.C, L.H, L.W,
                                 L.Cp, c.s);
    case Launch::NhwcToNchw:
      return launch_nhwc_to_nchw((const bf16_t*)c.ptr(L.x), c.ptr(L.y), L.dst_bf16, L.N, L.C, L.H,
                                 L.W, L.Cp, c.s);
    case Launch::RowsToPadded:
      return launch_rows_to_padded(c.ptr(L.x), L.src_bf16, (bf16_t*)c.ptr(L.y), L.M, L.K, L.Kp,
                                   c.s);
    case Launch::PaddedToRows:
      return launch_padded_to_rows((const bf16_t*)c.ptr(L.x), c.ptr(L.y), L.dst_bf16, L.M, L.K,
                                   L.Kp, c.s);
    case Launch::Cast:
      return launch_cast(c.ptr(L.x), L.src_bf16, c.ptr(L.y), L.dst_bf16, L.n, c.s);
    case Launch::ConvI8: {
      QConvParams q = L.qc;
      q.g.x = (const bf16_t*)c.ptr(L.x);
      q.g.w = (const bf16_t*)c.ptr(L.w);
      q.g.res = (const bf16_t*)c.ptr(L.res);
      q.g.y = (bf16_t*)c.ptr(L.y);
      q.qch = (const int32_t*)c.ptr(L.bias);
      q.wtap = (const int32_t*)c.ptr(L.other);
      if (L.tile.halo) return launch_conv_halo_i8(q, L.tile.bm, L.tile.bn, L.tile.stages, L.tile.lp, L.tile.npb, c.s);
      return launch_conv_i8(q, L.tile.bm, L.tile.bn, L.tile.stages, L.tile.threads, L.tile.kgroups, c.s);
    }
    case Launch::MaxPoolI8:
    case Launch::AvgPoolI8: {
      PoolParams p = L.pool;
      p.x = c.ptr(L.x);
      p.y = c.ptr(L.y);
      if (L.op == Launch::MaxPoolI8) return launch_maxpool_nhwc_i8(p, c.s);
      return launch_avgpool_nhwc_i8(p, L.qzx, L.qzy, L.qm, c.s);
    }
    case Launch::AddI8: {
      QAddParams a = L.qa;
      a.a = (const int8_t*)c.ptr(L.x);
      a.b = (const int8_t*)c.ptr(L.other);
      a.y = (int8_t*)c.ptr(L.y);
      return launch_add_i8(a, c.s);
    }
    case Launch::Bottleneck: {
      BottleneckParams p = L.bn;
      p.x = c.ptr(L.x);
      p.y = c.ptr(L.y);
      p.w1 = c.ptr(L.w);
      p.w2 = c.ptr(L.w2);
      p.w3 = c.ptr(L.w3);
      p.b1 = c.ptr(L.bias);
      p.b2 = c.ptr(L.b2);
      p.b3 = c.ptr(L.b3);
      p.wp = c.ptr(L.wp);
      p.bp = c.ptr(L.bp);
      return launch_bottleneck(p, L.bnI8, L.bnF, L.bnC, L.bnCout, L.bnS, L.tile.bnv, c.s);
    }
    case Launch::IrBlock: {
      IrParams p = L.ir;
      p.x = c.ptr(L.x);
      p.y = c.ptr(L.y);
      p.we = c.ptr(L.w);
      p.be = c.ptr(L.bias);
      p.wd = c.ptr(L.w2);
      p.bd = c.ptr(L.b2);
      p.wp = c.ptr(L.w3);
      p.bp = c.ptr(L.b3);
      return launch_ir_block(p, L.tile.bnv, c.s);
    }
    case Launch::DepthwiseI8: {
      QDwParams d = L.qd;
      d.x = (const int8_t*)c.ptr(L.x);
      d.w = (const int8_t*)c.ptr(L.w);
      d.qch = (const int32_t*)c.ptr(L.bias);
      d.res = (const int8_t*)c.ptr(L.res);
      d.y = (int8_t*)c.ptr(L.y);
      return launch_depthwise_i8(d, c.s);
    }
    case Launch::QuantizeIm2colI8:
      return launch_quantize_im2col_i8(c.ptr(L.x), L.src_bf16, (int8_t*)c.ptr(L.y), L.pool, L.qscale, L.qzero, c.s);
    case Launch::QuantizeI8:
      return launch_quantize_i8(c.ptr(L.x), L.src_bf16, (int8_t*)c.ptr(L.y), L.N, L.C, L.H, L.W, L.Cp, L.qscale,
                                L.qzero, c.s);
    case Launch::DequantizeI8:
      return launch_dequantize_i8((const int8_t*)c.ptr(L.x), c.ptr(L.y), L.dst_bf16, L.N, L.C, L.H, L.W, L.Cp,
                                  L.qscale, L.qzero, c.s);
    case Launch::StemConvPool: {
      StemParams p = L.stem;
      p.x = c.ptr(L.x);
      p.w = c.ptr(L.w);
      p.bias = c.ptr(L.bias);
      p.y = c.ptr(L.y);
      return launch_stem_conv_maxpool(p, c.s);
    }
  }
  return hipErrorInvalidValue;
}

void release(Engine* e) {
  if (!e) return;
  if (e->done) (void)hipEventDestroy(e->done);
  e->done = nullptr;
  for (hipEvent_t ev : e->lev)
    if (ev) (void)hipEventDestroy(ev);
  e->lev.clear();
  if (e->fork_ev) (void)hipEventDestroy(e->fork_ev);
  if (e->join_ev) (void)hipEventDestroy(e->join_ev);
  e->fork_ev = e->join_ev = nullptr;
  if (e->side) (void)hipStreamDestroy(e->side);
  e->side = nullptr;
  e->two_streams = false;
  if (e->gexec) (void)hipGraphExecDestroy(e->gexec);
  e->gexec = nullptr;
  for (hipEvent_t ev : e->events) (void)hipEventDestroy(ev);
  e->events.clear();
  if (e->arena) (void)hipFree(e->arena);
  if (e->weights) (void)hipFree(e->weights);
  e->arena = nullptr;
  e->weights = nullptr;
}

struct DeviceGuard {
  int prev = -1;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) (void)hipSetDevice(dev);
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

Status build_device_state(Engine* e, Planner& pl, const byoc_const* consts) {
  HIP_TRY(hipSetDevice(e->device), "hipSetDevice");
  layout_arena(e);
  e->weight_bytes = pl.wbytes;
  if (e->weight_bytes > 0) HIP_TRY(hipMalloc(&e->weights, e->weight_bytes), "weights hipMalloc");
  if (e->arena_bytes > 0) HIP_TRY(hipMalloc(&e->arena, e->arena_bytes), "arena hipMalloc");
  // Stage every constant used by a pack job, then pack on the device.
  std::vector<int64_t> stage_off(pl.g.const_values.size(), -1);
  int64_t stage_bytes = 0;
  for (const PackJob& j : pl.jobs) {
    if (j.cidx < 0 || stage_off[j.cidx] >= 0) continue;
    const Value& v = pl.g.values[pl.g.const_values[j.cidx]];
    stage_off[j.cidx] = stage_bytes;
    stage_bytes += rup(numel(v.shape) * (v.dtype == DType::BF16 ? 2 : 4), 256);
  }
  char* stage = nullptr;
  if (stage_bytes > 0) HIP_TRY(hipMalloc(&stage, stage_bytes), "staging hipMalloc");
  Status st;
  for (size_t ci = 0; ci < stage_off.size() && st.ok(); ++ci) {
    if (stage_off[ci] < 0) continue;
    const Value& v = pl.g.values[pl.g.const_values[ci]];
    const int64_t bytes = numel(v.shape) * (v.dtype == DType::BF16 ? 2 : 4);
    hipError_t err = hipMemcpy(stage + stage_off[ci], consts[ci].data, bytes, hipMemcpyHostToDevice);
    if (err != hipSuccess) st = Status::Err(BYOC_ERR_DEVICE, std::string("constant upload: ") + hipGetErrorString(err));
  }
  for (const PackJob& j : pl.jobs) {
    if (!st.ok()) break;
    hipError_t err = hipSuccess;
    char* dst = e->weights + j.dst;
    if (j.kind == PackJob::Host) {
      const auto& b = pl.blobs[j.n];
      err = hipMemcpy(dst, b.data(), b.size(), hipMemcpyHostToDevice);
    } else if (j.cidx < 0) {
      err = hipMemsetAsync(dst, 0, (size_t)j.n_out * 4, nullptr);
    } else {
      const Value& v = pl.g.values[pl.g.const_values[j.cidx]];
      const bool sb = v.dtype == DType::BF16;
      const void* src = stage + stage_off[j.cidx];
      switch (j.kind) {
        case PackJob::ConvW:
          err = launch_pack_conv_weights(src, sb, (bf16_t*)dst, j.K, j.Cg, j.R, j.S, j.Cp, j.Kgp,
                                         j.rows, nullptr);
          break;
        case PackJob::DwW:
          err = launch_pack_dw_weights(src, sb, (bf16_t*)dst, j.K, j.R, j.S, j.Cp, nullptr);
          break;
        case PackJob::DwW32:
          err = launch_pack_dw_weights_f32(src, sb, (float*)dst, j.K, j.R, j.S, j.Cp, nullptr);
          break;
        case PackJob::Vec:
          err = launch_pack_vector_f32(src, sb, (float*)dst, j.n, j.n_out, nullptr);
          break;
        case PackJob::Copy:
          err = launch_cast(src, sb, dst, false, j.n, nullptr);
          break;
        case PackJob::StemW:
          err = launch_pack_stem_weights(src, sb, (bf16_t*)dst, j.Cg, j.R, j.S, j.n, nullptr);
          break;
      }
    }
    if (err != hipSuccess) st = Status::Err(BYOC_ERR_DEVICE, std::string("constant packing: ") + hipGetErrorString(err));
  }
  hipError_t serr = hipDeviceSynchronize();
  if (stage) (void)hipFree(stage);
  if (st.ok() && serr != hipSuccess)
    st = Status::Err(BYOC_ERR_DEVICE, std::string("constant packing: ") + hipGetErrorString(serr));
  return st;
}

// Memory a launch reads and writes, for the dependencies of two-stream
// execution: an arena buffer by its byte range (arena reuse makes a later
// buffer overlap an earlier one), a caller input or output as a whole.
// Packed weights are read-only and need no order.
struct Span {
  int space;  // 0 arena, 1 + i input i, (1 << 20) + j output j
  int64_t lo, hi;
};

bool span_of(const Engine* e, const Ref& r, Span* s) {
  switch (r.kind) {
    case Ref::Arena: {
      const ArenaBuf& b = e->bufs[r.idx];
      *s = Span{0, b.off, b.off + b.bytes};
      return true;
    }
    case Ref::Input: *s = Span{1 + r.idx, 0, 1}; return true;
    case Ref::Output: *s = Span{(1 << 20) + r.idx, 0, 1}; return true;
    default: return false;
  }
}

bool overlap(const std::vector<Span>& a, const std::vector<Span>& b) {
  for (const Span& x : a)
    for (const Span& y : b)
      if (x.space == y.space && x.lo < y.hi && y.lo < x.hi) return true;
  return false;
}

// Assigns every launch to the caller's stream or the side stream: a launch
// that does not depend on the launch before it (a branch, such as the
// projection shortcut of a ResNet block next to its 1x1 -> 3x3 path) goes to
// the other stream, so the two can run at once; any other launch stays on
// its predecessor's stream.  A launch that depends on an earlier one on the
// other stream waits for the event recorded after the latest such launch
// (read-after-write, write-after-read and write-after-write on any byte,
// arena reuse included).  Opt-in (BYOC_STREAMS=2): measured on MI355X,
// ResNet-50 bs32 took 0.807 ms per step with it against 0.743 ms on one
// stream, batch 1 0.453 against 0.370 ms and Inception V3 bs32 1.52
// against 1.34 ms - kernels of two queues running at once slow each other
// more than the overlap gains.
Status plan_streams(Engine* e) {
  const size_t n = e->launches.size();
  e->lstream.assign(n, 0);
  e->lrecord.assign(n, 0);
  e->lwait.assign(n, -1);
  e->two_streams = false;
  const char* env = std::getenv("BYOC_STREAMS");
  if (n < 2 || !(env && env[0] == '2')) return Status::Ok();
  std::vector<std::vector<Span>> rd(n), wr(n);
  for (size_t i = 0; i < n; ++i) {
    const Launch& L = e->launches[i];
    Span sp;
    for (const Ref* r : {&L.x, &L.w, &L.bias, &L.res, &L.other})
      if (span_of(e, *r, &sp)) rd[i].push_back(sp);
    if (span_of(e, L.partial, &sp)) {
      rd[i].push_back(sp);
      wr[i].push_back(sp);
    }
    if (span_of(e, L.y, &sp)) wr[i].push_back(sp);
  }
  auto dep = [&](size_t i, size_t j) {  // launch j (> i) must follow launch i
    return overlap(wr[i], rd[j]) || overlap(wr[i], wr[j]) || overlap(rd[i], wr[j]);
  };
  bool side_used = false;
  int waited[2] = {-1, -1};  // latest event each stream already waits for
  for (size_t j = 1; j < n; ++j) {
    e->lstream[j] = dep(j - 1, j) ? e->lstream[j - 1] : (int8_t)(1 - e->lstream[j - 1]);
    side_used |= e->lstream[j] == 1;
    int w = -1;
    for (size_t i = j; i-- > 0;)
      if (e->lstream[i] != e->lstream[j] && dep(i, j)) {
        w = (int)i;
        break;
      }
    const int sj = e->lstream[j];
    if (w >= 0 && w > waited[sj]) {
      e->lwait[j] = w;
      e->lrecord[w] = 1;
      waited[sj] = w;
    }
  }
  if (!side_used) return Status::Ok();
  HIP_TRY(hipStreamCreateWithFlags(&e->side, hipStreamNonBlocking), "side stream");
  // both streams are on the engine's device: device-scope events (no
  // system-scope release, which would write back the L2 at every record)
  const unsigned evf = hipEventDisableTiming | hipEventDisableSystemFence;
  HIP_TRY(hipEventCreateWithFlags(&e->fork_ev, evf), "hipEventCreate");
  HIP_TRY(hipEventCreateWithFlags(&e->join_ev, evf), "hipEventCreate");
  e->lev.assign(n, nullptr);
  for (size_t i = 0; i < n; ++i)
    if (e->lrecord[i]) HIP_TRY(hipEventCreateWithFlags(&e->lev[i], evf), "hipEventCreate");
  e->two_streams = true;
  return Status::Ok();
}

}  // namespace

Status engine_create(Graph&& g, const byoc_const* consts, int32_t n_consts, int device,
                     Engine** out) {
  (void)n_consts;
  *out = nullptr;
  if (device < 0) return Status::Err(BYOC_ERR_INVALID_ARG, "device " + std::to_string(device) + " out of range");
  Engine* e = new Engine();
  e->graph = std::move(g);
  e->device = device;
  // The launch plan is host work: planning errors are reported before any
  // device call (also on a host without a GPU).
  Planner pl(e, e->graph);
  pl.consts = consts;
  Status st = pl.plan();
  if (st.ok()) {
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev == 0)
      st = Status::Err(BYOC_ERR_DEVICE, "no HIP device available");
    else if (device >= ndev)
      st = Status::Err(BYOC_ERR_INVALID_ARG, "device " + std::to_string(device) + " out of range");
  }
  if (st.ok()) {
    DeviceGuard guard(device);
    st = build_device_state(e, pl, consts);
    if (st.ok()) {
      hipError_t err = hipEventCreateWithFlags(&e->done, hipEventDisableTiming | hipEventDisableSystemFence);
      if (err != hipSuccess) st = Status::Err(BYOC_ERR_DEVICE, std::string("hipEventCreate: ") + hipGetErrorString(err));
    }
    if (st.ok()) st = plan_streams(e);
  }
  if (!st.ok()) {
    release(e);
    delete e;
    return st;
  }
  *out = e;
  return Status::Ok();
}

namespace {

void drop_graph(Engine* e) {
  if (e->gexec) (void)hipGraphExecDestroy(e->gexec);
  e->gexec = nullptr;
  e->g_in.clear();
  e->g_out.clear();
  e->g_stream = nullptr;
}

Status launch_all(Engine* e, const RunCtx& c, bool prof);

// Replays the recorded graph when stream and I/O pointers match the
// recording, otherwise records the launch sequence anew.
Status run_graph(Engine* e, const RunCtx& c, int32_t n_in, int32_t n_out) {
  const bool same = e->gexec && e->g_stream == c.s &&
                    std::equal(e->g_in.begin(), e->g_in.end(), c.in) &&
                    std::equal(e->g_out.begin(), e->g_out.end(), c.out) &&
                    (int32_t)e->g_in.size() == n_in && (int32_t)e->g_out.size() == n_out;
  if (!same) {
    drop_graph(e);
    HIP_TRY(hipStreamBeginCapture(c.s, hipStreamCaptureModeThreadLocal), "hipStreamBeginCapture");
    Status lst = launch_all(e, c, false);
    hipGraph_t graph = nullptr;
    hipError_t cerr = hipStreamEndCapture(c.s, &graph);
    if (!lst.ok() || cerr != hipSuccess) {
      if (graph) (void)hipGraphDestroy(graph);
      if (!lst.ok()) return Status::Err(lst.code, lst.msg + " (during graph capture)");
      return Status::Err(BYOC_ERR_DEVICE, std::string("hipStreamEndCapture: ") + hipGetErrorString(cerr));
    }
    hipError_t ierr = hipGraphInstantiate(&e->gexec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    if (ierr != hipSuccess) {
      e->gexec = nullptr;
      return Status::Err(BYOC_ERR_DEVICE, std::string("hipGraphInstantiate: ") + hipGetErrorString(ierr));
    }
    e->g_stream = c.s;
    e->g_in.assign(c.in, c.in + n_in);
    e->g_out.assign(c.out, c.out + n_out);
  }
  HIP_TRY(hipGraphLaunch(e->gexec, c.s), "hipGraphLaunch");
  return Status::Ok();
}

}  // namespace

namespace {

// Result-identical kernel variants of one conv launch: every variant keeps
// the 16x16x32 MFMA and the reduction order of the built-in choice, so only
// the speed differs.  Split-K launches keep their plan.
std::vector<ConvTile> conv_candidates(const Launch& L) {
  std::vector<ConvTile> c;
  c.push_back(L.tile_default);
  if (L.tile_default.halo) {  // the halo kernel: other tiles and weight ring depths (same reduction order)
    for (int bm : {128, 64})
      for (int ns : {2, 3, 4, 6, 8}) {
        ConvTile t = L.tile_default;
        if ((bm == t.bm && ns == t.stages) || !conv_halo_plan(L.conv, bm, t.bn, ns, &t.lp, &t.npb)) continue;
        t.bm = bm;
        t.stages = ns;
        c.push_back(t);
      }
    return c;
  }
  if (L.conv.splits > 1 || L.tile_default.mf != 16) return c;
  const ConvParams& p = L.conv;
  const int kgr = L.tile_default.kgroups;  // the reduction order class of the built-in choice
  const int bms[] = {32, 64, 128, 256}, bns[] = {64, 128, 256};
  for (int nt : {256, 512})
    for (int bm : bms)
      for (int bn : bns) {
        if (bm == 32 && p.M >= 48) continue;
        // large tiles only where they still give the CUs a useful share of
        // tiles (wide GEMMs with few rows, such as a transformer FFN, have
        // many column tiles)
        if (bm >= 128 && ((int64_t)(p.M + bm - 1) / bm) * ((p.Kp + bn - 1) / bn) < 96) continue;
        if (bn >= 128 && p.Kp < bn) continue;
        for (int ns = 1; ns <= 4; ++ns) {
          const int threads = nt * kgr;
          if (kgr > 1 && nt != 256) continue;
          if (!conv_dma_tile_supported(bm, bn, ns, threads, kgr)) continue;
          ConvTile t;
          t.bm = bm;
          t.bn = bn;
          t.mf = 16;
          t.stages = ns;
          t.threads = threads;
          t.kgroups = kgr;
          if (t.bm == L.tile_default.bm && t.bn == L.tile_default.bn && t.stages == L.tile_default.stages &&
              t.threads == L.tile_default.threads)
            continue;  // the built-in choice is candidate 0 already
          c.push_back(t);
        }
      }
  if (kgr == 1 && L.tile_default.stages > 0) {  // the register-staged kernel as well
    ConvTile t;
    t.bm = L.conv.M >= 48 ? 64 : 32;
    t.bn = 64;
    c.push_back(t);
  }
  return c;
}

// int8 convs: every tile and ring depth (the integer sums, hence the
// codes, do not depend on the tiling)
std::vector<ConvTile> conv_i8_candidates(const Launch& L) {
  std::vector<ConvTile> c{L.tile_default};
  // the windowed 3x3 kernel, both tiles, every weight ring depth (int32
  // sums: every variant gives the same codes)
  for (int bm : {128, 64})
    for (int ns : {2, 3, 4, 6, 8}) {
      ConvTile t = ConvTile{};
      t.bm = bm, t.bn = 64, t.stages = ns, t.threads = 512, t.halo = 1;
      if (!conv_halo_plan(L.qc.g, bm, 64, ns, &t.lp, &t.npb, true)) continue;
      if (L.tile_default.halo && bm == L.tile_default.bm && ns == L.tile_default.stages) continue;
      c.push_back(t);
    }
  // single-group tiles of 4 or 8 waves, and 2 or 4 reduction groups of 4
  // waves (long reductions over few tiles)
  for (int nt : {256, 512, 1024})
    for (int kgr : {1, 2, 4})
      for (auto bmn : {std::pair<int, int>{128, 128}, {128, 64}, {64, 128}, {64, 64}, {32, 64}})
        for (int ns : {2, 3, 4}) {
          ConvTile t = ConvTile{};
          t.bm = bmn.first;
          t.bn = bmn.second;
          t.stages = ns;
          t.threads = nt;
          t.kgroups = kgr;
          if (!conv_i8_tile_supported(t.bm, t.bn, t.stages, t.threads, t.kgroups)) continue;
          if (t.bm == L.tile_default.bm && t.bn == L.tile_default.bn && t.stages == L.tile_default.stages &&
              t.threads == L.tile_default.threads && t.kgroups == L.tile_default.kgroups && !L.tile_default.halo)
            continue;
          c.push_back(t);
        }
  return c;
}

// fused bottleneck blocks: every tile variant of the block's (F, CIN) pair
// (one summation order for all of them)
std::vector<ConvTile> block_candidates(const Launch& L) {
  std::vector<ConvTile> c{L.tile_default};
  for (int v = 0; v < bottleneck_variants(L.bnI8, L.bnF, L.bnC, L.bnCout, L.bnS); ++v) {
    if (v == L.tile_default.bnv) continue;
    ConvTile t = L.tile_default;
    t.bnv = v;
    c.push_back(t);
  }
  return c;
}

// fused inverted-residual blocks: every variant of the kind (one summation
// order for all of them)
std::vector<ConvTile> ir_candidates(const Launch& L) {
  std::vector<ConvTile> c{L.tile_default};
  const IrParams& p = L.ir;
  for (int v = 0; v < ir_block_variants(p.CIN, p.F, p.COUT, p.S); ++v) {
    if (v == L.tile_default.bnv) continue;
    ConvTile t = L.tile_default;
    t.bnv = v;
    c.push_back(t);
  }
  return c;
}

bool tunable(const Launch& L) {
  return L.op == Launch::ConvMfma || L.op == Launch::ConvI8 || L.op == Launch::Bottleneck || L.op == Launch::IrBlock;
}

void apply_tile(Launch& L, const ConvTile& t) {
  L.tile = t;
  if (L.op == Launch::Bottleneck) {
    std::snprintf(L.info.name, sizeof(L.info.name), "%s",
                  bottleneck_variant_name(L.bnI8, L.bnF, L.bnC, L.bnCout, L.bnS, t.bnv));
    return;
  }
  if (L.op == Launch::IrBlock) {
    std::snprintf(L.info.name, sizeof(L.info.name), "%s", ir_block_name(L.ir.CIN, L.ir.F, L.ir.COUT, L.ir.S, t.bnv));
    return;
  }
  if (L.op == Launch::ConvI8) {
    L.qc.g.xcd_py = choose_xcd_split(L.qc.g, t);
    name_conv_i8(L);
    return;
  }
  L.conv.xcd_py = t.stages > 0 ? choose_xcd_split(L.conv, t) : 0;
  name_conv(L);
}

struct DevBuf {
  void* p = nullptr;
  ~DevBuf() {
    if (p) (void)hipFree(p);
  }
};

Status autotune(Engine* e) {
  const Graph& g = e->graph;
  std::vector<DevBuf> ins(g.inputs.size()), outs(g.outputs.size());
  std::vector<const void*> in_ptr(g.inputs.size());
  std::vector<void*> out_ptr(g.outputs.size());
  for (size_t i = 0; i < g.inputs.size(); ++i) {
    const IoDesc& io = g.inputs[i];
    const int64_t bytes = numel(g.values[io.value].shape) * (io.dtype == DType::BF16 ? 2 : 4);
    HIP_TRY(hipMalloc(&ins[i].p, (size_t)std::max<int64_t>(bytes, 16)), "autotune hipMalloc");
    HIP_TRY(hipMemset(ins[i].p, 0, (size_t)std::max<int64_t>(bytes, 16)), "autotune hipMemset");
    in_ptr[i] = ins[i].p;
  }
  for (size_t i = 0; i < g.outputs.size(); ++i) {
    const IoDesc& io = g.outputs[i];
    const int64_t bytes = numel(g.values[io.value].shape) * (io.dtype == DType::BF16 ? 2 : 4);
    HIP_TRY(hipMalloc(&outs[i].p, (size_t)std::max<int64_t>(bytes, 16)), "autotune hipMalloc");
    out_ptr[i] = outs[i].p;
  }
  hipStream_t s = nullptr;
  HIP_TRY(hipStreamCreate(&s), "autotune hipStreamCreate");
  const size_t nl = e->launches.size();
  std::vector<hipEvent_t> ev(nl + 1, nullptr);
  hipError_t err = hipSuccess;
  // no system-scope fence per event: timing only, the stream orders the work
  for (size_t i = 0; i <= nl && err == hipSuccess; ++i) err = hipEventCreateWithFlags(&ev[i], hipEventDisableSystemFence);
  RunCtx c{e, in_ptr.data(), out_ptr.data(), s};
  // Candidate k of every conv launch is timed inside full runs of the whole
  // launch sequence (each launch between its real neighbours, so with the
  // cache state the run leaves it), best of kReps runs; round k uses each
  // launch's k-th candidate (its built-in choice when it has fewer).
  std::vector<std::vector<ConvTile>> cand(nl);
  size_t rounds = 1;
  for (size_t i = 0; i < nl; ++i)
    if (tunable(e->launches[i])) {
      const Launch& L = e->launches[i];
      cand[i] = L.op == Launch::ConvI8       ? conv_i8_candidates(L)
                : L.op == Launch::Bottleneck ? block_candidates(L)
                : L.op == Launch::IrBlock    ? ir_candidates(L)
                                             : conv_candidates(L);
      rounds = std::max(rounds, cand[i].size());
    }
  std::vector<float> best_ms(nl, 0.f);
  std::vector<size_t> best_k(nl, 0);
  constexpr int kReps = 3;
  for (size_t k = 0; k < rounds && err == hipSuccess; ++k) {
    for (size_t i = 0; i < nl; ++i)
      if (!cand[i].empty()) apply_tile(e->launches[i], cand[i][k < cand[i].size() ? k : 0]);
    std::vector<float> round_ms(nl, 0.f);
    for (int rep = -1; rep < kReps && err == hipSuccess; ++rep) {  // rep -1: warm-up run
      err = hipEventRecord(ev[0], s);
      for (size_t i = 0; i < nl && err == hipSuccess; ++i) {
        err = exec(e->launches[i], c);
        if (err == hipSuccess) err = hipEventRecord(ev[i + 1], s);
      }
      if (err == hipSuccess) err = hipEventSynchronize(ev[nl]);
      for (size_t i = 0; i < nl && err == hipSuccess && rep >= 0; ++i) {
        float ms = 0.f;
        err = hipEventElapsedTime(&ms, ev[i], ev[i + 1]);
        if (rep == 0 || ms < round_ms[i]) round_ms[i] = ms;
      }
    }
    for (size_t i = 0; i < nl && err == hipSuccess; ++i)
      if (k < cand[i].size() && (k == 0 || round_ms[i] < best_ms[i])) {
        best_ms[i] = round_ms[i];
        best_k[i] = k;
      }
  }
  for (size_t i = 0; i < nl; ++i)
    if (!cand[i].empty()) apply_tile(e->launches[i], err == hipSuccess ? cand[i][best_k[i]] : e->launches[i].tile_default);
  for (hipEvent_t x : ev)
    if (x) (void)hipEventDestroy(x);
  hipError_t serr = hipStreamSynchronize(s);
  (void)hipStreamDestroy(s);
  if (err == hipSuccess) err = serr;
  if (err != hipSuccess) {
    for (Launch& L : e->launches)
      if (tunable(L)) apply_tile(L, L.tile_default);
    return Status::Err(BYOC_ERR_DEVICE, std::string("autotune: ") + hipGetErrorString(err));
  }
  return Status::Ok();
}

}  // namespace

Status engine_set_options(Engine* e, int flags) {
  if (flags & ~(BYOC_OPT_GRAPH_REPLAY | BYOC_OPT_AUTOTUNE))
    return Status::Err(BYOC_ERR_INVALID_ARG, "unknown option bits " + std::to_string(flags));
  DeviceGuard guard(e->device);
  const bool tune_on = (flags & BYOC_OPT_AUTOTUNE) && !(e->options & BYOC_OPT_AUTOTUNE);
  const bool tune_off = !(flags & BYOC_OPT_AUTOTUNE) && (e->options & BYOC_OPT_AUTOTUNE);
  if (!(flags & BYOC_OPT_GRAPH_REPLAY) || tune_on || tune_off) drop_graph(e);
  if (tune_on) {
    Status st = autotune(e);
    if (!st.ok()) return st;
  }
  if (tune_off)
    for (Launch& L : e->launches)
      if (tunable(L)) apply_tile(L, L.tile_default);
  e->options = flags;
  return Status::Ok();
}

namespace {

Status check_run_args(const Engine* e, const void* const* inputs, int32_t n_in, void* const* outputs,
                      int32_t n_out) {
  if (n_in != (int32_t)e->graph.inputs.size())
    return Status::Err(BYOC_ERR_INVALID_ARG, "expected " + std::to_string(e->graph.inputs.size()) +
                                                 " inputs, got " + std::to_string(n_in));
  if (n_out != (int32_t)e->graph.outputs.size())
    return Status::Err(BYOC_ERR_INVALID_ARG, "expected " + std::to_string(e->graph.outputs.size()) +
                                                 " outputs, got " + std::to_string(n_out));
  if (n_in > 0 && !inputs) return Status::Err(BYOC_ERR_INVALID_ARG, "inputs is NULL");
  if (!outputs) return Status::Err(BYOC_ERR_INVALID_ARG, "outputs is NULL");
  for (int i = 0; i < n_in; ++i)
    if (!inputs[i]) return Status::Err(BYOC_ERR_INVALID_ARG, "input " + std::to_string(i) + " is NULL");
  for (int i = 0; i < n_out; ++i)
    if (!outputs[i]) return Status::Err(BYOC_ERR_INVALID_ARG, "output " + std::to_string(i) + " is NULL");
  return Status::Ok();
}

// The launch sequence on the caller's stream and the side stream: the side
// stream first waits for the caller's stream (work enqueued before the
// run), cross-stream dependencies wait on recorded events, and the
// caller's stream finally waits for the side stream, so the run completes
// on the caller's stream (also as a captured graph: fork and join edges).
Status launch_two_streams(Engine* e, const RunCtx& c) {
  const size_t nl = e->launches.size();
  HIP_TRY(hipEventRecord(e->fork_ev, c.s), "hipEventRecord");
  HIP_TRY(hipStreamWaitEvent(e->side, e->fork_ev, 0), "hipStreamWaitEvent");
  RunCtx cs[2] = {c, c};
  cs[1].s = e->side;
  for (size_t i = 0; i < nl; ++i) {
    const int st = e->lstream[i];
    if (e->lwait[i] >= 0) HIP_TRY(hipStreamWaitEvent(cs[st].s, e->lev[e->lwait[i]], 0), "hipStreamWaitEvent");
    hipError_t err = exec(e->launches[i], cs[st]);
    if (err != hipSuccess)
      return Status::Err(BYOC_ERR_DEVICE, std::string("launch ") + std::to_string(i) + " (" +
                                              e->launches[i].info.name + "): " + hipGetErrorString(err));
    if (e->lrecord[i]) HIP_TRY(hipEventRecord(e->lev[i], cs[st].s), "hipEventRecord");
  }
  HIP_TRY(hipEventRecord(e->join_ev, e->side), "hipEventRecord");
  HIP_TRY(hipStreamWaitEvent(c.s, e->join_ev, 0), "hipStreamWaitEvent");
  return Status::Ok();
}

Status launch_all(Engine* e, const RunCtx& c, bool prof) {
  if (e->two_streams && !prof && c.arena == nullptr) return launch_two_streams(e, c);
  hipStream_t stream = c.s;
  const size_t nl = e->launches.size();
  hipEvent_t* ev = prof ? &e->events[(size_t)e->prof_runs * (nl + 1)] : nullptr;
  if (prof) HIP_TRY(hipEventRecord(ev[0], stream), "hipEventRecord");
  for (size_t i = 0; i < nl; ++i) {
    hipError_t err = exec(e->launches[i], c);
    if (err != hipSuccess)
      return Status::Err(BYOC_ERR_DEVICE, std::string("launch ") + std::to_string(i) + " (" +
                                              e->launches[i].info.name + "): " + hipGetErrorString(err));
    if (prof) HIP_TRY(hipEventRecord(ev[i + 1], stream), "hipEventRecord");
  }
  if (prof) {
    e->prof_runs++;
    e->prof_last_stream = stream;
  }
  return Status::Ok();
}

}  // namespace

Status engine_run(Engine* e, const void* const* inputs, int32_t n_in, void* const* outputs,
                  int32_t n_out, hipStream_t stream) {
  Status ast = check_run_args(e, inputs, n_in, outputs, n_out);
  if (!ast.ok()) return ast;
  DeviceGuard guard(e->device);
  RunCtx c{e, inputs, outputs, stream};
  const bool prof = !e->events.empty() && e->prof_runs < e->prof_max_runs;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (stream != nullptr) HIP_TRY(hipStreamIsCapturing(stream, &cs), "hipStreamIsCapturing");
  if ((e->options & BYOC_OPT_GRAPH_REPLAY) && !prof && stream != nullptr && cs == hipStreamCaptureStatusNone) {
    Status st = run_graph(e, c, n_in, n_out);
    if (st.ok()) HIP_TRY(hipEventRecord(e->done, stream), "hipEventRecord");
    return st;
  }
  Status st = launch_all(e, c, prof);
  // completion marker for destroy (not inside a capture of the caller's)
  if (st.ok() && cs == hipStreamCaptureStatusNone) HIP_TRY(hipEventRecord(e->done, stream), "hipEventRecord");
  return st;
}

Status engine_run_static(Engine* e, const void* const* inputs, int32_t n_in, void* const* outputs,
                         int32_t n_out, hipStream_t stream) {
  Status st = check_run_args(e, inputs, n_in, outputs, n_out);
  if (!st.ok()) return st;
  if (e->arena_bytes > kStaticScratchBytes)
    return Status::Err(BYOC_ERR_INVALID_ARG, "the engine's intermediates need " + std::to_string(e->arena_bytes) +
                                                 " bytes, more than the static scratch of " +
                                                 std::to_string(kStaticScratchBytes) + " bytes");
  DeviceGuard guard(e->device);
  void* scratch = nullptr;
  HIP_TRY(static_scratch_ptr(e->device, &scratch), "static scratch address");
  RunCtx c{e, inputs, outputs, stream};
  c.arena = static_cast<char*>(scratch);
  return launch_all(e, c, false);
}

Status engine_profile_begin(Engine* e, int max_runs) {
  if (max_runs < 1 || max_runs > 100000)
    return Status::Err(BYOC_ERR_INVALID_ARG, "max_runs must be in [1, 100000]");
  DeviceGuard guard(e->device);
  for (hipEvent_t ev : e->events) (void)hipEventDestroy(ev);
  e->events.clear();
  const size_t n = (size_t)max_runs * (e->launches.size() + 1);
  e->events.resize(n);
  for (size_t i = 0; i < n; ++i) {
    hipError_t err = hipEventCreateWithFlags(&e->events[i], hipEventDisableSystemFence);
    if (err != hipSuccess) {
      e->events.resize(i);
      for (hipEvent_t ev : e->events) (void)hipEventDestroy(ev);
      e->events.clear();
      return Status::Err(BYOC_ERR_DEVICE, std::string("hipEventCreate: ") + hipGetErrorString(err));
    }
  }
  e->prof_max_runs = max_runs;
  e->prof_runs = 0;
  return Status::Ok();
}

Status engine_profile_end(Engine* e, float* ms, int n, int* runs) {
  const size_t nl = e->launches.size();
  if (e->events.empty()) return Status::Err(BYOC_ERR_INVALID_ARG, "profiling was not begun");
  if (ms && n < (int)nl)
    return Status::Err(BYOC_ERR_INVALID_ARG, "ms holds " + std::to_string(n) + " entries, need " +
                                                 std::to_string(nl));
  DeviceGuard guard(e->device);
  Status st;
  if (ms)
    for (size_t i = 0; i < nl; ++i) ms[i] = 0.f;
  if (e->prof_runs > 0) {
    hipEvent_t* last = &e->events[(size_t)(e->prof_runs - 1) * (nl + 1)];
    hipError_t err = hipEventSynchronize(last[nl]);
    if (err != hipSuccess) st = Status::Err(BYOC_ERR_DEVICE, std::string("hipEventSynchronize: ") + hipGetErrorString(err));
    for (int r = 0; r < e->prof_runs && st.ok() && ms; ++r) {
      hipEvent_t* ev = &e->events[(size_t)r * (nl + 1)];
      for (size_t i = 0; i < nl; ++i) {
        float t = 0.f;
        err = hipEventElapsedTime(&t, ev[i], ev[i + 1]);
        if (err != hipSuccess) {
          st = Status::Err(BYOC_ERR_DEVICE, std::string("hipEventElapsedTime: ") + hipGetErrorString(err));
          break;
        }
        ms[i] += t;
      }
    }
  }
  if (runs) *runs = e->prof_runs;
  for (hipEvent_t ev : e->events) (void)hipEventDestroy(ev);
  e->events.clear();
  e->prof_runs = 0;
  e->prof_max_runs = 0;
  return st;
}

Status engine_destroy(Engine* e) {
  if (!e) return Status::Ok();
  Status st;
  {
    DeviceGuard guard(e->device);
    // the last run enqueued through run() (the event completes at once when
    // there was none); runs of run_static are the caller's to synchronise
    hipError_t err = e->done ? hipEventSynchronize(e->done) : hipSuccess;
    if (err != hipSuccess) st = Status::Err(BYOC_ERR_DEVICE, std::string("destroy: ") + hipGetErrorString(err));
    release(e);
  }
  delete e;
  return st;
}

}  // namespace byoc
