// Bandwidth-bound kernels: depthwise conv, pooling, elementwise add, the
// boundary layout/dtype transforms and the constant packers.  No MFMA: each
// lane moves 16-byte vectors (8 bf16 channels of one NHWC pixel) and
// consecutive lanes take consecutive channel groups of a pixel, so a wave
// reads and writes contiguous runs of memory.
#include <algorithm>
#include <cstdio>
#include <cstdlib>

#include "device_common.h"

namespace byoc {
namespace {

constexpr int kThreads = 256;

inline unsigned grid_for(int64_t n) { return (unsigned)((n + kThreads - 1) / kThreads); }

// ---------------------------------------------------------------------------
// Depthwise conv, NHWC bf16, one thread per (pixel, 8-channel group).
__global__ __launch_bounds__(kThreads) void depthwise_kernel(DwParams p) {
  const int G = p.Cp / 8;
  const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t total = (int64_t)p.N * p.P * p.Q * G;
  if (idx >= total) return;
  const int g = (int)(idx % G);
  int64_t t = idx / G;
  const int q = (int)(t % p.Q);
  t /= p.Q;
  const int pp = (int)(t % p.P);
  const int n = (int)(t / p.P);
  float acc[8];
  const float4 b0 = *(const float4*)(p.bias + g * 8);
  const float4 b1 = *(const float4*)(p.bias + g * 8 + 4);
  acc[0] = b0.x; acc[1] = b0.y; acc[2] = b0.z; acc[3] = b0.w;
  acc[4] = b1.x; acc[5] = b1.y; acc[6] = b1.z; acc[7] = b1.w;
  const int ih0 = pp * p.sh - p.pt;
  const int iw0 = q * p.sw - p.pl;
  const bf16_t* xn = p.x + (size_t)n * p.H * p.W * p.Cp + g * 8;
  for (int r = 0; r < p.R; ++r) {
    const int ih = ih0 + r;
    if ((unsigned)ih >= (unsigned)p.H) continue;
    for (int s = 0; s < p.S; ++s) {
      const int iw = iw0 + s;
      if ((unsigned)iw >= (unsigned)p.W) continue;
      float xv[8], wv[8];
      unpack8(*(const uint4*)(xn + ((size_t)ih * p.W + iw) * p.Cp), xv);
      unpack8(*(const uint4*)(p.w + (size_t)(r * p.S + s) * p.Cp + g * 8), wv);
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] = fmaf(xv[i], wv[i], acc[i]);
    }
  }
  const size_t o = (((size_t)n * p.P + pp) * p.Q + q) * p.Cp + g * 8;
  if (p.res) {
    float rv[8];
    unpack8(*(const uint4*)(p.res + o), rv);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] += rv[i];
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = apply_act(acc[i], p.act, p.alpha);
  *(uint4*)(p.y + o) = pack8(acc);
}

// Depthwise 3x3 conv, NHWC bf16, stride ST (1 or 2), any padding: every
// thread finishes V vertically adjacent output pixels of one column for 8
// channels.  It loads the (V - 1) * ST + 3 input rows x 3 columns that the
// strip covers once into registers (16-byte buffer loads; an offset outside
// the image reads zeros, which is the zero padding), the 9 tap weights and
// the bias once, and then forms the V outputs from registers, so each input
// row is fetched once per strip instead of once per tap and output.  Lanes
// take consecutive channel groups, then consecutive columns, so every load
// instruction of a wave reads one contiguous run of NHWC memory.  Blocks:
// xb blocks of kThreads over (column, channel group) per (image, strip),
// image-major.  The hardware deals workgroups round-robin to the 8 XCDs, so
// XCD x takes the contiguous run of blocks [x * per_xcd, (x + 1) * per_xcd):
// the blocks of one image, which read each other's halo rows and edge
// columns, share one L2 and fetch each input line from HBM once.  The taps
// are summed in the order (row, column) like the generic kernel, each output
// from the bias up, so both kernels give the same bits.
template <int ST, int V, int MODE>
__global__ __launch_bounds__(kThreads) void depthwise3x3_kernel(DwParams p, int x_bytes, int strips, int xb,
                                                                  int per_xcd, int blocks, uint64_t mg_g,
                                                                  uint64_t mg_strips, uint64_t mg_xb) {
  constexpr int NR = (V - 1) * ST + 3;  // input rows of a strip
  const int G = p.Cp / 8;
  const int blk = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (blk >= blocks) return;
  const int ns = mdiv(blk, mg_xb);  // (image, strip)
  const int pos = (blk - ns * xb) * kThreads + threadIdx.x;
  if (pos >= G * p.Q) return;
  const int q = mdiv(pos, mg_g);
  const int g = pos - q * G;
  const int n = mdiv(ns, mg_strips);
  const int p0 = (ns - n * strips) * V;
  const int ih0 = p0 * ST - p.pt, iw0 = q * ST - p.pl;
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(p.x), (short)0, x_bytes, kBufferFlags);
  // image n's rows, element offsets (32-bit: x_bytes < 2^31)
  const int img = n * p.H * p.W * p.Cp + g * 8;
  uint4 xv[NR][3];
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const int ih = ih0 + r;
    const bool rok = (unsigned)ih < (unsigned)p.H;
#pragma unroll
    for (int c = 0; c < 3; ++c) {
      const int iw = iw0 + c;
      const bool ok = rok && (unsigned)iw < (unsigned)p.W;
      const uint32_t off = ok ? (uint32_t)(img + (ih * p.W + iw) * p.Cp) * 2u : kOOB;
      xv[r][c] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
    }
  }
  uint4 wv[9];
#pragma unroll
  for (int t = 0; t < 9; ++t) wv[t] = *(const uint4*)(p.w + t * p.Cp + g * 8);
  const float4 b0 = *(const float4*)(p.bias + g * 8);
  const float4 b1 = *(const float4*)(p.bias + g * 8 + 4);
  const ActClamp ac = act_clamp_of(p.act, p.alpha);
#pragma unroll
  for (int v = 0; v < V; ++v) {
    const int pp = p0 + v;
    if (pp >= p.P) break;
    float acc[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
      for (int c = 0; c < 3; ++c) {
        float xf[8], wf[8];
        unpack8(xv[v * ST + r][c], xf);
        unpack8(wv[r * 3 + c], wf);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = fmaf(xf[i], wf[i], acc[i]);
      }
    const int o = ((n * p.P + pp) * p.Q + q) * p.Cp + g * 8;
    float rv[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (p.res) unpack8(*(const uint4*)(p.res + o), rv);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = act_apply<MODE>(acc[i] + rv[i], ac);
    *(uint4*)(p.y + o) = pack8(acc);
  }
}

// Max pool NHWC bf16; the max of bf16 values is exact, no rounding.
__global__ __launch_bounds__(kThreads) void maxpool_nhwc_kernel(PoolParams p) {
  const int G = p.Cp / 8;
  const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t total = (int64_t)p.N * p.P * p.Q * G;
  if (idx >= total) return;
  const int g = (int)(idx % G);
  int64_t t = idx / G;
  const int q = (int)(t % p.Q);
  t /= p.Q;
  const int pp = (int)(t % p.P);
  const int n = (int)(t / p.P);
  const bf16_t* x = (const bf16_t*)p.x + (size_t)n * p.H * p.W * p.Cp + g * 8;
  float m[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) m[i] = -INFINITY;
  const int ih0 = pp * p.sh - p.pt;
  const int iw0 = q * p.sw - p.pl;
  for (int r = 0; r < p.R; ++r) {
    const int ih = ih0 + r;
    if ((unsigned)ih >= (unsigned)p.H) continue;
    for (int s = 0; s < p.S; ++s) {
      const int iw = iw0 + s;
      if ((unsigned)iw >= (unsigned)p.W) continue;
      float v[8];
      unpack8(*(const uint4*)(x + ((size_t)ih * p.W + iw) * p.Cp), v);
#pragma unroll
      for (int i = 0; i < 8; ++i) m[i] = fmaxf(m[i], v[i]);
    }
  }
  *(uint4*)((bf16_t*)p.y + (((size_t)n * p.P + pp) * p.Q + q) * (p.ldy ? p.ldy : p.Cp) + g * 8) = pack8(m);
}

// Windowed average pool, NHWC bf16, 8 channels per thread: fp32 sum of the
// taps inside the image, divided by their count (or by the full window).
__global__ __launch_bounds__(kThreads) void avgpool_win_nhwc_kernel(PoolParams p, int incl) {
  const int G = p.Cp / 8;
  const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t total = (int64_t)p.N * p.P * p.Q * G;
  if (idx >= total) return;
  const int g = (int)(idx % G);
  int64_t t = idx / G;
  const int q = (int)(t % p.Q);
  t /= p.Q;
  const int pp = (int)(t % p.P);
  const int n = (int)(t / p.P);
  const bf16_t* x = (const bf16_t*)p.x + (size_t)n * p.H * p.W * p.Cp + g * 8;
  float m[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) m[i] = 0.0f;
  int cnt = 0;
  const int ih0 = pp * p.sh - p.pt;
  const int iw0 = q * p.sw - p.pl;
  for (int r = 0; r < p.R; ++r) {
    const int ih = ih0 + r;
    if ((unsigned)ih >= (unsigned)p.H) continue;
    for (int s = 0; s < p.S; ++s) {
      const int iw = iw0 + s;
      if ((unsigned)iw >= (unsigned)p.W) continue;
      float v[8];
      unpack8(*(const uint4*)(x + ((size_t)ih * p.W + iw) * p.Cp), v);
#pragma unroll
      for (int i = 0; i < 8; ++i) m[i] += v[i];
      ++cnt;
    }
  }
  const float d = (float)(incl ? p.R * p.S : cnt);
#pragma unroll
  for (int i = 0; i < 8; ++i) m[i] = m[i] / d;
  *(uint4*)((bf16_t*)p.y + (((size_t)n * p.P + pp) * p.Q + q) * (p.ldy ? p.ldy : p.Cp) + g * 8) = pack8(m);
}

// 8 channels (16 bytes) per thread.
__global__ __launch_bounds__(kThreads) void copy_channels_kernel(const bf16_t* src, int src_ld, bf16_t* dst,
                                                                 int dst_ld, int64_t pixels, int G) {
  const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (idx >= pixels * G) return;
  const int g = (int)(idx % G);
  const int64_t px = idx / G;
  *(uint4*)(dst + px * dst_ld + g * 8) = *(const uint4*)(src + px * src_ld + g * 8);
}

// Global average pool NHWC bf16 -> [N][Cp] bf16.  Workgroup = one image x
// 32 channel groups of 8.  The 8 lanes of a group are consecutive: lane j
// sums pixels j, j + 8, ... in order (eight loads in flight), then the 8
// partial sums meet in a 3-step butterfly (a fixed pairing; addition is
// commutative, so every lane holds the same bits) and are scaled by
// 1 / (H W).  Run-to-run identical.
__global__ __launch_bounds__(kThreads) void avgpool_nhwc_kernel(PoolParams p) {
  const int G = p.Cp / 8;
  const int n = blockIdx.x;
  const int pl = threadIdx.x & 7;
  const int g = blockIdx.y * (kThreads / 8) + (threadIdx.x >> 3);
  const int HW = p.H * p.W;
  const bool ok = g < G;
  const bf16_t* x = (const bf16_t*)p.x + (size_t)n * HW * p.Cp + (size_t)(ok ? g : 0) * 8;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  auto add = [&](const uint4& u) {
    float v[8];
    unpack8(u, v);
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] += v[c];
  };
  // chunks of 64 pixels: the thread's (up to) 8 loads of a chunk are all
  // issued before the first add (pixels past the image read pixel 0 and
  // are not added)
  for (int i0 = 0; i0 < HW; i0 += 64) {
    uint4 u[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int i = i0 + pl + 8 * j;
      u[j] = *(const uint4*)(x + (size_t)(i < HW ? i : 0) * p.Cp);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (i0 + pl + 8 * j < HW) add(u[j]);
  }
#pragma unroll
  for (int o = 1; o < 8; o <<= 1)
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] += __shfl_xor(acc[c], o);
  if (ok && pl == 0) {
    const float inv = 1.0f / (float)HW;
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] *= inv;
    *(uint4*)((bf16_t*)p.y + (size_t)n * p.Cp + g * 8) = pack8(acc);
  }
}

// fp32 NCHW pools, one thread per output.
__global__ __launch_bounds__(kThreads) void maxpool_nchw_f32_kernel(PoolParams p) {
  const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t total = (int64_t)p.N * p.C * p.P * p.Q;
  if (idx >= total) return;
  const int q = (int)(idx % p.Q);
  int64_t t = idx / p.Q;
  const int pp = (int)(t % p.P);
  t /= p.P;
  const float* x = (const float*)p.x + (size_t)t * p.H * p.W;
  float m = -INFINITY;
  for (int r = 0; r < p.R; ++r) {
    const int ih = pp * p.sh - p.pt + r;
    if ((unsigned)ih >= (unsigned)p.H) continue;
    for (int s = 0; s < p.S; ++s) {
      const int iw = q * p.sw - p.pl + s;
      if ((unsigned)iw >= (unsigned)p.W) continue;
      m = fmaxf(m, x[ih * p.W + iw]);
    }
  }
  ((float*)p.y)[idx] = m;
}

__global__ __launch_bounds__(kThreads) void avgpool_nchw_f32_kernel(PoolParams p) {
  const int idx = blockIdx.x * kThreads + threadIdx.x;
  if (idx >= p.N * p.C) return;
  const float* x = (const float*)p.x + (size_t)idx * p.H * p.W;
  float acc = 0.f;
  for (int i = 0; i < p.H * p.W; ++i) acc += x[i];
  ((float*)p.y)[idx] = acc / (float)(p.H * p.W);
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void add_bf16_kernel(const bf16_t* a, const bf16_t* b,
                                                            bf16_t* y, int64_t n8, int act, float alpha) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= n8) return;
  float va[8], vb[8];
  unpack8(((const uint4*)a)[i], va);
  unpack8(((const uint4*)b)[i], vb);
#pragma unroll
  for (int c = 0; c < 8; ++c) va[c] = apply_act(va[c] + vb[c], act, alpha);
  ((uint4*)y)[i] = pack8(va);
}

__global__ __launch_bounds__(kThreads) void add_f32_kernel(const float* a, const float* b,
                                                           float* y, int64_t n, int act, float alpha) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= n) return;
  y[i] = apply_act(a[i] + b[i], act, alpha);
}

// ---------------------------------------------------------------------------
// NCHW (f32 or bf16) -> NHWC bf16 with Cp >= C channels (pad zero).  Thread
// per (n, channel group, h, w) with w fastest: reads are contiguous along w
// for each channel; each thread writes one 16-byte vector.
// Grid x over the pixels of an image, y over (image, channel group): every
// thread moves 8 channels of one pixel, 32-bit index math (a plane holds
// fewer than 2^31 pixels; image offsets in size_t).
template <typename SrcT>
__global__ __launch_bounds__(kThreads) void nchw_to_nhwc_kernel(const SrcT* x, bf16_t* y, int N, int C, int HW,
                                                                int Cp) {
  const int hw = blockIdx.x * kThreads + threadIdx.x;
  if (hw >= HW) return;
  const int G = Cp / 8;
  const int n = blockIdx.y / G;
  const int g = blockIdx.y - n * G;
  const SrcT* xn = x + (size_t)n * C * HW + hw;
  float v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int c = g * 8 + i;
    float f = 0.f;
    if (c < C) {
      const SrcT e = xn[(size_t)c * HW];
      if constexpr (sizeof(SrcT) == 2) f = bf16_to_f32(e);
      else f = e;
    }
    v[i] = f;
  }
  *(uint4*)(y + ((size_t)n * HW + hw) * Cp + g * 8) = pack8(v);
}

template <typename DstT>
__global__ __launch_bounds__(kThreads) void nhwc_to_nchw_kernel(const bf16_t* x, DstT* y, int N, int C, int HW,
                                                                int Cp) {
  const int hw = blockIdx.x * kThreads + threadIdx.x;
  if (hw >= HW) return;
  const int G = Cp / 8;
  const int n = blockIdx.y / G;
  const int g = blockIdx.y - n * G;
  const uint4 u = *(const uint4*)(x + ((size_t)n * HW + hw) * Cp + g * 8);
  const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
  DstT* yn = y + (size_t)n * C * HW + hw;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int c = g * 8 + i;
    if (c >= C) break;
    const bf16_t h = (bf16_t)((i & 1) ? (w4[i >> 1] >> 16) : (w4[i >> 1] & 0xFFFF));
    if constexpr (sizeof(DstT) == 2) yn[(size_t)c * HW] = h;
    else yn[(size_t)c * HW] = bf16_to_f32(h);
  }
}

template <typename SrcT>
__global__ __launch_bounds__(kThreads) void rows_to_padded_kernel(const SrcT* x, bf16_t* y, int M,
                                                                  int K, int Kp) {
  const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (idx >= (int64_t)M * Kp) return;
  const int k = (int)(idx % Kp);
  const int64_t m = idx / Kp;
  bf16_t o = 0;
  if (k < K) {
    const SrcT e = x[m * K + k];
    if constexpr (sizeof(SrcT) == 2) o = e;
    else o = f32_to_bf16(e);
  }
  y[idx] = o;
}

template <typename DstT>
__global__ __launch_bounds__(kThreads) void padded_to_rows_kernel(const bf16_t* x, DstT* y, int M,
                                                                  int K, int Kp) {
  const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (idx >= (int64_t)M * K) return;
  const int k = (int)(idx % K);
  const int64_t m = idx / K;
  const bf16_t h = x[m * Kp + k];
  if constexpr (sizeof(DstT) == 2) y[idx] = h;
  else y[idx] = bf16_to_f32(h);
}

template <typename SrcT, typename DstT>
__global__ __launch_bounds__(kThreads) void cast_kernel(const SrcT* x, DstT* y, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= n) return;
  float f;
  if constexpr (sizeof(SrcT) == 2) f = bf16_to_f32(x[i]);
  else f = x[i];
  if constexpr (sizeof(DstT) == 2) y[i] = f32_to_bf16(f);
  else y[i] = f;
}

// ---------------------------------------------------------------------------
// Constant packers (engine creation only).
template <typename SrcT>
__device__ __forceinline__ float load_f(const SrcT* p, size_t i) {
  if constexpr (sizeof(SrcT) == 2) return bf16_to_f32(p[i]);
  else return p[i];
}

template <typename SrcT>
__global__ __launch_bounds__(kThreads) void pack_conv_weights_kernel(const SrcT* src, bf16_t* dst,
                                                                     int K, int Cg, int R, int S,
                                                                     int Cp, int Kgp, int rows) {
  const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (idx >= (int64_t)rows * Kgp) return;
  const int kk = (int)(idx % Kgp);
  const int k = (int)(idx / Kgp);
  const int rs = kk / Cp;
  const int c = kk - rs * Cp;
  bf16_t o = 0;
  if (k < K && rs < R * S && c < Cg) {
    const int r = rs / S;
    const int s = rs - r * S;
    o = f32_to_bf16(load_f(src, (((size_t)k * Cg + c) * R + r) * S + s));
  }
  dst[idx] = o;
}

template <typename SrcT>
__global__ __launch_bounds__(kThreads) void pack_dw_weights_kernel(const SrcT* src, bf16_t* dst,
                                                                   int C, int R, int S, int Cp) {
  const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (idx >= (int64_t)R * S * Cp) return;
  const int c = (int)(idx % Cp);
  const int rs = (int)(idx / Cp);
  dst[idx] = c < C ? f32_to_bf16(load_f(src, (size_t)c * R * S + rs)) : (bf16_t)0;
}

// The same taps as float32 values of the bf16 weights (the fused
// inverted-residual kernel reads them unpacked).
template <typename SrcT>
__global__ __launch_bounds__(kThreads) void pack_dw_weights_f32_kernel(const SrcT* src, float* dst, int C, int R,
                                                                       int S, int Cp) {
  const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (idx >= (int64_t)R * S * Cp) return;
  const int c = (int)(idx % Cp);
  const int rs = (int)(idx / Cp);
  dst[idx] = c < C ? bf16_to_f32(f32_to_bf16(load_f(src, (size_t)c * R * S + rs))) : 0.f;
}

template <typename SrcT>
__global__ __launch_bounds__(kThreads) void pack_vector_kernel(const SrcT* src, float* dst, int K,
                                                               int n_out) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i >= n_out) return;
  dst[i] = i < K ? load_f(src, i) : 0.f;
}

}  // namespace

namespace {

template <int ST, int V>
hipError_t launch_dw3x3(const DwParams& p, int x_bytes, hipStream_t s) {
  const int G = p.Cp / 8;
  const int strips = (p.P + V - 1) / V;
  const int xb = (G * p.Q + kThreads - 1) / kThreads;
  const int blocks = xb * p.N * strips;  // < 2^25 (checked by the caller)
  const int per_xcd = (blocks + 7) / 8;
  const unsigned grid = 8u * (unsigned)per_xcd;
  const int mode = act_mode(p.act);
  const uint64_t mg = magic40(G), ms = magic40(strips), mx = magic40(xb);
  if (mode == 1)
    depthwise3x3_kernel<ST, V, 1><<<grid, kThreads, 0, s>>>(p, x_bytes, strips, xb, per_xcd, blocks, mg, ms, mx);
  else if (mode == 0)
    depthwise3x3_kernel<ST, V, 0><<<grid, kThreads, 0, s>>>(p, x_bytes, strips, xb, per_xcd, blocks, mg, ms, mx);
  else
    depthwise3x3_kernel<ST, V, 2><<<grid, kThreads, 0, s>>>(p, x_bytes, strips, xb, per_xcd, blocks, mg, ms, mx);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_depthwise(const DwParams& p, hipStream_t s) {
  const int64_t x_bytes = (int64_t)p.N * p.H * p.W * p.Cp * 2;
  const int64_t y_elems = (int64_t)p.N * p.P * p.Q * p.Cp;
  // strip kernel: 3x3 taps, equal strides of 1 or 2, 32-bit offsets, the
  // index products of the magic divisions below 2^40 and fewer than 2^25
  // workgroups
  const bool strip = p.R == 3 && p.S == 3 && p.sh == p.sw && (p.sh == 1 || p.sh == 2) && p.Cp % 8 == 0 &&
                     x_bytes < (int64_t(1) << 31) && y_elems < (int64_t(1) << 31) &&
                     (int64_t)(p.Cp / 8) * p.Q < (int64_t(1) << 20) && (int64_t)p.N * p.P < (int64_t(1) << 20) &&
                     ((int64_t)(p.Cp / 8) * p.Q + kThreads - 1) / kThreads * p.N * p.P < (int64_t(1) << 25);
  if (strip) {
    // strip height (output rows per thread): 4 (stride 1) and 2 (stride 2)
    // by default; BYOC_DW_STRIP=<v1>,<v2> picks 2, 4 or 8 and 1, 2 or 4
    int v1 = 4, v2 = 2;
    if (const char* e = std::getenv("BYOC_DW_STRIP")) std::sscanf(e, "%d,%d", &v1, &v2);
    if (p.sh == 1) {
      if (v1 == 2) return launch_dw3x3<1, 2>(p, (int)x_bytes, s);
      if (v1 == 8) return launch_dw3x3<1, 8>(p, (int)x_bytes, s);
      return launch_dw3x3<1, 4>(p, (int)x_bytes, s);
    }
    if (v2 == 1) return launch_dw3x3<2, 1>(p, (int)x_bytes, s);
    if (v2 == 4) return launch_dw3x3<2, 4>(p, (int)x_bytes, s);
    return launch_dw3x3<2, 2>(p, (int)x_bytes, s);
  }
  const int64_t n = (int64_t)p.N * p.P * p.Q * (p.Cp / 8);
  depthwise_kernel<<<grid_for(n), kThreads, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_maxpool_nhwc_bf16(const PoolParams& p, hipStream_t s) {
  const int64_t n = (int64_t)p.N * p.P * p.Q * (p.Cp / 8);
  maxpool_nhwc_kernel<<<grid_for(n), kThreads, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_avgpool_win_nhwc_bf16(const PoolParams& p, bool count_include_pad, hipStream_t s) {
  if (p.Cp % 8 != 0 || (p.ldy && p.ldy % 8 != 0)) return hipErrorInvalidValue;
  const int64_t n = (int64_t)p.N * p.P * p.Q * (p.Cp / 8);
  avgpool_win_nhwc_kernel<<<grid_for(n), kThreads, 0, s>>>(p, count_include_pad ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_copy_channels_bf16(const bf16_t* src, int src_ld, bf16_t* dst, int dst_ld, int64_t pixels, int C,
                                     hipStream_t s) {
  if (C % 8 != 0 || src_ld % 8 != 0 || dst_ld % 8 != 0 || C > src_ld || C > dst_ld) return hipErrorInvalidValue;
  if (pixels * (C / 8) == 0) return hipSuccess;
  copy_channels_kernel<<<grid_for(pixels * (C / 8)), kThreads, 0, s>>>(src, src_ld, dst, dst_ld, pixels, C / 8);
  return hipGetLastError();
}

hipError_t launch_avgpool_nhwc_bf16(const PoolParams& p, hipStream_t s) {
  avgpool_nhwc_kernel<<<dim3(p.N, (p.Cp / 8 + kThreads / 8 - 1) / (kThreads / 8)), kThreads, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_maxpool_nchw_f32(const PoolParams& p, hipStream_t s) {
  const int64_t n = (int64_t)p.N * p.C * p.P * p.Q;
  maxpool_nchw_f32_kernel<<<grid_for(n), kThreads, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_avgpool_nchw_f32(const PoolParams& p, hipStream_t s) {
  avgpool_nchw_f32_kernel<<<grid_for((int64_t)p.N * p.C), kThreads, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_add_bf16(const bf16_t* a, const bf16_t* b, bf16_t* y, int64_t n, int act, float alpha,
                           hipStream_t s) {
  add_bf16_kernel<<<grid_for(n / 8), kThreads, 0, s>>>(a, b, y, n / 8, act, alpha);
  return hipGetLastError();
}

hipError_t launch_add_f32(const float* a, const float* b, float* y, int64_t n, int act, float alpha,
                          hipStream_t s) {
  add_f32_kernel<<<grid_for(n), kThreads, 0, s>>>(a, b, y, n, act, alpha);
  return hipGetLastError();
}

// Both layout transforms launch one grid row per (image, channel group);
// batches with more rows than a grid dimension holds go in image chunks.
constexpr int64_t kMaxGridY = 65535;

hipError_t launch_nchw_to_nhwc(const void* x, bool src_bf16, bf16_t* y, int N, int C, int H,
                               int W, int Cp, hipStream_t s) {
  const int64_t HW = (int64_t)H * W, G = Cp / 8;
  if (HW == 0 || G == 0 || N == 0) return hipSuccess;
  if (HW >= (int64_t(1) << 31) || G > kMaxGridY) return hipErrorInvalidValue;
  const int chunk = (int)std::min<int64_t>(N, kMaxGridY / G);
  const size_t esz = src_bf16 ? 2 : 4;
  for (int n0 = 0; n0 < N; n0 += chunk) {
    const int nn = std::min(chunk, N - n0);
    const dim3 grid(grid_for(HW), (unsigned)(nn * G));
    const char* xs = (const char*)x + (size_t)n0 * C * HW * esz;
    bf16_t* yd = y + (size_t)n0 * HW * Cp;
    if (src_bf16)
      nchw_to_nhwc_kernel<bf16_t><<<grid, kThreads, 0, s>>>((const bf16_t*)xs, yd, nn, C, (int)HW, Cp);
    else
      nchw_to_nhwc_kernel<float><<<grid, kThreads, 0, s>>>((const float*)xs, yd, nn, C, (int)HW, Cp);
  }
  return hipGetLastError();
}

hipError_t launch_nhwc_to_nchw(const bf16_t* x, void* y, bool dst_bf16, int N, int C, int H,
                               int W, int Cp, hipStream_t s) {
  const int64_t HW = (int64_t)H * W, G = Cp / 8;
  if (HW == 0 || G == 0 || N == 0) return hipSuccess;
  if (HW >= (int64_t(1) << 31) || G > kMaxGridY) return hipErrorInvalidValue;
  const int chunk = (int)std::min<int64_t>(N, kMaxGridY / G);
  const size_t esz = dst_bf16 ? 2 : 4;
  for (int n0 = 0; n0 < N; n0 += chunk) {
    const int nn = std::min(chunk, N - n0);
    const dim3 grid(grid_for(HW), (unsigned)(nn * G));
    const bf16_t* xs = x + (size_t)n0 * HW * Cp;
    char* yd = (char*)y + (size_t)n0 * C * HW * esz;
    if (dst_bf16)
      nhwc_to_nchw_kernel<bf16_t><<<grid, kThreads, 0, s>>>(xs, (bf16_t*)yd, nn, C, (int)HW, Cp);
    else
      nhwc_to_nchw_kernel<float><<<grid, kThreads, 0, s>>>(xs, (float*)yd, nn, C, (int)HW, Cp);
  }
  return hipGetLastError();
}

hipError_t launch_rows_to_padded(const void* x, bool src_bf16, bf16_t* y, int M, int K, int Kp,
                                 hipStream_t s) {
  const int64_t n = (int64_t)M * Kp;
  if (src_bf16)
    rows_to_padded_kernel<bf16_t><<<grid_for(n), kThreads, 0, s>>>((const bf16_t*)x, y, M, K, Kp);
  else
    rows_to_padded_kernel<float><<<grid_for(n), kThreads, 0, s>>>((const float*)x, y, M, K, Kp);
  return hipGetLastError();
}

hipError_t launch_padded_to_rows(const bf16_t* x, void* y, bool dst_bf16, int M, int K, int Kp,
                                 hipStream_t s) {
  const int64_t n = (int64_t)M * K;
  if (dst_bf16)
    padded_to_rows_kernel<bf16_t><<<grid_for(n), kThreads, 0, s>>>(x, (bf16_t*)y, M, K, Kp);
  else
    padded_to_rows_kernel<float><<<grid_for(n), kThreads, 0, s>>>(x, (float*)y, M, K, Kp);
  return hipGetLastError();
}

hipError_t launch_cast(const void* x, bool src_bf16, void* y, bool dst_bf16, int64_t n,
                       hipStream_t s) {
  const unsigned g = grid_for(n);
  if (src_bf16 && dst_bf16)
    cast_kernel<bf16_t, bf16_t><<<g, kThreads, 0, s>>>((const bf16_t*)x, (bf16_t*)y, n);
  else if (src_bf16)
    cast_kernel<bf16_t, float><<<g, kThreads, 0, s>>>((const bf16_t*)x, (float*)y, n);
  else if (dst_bf16)
    cast_kernel<float, bf16_t><<<g, kThreads, 0, s>>>((const float*)x, (bf16_t*)y, n);
  else
    cast_kernel<float, float><<<g, kThreads, 0, s>>>((const float*)x, (float*)y, n);
  return hipGetLastError();
}

hipError_t launch_pack_conv_weights(const void* src, bool src_bf16, bf16_t* dst, int K, int Cg,
                                    int R, int S, int Cp, int Kgp, int rows, hipStream_t s) {
  const int64_t n = (int64_t)rows * Kgp;
  if (src_bf16)
    pack_conv_weights_kernel<bf16_t><<<grid_for(n), kThreads, 0, s>>>((const bf16_t*)src, dst, K, Cg,
                                                                      R, S, Cp, Kgp, rows);
  else
    pack_conv_weights_kernel<float><<<grid_for(n), kThreads, 0, s>>>((const float*)src, dst, K, Cg,
                                                                     R, S, Cp, Kgp, rows);
  return hipGetLastError();
}

hipError_t launch_pack_dw_weights(const void* src, bool src_bf16, bf16_t* dst, int C, int R,
                                  int S, int Cp, hipStream_t s) {
  const int64_t n = (int64_t)R * S * Cp;
  if (src_bf16)
    pack_dw_weights_kernel<bf16_t><<<grid_for(n), kThreads, 0, s>>>((const bf16_t*)src, dst, C, R, S, Cp);
  else
    pack_dw_weights_kernel<float><<<grid_for(n), kThreads, 0, s>>>((const float*)src, dst, C, R, S, Cp);
  return hipGetLastError();
}

hipError_t launch_pack_dw_weights_f32(const void* src, bool src_bf16, float* dst, int C, int R, int S, int Cp,
                                      hipStream_t s) {
  const int64_t n = (int64_t)R * S * Cp;
  if (src_bf16)
    pack_dw_weights_f32_kernel<bf16_t><<<grid_for(n), kThreads, 0, s>>>((const bf16_t*)src, dst, C, R, S, Cp);
  else
    pack_dw_weights_f32_kernel<float><<<grid_for(n), kThreads, 0, s>>>((const float*)src, dst, C, R, S, Cp);
  return hipGetLastError();
}

hipError_t launch_pack_vector_f32(const void* src, bool src_bf16, float* dst, int K, int n_out,
                                  hipStream_t s) {
  if (src_bf16)
    pack_vector_kernel<bf16_t><<<grid_for(n_out), kThreads, 0, s>>>((const bf16_t*)src, dst, K, n_out);
  else
    pack_vector_kernel<float><<<grid_for(n_out), kThreads, 0, s>>>((const float*)src, dst, K, n_out);
  return hipGetLastError();
}

}  // namespace byoc
