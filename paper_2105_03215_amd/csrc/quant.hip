// Memory-bound kernels of partially quantized subgraphs (Sec. 3.2,
// Fig. 4a): the boundary quantize / dequantize nodes (with the NCHW <-> NHWC
// layout change of the boundary fused in), max and global average pooling
// of codes, and the standalone add.  All of them move int8 codes in 16-byte
// (16-channel) groups where the layout allows.
#include "device_common.h"

namespace byoc {
namespace {

constexpr int kThreads = 256;

inline int grid_for(int64_t n) {
  const int64_t b = (n + kThreads - 1) / kThreads;
  return (int)(b < 1 ? 1 : (b > (int64_t(1) << 30) ? (int64_t(1) << 30) : b));
}

__device__ __forceinline__ float load_f(const void* x, bool bf16, int64_t i) {
  return bf16 ? bf16_to_f32(reinterpret_cast<const bf16_t*>(x)[i]) : reinterpret_cast<const float*>(x)[i];
}

// One thread per (n, 16-channel group, h, w), w fastest: the 16 reads of a
// thread are coalesced across the wave along w, the write is 16 bytes.
__global__ __launch_bounds__(kThreads) void quantize_kernel(const void* x, int src_bf16, int8_t* y, int N, int C,
                                                            int H, int W, int Cp, float inv, int zp) {
  const int HW = H * W, G = Cp / 16;
  const int total = N * G * HW;  // < 2^31: the element count is bounded at parse
  for (int i = blockIdx.x * kThreads + threadIdx.x; i < total; i += gridDim.x * kThreads) {
    const int hw = i % HW;
    const int ng = i / HW;
    const int g = ng % G;
    const int n = ng / G;
    uint32_t w4[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int c = g * 16 + j;
      int code = 0;
      if (c < C) {
        float t = rintf(load_f(x, src_bf16, ((int64_t)n * C + c) * HW + hw) * inv);
        t = fminf(fmaxf(t, -512.0f), 512.0f);
        code = clip_i8((int)t + zp);
      }
      w4[j >> 2] |= ((uint32_t)code & 0xFFu) << (8 * (j & 3));
    }
    *(uint4*)(y + ((int64_t)n * HW + hw) * Cp + g * 16) = make_uint4(w4[0], w4[1], w4[2], w4[3]);
  }
}

// One workgroup per output row (n, p): the R input rows it reads are
// quantized once into LDS as one dword of 4 channel codes per pixel (the
// zero point for rows outside the image; coalesced loads along w), then the
// Q im2col rows of the output row are written from LDS as consecutive
// dwords (fully coalesced stores).
constexpr int kIm2colLds = 48 * 1024;  // bytes of staged input rows (R * W * 4)

__global__ __launch_bounds__(kThreads) void quantize_im2col_kernel(const void* x, int src_bf16, int8_t* y,
                                                                   PoolParams g, float inv, int zp) {
  extern __shared__ uint32_t rows[];  // R * W dwords (dynamic: the launch sizes it)
  const int n = blockIdx.x / g.P, pp = blockIdx.x - n * g.P;
  const int HW = g.H * g.W;
  const uint32_t zrow = ((uint32_t)zp & 0xFFu) * 0x01010101u;
  for (int t = threadIdx.x; t < g.R * g.W; t += kThreads) {
    const int r = t / g.W, iw = t - r * g.W;
    const int ih = pp * g.sh - g.pt + r;
    uint32_t w = zrow;
    if ((unsigned)ih < (unsigned)g.H) {
      w = 0u;
      for (int c = 0; c < g.C; ++c) {
        float v = rintf(load_f(x, src_bf16, ((int64_t)(n * g.C + c) * g.H + ih) * g.W + iw) * inv);
        v = fminf(fmaxf(v, -512.0f), 512.0f);
        w |= ((uint32_t)clip_i8((int)v + zp) & 0xFFu) << (8 * c);
      }
    }
    rows[t] = w;
  }
  __syncthreads();
  // each thread keeps one dword k of the row (its tap fixed) and walks the
  // pixels: lanes 0..63 of a wave store 64 consecutive dwords of a row
  const int KW = g.Cp / 4, RS = g.R * g.S;
  uint32_t* out = reinterpret_cast<uint32_t*>(y + ((int64_t)n * g.P + pp) * g.Q * g.Cp);
  for (int k = threadIdx.x & 63; k < KW; k += 64) {
    const int r = k / g.S, s = k - r * g.S;
    const uint32_t* src = rows + r * g.W;
    for (int qq = threadIdx.x >> 6; qq < g.Q; qq += kThreads / 64) {
      const int iw = qq * g.sw - g.pl + s;
      out[qq * KW + k] = k >= RS ? 0u : ((unsigned)iw < (unsigned)g.W ? src[iw] : zrow);
    }
  }
}

// One thread per output element (n, c, h, w), w fastest.
__global__ __launch_bounds__(kThreads) void dequantize_kernel(const int8_t* x, void* y, int dst_bf16, int N, int C,
                                                              int H, int W, int Cp, float scale, int zp) {
  const int HW = H * W;
  const int total = N * C * HW;  // < 2^31: the element count is bounded at parse
  for (int i = blockIdx.x * kThreads + threadIdx.x; i < total; i += gridDim.x * kThreads) {
    const int hw = i % HW;
    const int nc = i / HW;
    const int c = nc % C;
    const int n = nc / C;
    const float v = scale * (float)((int)x[((int64_t)n * HW + hw) * Cp + c] - zp);
    if (dst_bf16) reinterpret_cast<bf16_t*>(y)[i] = f32_to_bf16(v);
    else reinterpret_cast<float*>(y)[i] = v;
  }
}

// One thread per (n, p, q, 16-channel group): bytewise maximum over the
// window's taps inside the image.
__global__ __launch_bounds__(kThreads) void maxpool_i8_kernel(PoolParams p) {
  const int G = p.Cp / 16;
  const int total = p.N * p.P * p.Q * G;  // < 2^31 / 16: bytes of the output
  const int8_t* x = reinterpret_cast<const int8_t*>(p.x);
  int8_t* y = reinterpret_cast<int8_t*>(p.y);
  for (int i = blockIdx.x * kThreads + threadIdx.x; i < total; i += gridDim.x * kThreads) {
    const int g = i % G;
    const int pix = i / G;
    const int qq = pix % p.Q;
    const int pq = pix / p.Q;
    const int pp = pq % p.P;
    const int n = pq / p.P;
    int m[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) m[j] = -128;
    for (int r = 0; r < p.R; ++r) {
      const int ih = pp * p.sh - p.pt + r;
      if ((unsigned)ih >= (unsigned)p.H) continue;
      for (int s = 0; s < p.S; ++s) {
        const int iw = qq * p.sw - p.pl + s;
        if ((unsigned)iw >= (unsigned)p.W) continue;
        const uint4 u = *(const uint4*)(x + (((int64_t)n * p.H + ih) * p.W + iw) * p.Cp + g * 16);
        const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int j = 0; j < 16; ++j) m[j] = max(m[j], (int)(int8_t)(w4[j >> 2] >> (8 * (j & 3))));
      }
    }
    uint32_t o[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < 16; ++j) o[j >> 2] |= ((uint32_t)m[j] & 0xFFu) << (8 * (j & 3));
    *(uint4*)(y + (int64_t)i * 16) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// One thread per (n, p, q, 16-channel group): exact integer taps, 16 codes
// per 16-byte load of activations and of weights.  Blocks of kThreads
// threads in XCD-contiguous order (the hardware deals workgroups
// round-robin to the 8 XCDs; XCD x takes blocks [x * per_xcd, (x + 1) *
// per_xcd)), so neighbouring rows, which share the taps' input rows, are
// fetched through one L2.
__global__ __launch_bounds__(kThreads) void depthwise_i8_kernel(QDwParams p, int per_xcd) {
  const int G = p.Cp / 16;
  const int total = p.N * p.P * p.Q * G;  // < 2^31 / 16: bytes of the output
  const int i = ((blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3)) * kThreads + threadIdx.x;
  if (i < total) {
    const int g = i % G;
    const int pix = i / G;
    const int qq = pix % p.Q;
    const int pq = pix / p.Q;
    const int pp = pq % p.P;
    const int n = pq / p.P;
    int acc[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[j] = 0;
    for (int r = 0; r < p.R; ++r) {
      const int ih = pp * p.sh - p.pt + r;
      if ((unsigned)ih >= (unsigned)p.H) continue;
      for (int s = 0; s < p.S; ++s) {
        const int iw = qq * p.sw - p.pl + s;
        if ((unsigned)iw >= (unsigned)p.W) continue;
        const uint4 xv = *(const uint4*)(p.x + (((int64_t)n * p.H + ih) * p.W + iw) * p.Cp + g * 16);
        const uint4 wv = *(const uint4*)(p.w + (int64_t)(r * p.S + s) * p.Cp + g * 16);
        const uint32_t xw[4] = {xv.x, xv.y, xv.z, xv.w}, ww[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
        for (int j = 0; j < 16; ++j)
          acc[j] += ((int)(int8_t)(xw[j >> 2] >> (8 * (j & 3))) - p.zx) * (int)(int8_t)(ww[j >> 2] >> (8 * (j & 3)));
      }
    }
    uint32_t rw[4] = {0u, 0u, 0u, 0u};
    if (p.res) {
      const uint4 rv = *(const uint4*)(p.res + (int64_t)pix * p.Cp + g * 16);
      rw[0] = rv.x, rw[1] = rv.y, rw[2] = rv.z, rw[3] = rv.w;
    }
    const int2* qc = reinterpret_cast<const int2*>(p.qch) + g * 16;
    uint32_t o[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int2 q = qc[j];
      int v = p.zy + rescale(acc[j] + q.x, __int_as_float(q.y));
      if (p.res) v += rescale((int)(int8_t)(rw[j >> 2] >> (8 * (j & 3))) - p.zr, p.mr);
      if (p.leaky) v = leaky_code(v, p.zy, p.slope);
      v = min(max(v, p.lo), p.hi);
      o[j >> 2] |= ((uint32_t)v & 0xFFu) << (8 * (j & 3));
    }
    *(uint4*)(p.y + (int64_t)pix * p.Cp + g * 16) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// Global average pool of codes.  Workgroup = one image x 32 groups of 16
// channels; the 8 lanes of a group are consecutive, lane j sums pixels j,
// j + 8, ... (16-byte loads, eight in flight), then the 8 partial sums meet
// in a butterfly.  Integer sums: exact, so the order does not matter.
__global__ __launch_bounds__(kThreads) void avgpool_i8_kernel(PoolParams p, int zx, int zy, float m) {
  const int G = p.Cp / 16;
  const int n = blockIdx.x;
  const int pl = threadIdx.x & 7;
  const int g = blockIdx.y * (kThreads / 8) + (threadIdx.x >> 3);
  const int HW = p.H * p.W;
  const bool ok = g < G;
  const int8_t* x = reinterpret_cast<const int8_t*>(p.x) + (size_t)n * HW * p.Cp + (size_t)(ok ? g : 0) * 16;
  int acc[16];
#pragma unroll
  for (int c = 0; c < 16; ++c) acc[c] = 0;
  for (int i0 = 0; i0 < HW; i0 += 64) {
    uint4 u[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int i = i0 + pl + 8 * j;
      u[j] = *(const uint4*)(x + (size_t)(i < HW ? i : 0) * p.Cp);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (i0 + pl + 8 * j >= HW) continue;
      const uint32_t w[4] = {u[j].x, u[j].y, u[j].z, u[j].w};
#pragma unroll
      for (int c = 0; c < 16; ++c) acc[c] += (int)(int8_t)(w[c >> 2] >> (8 * (c & 3)));
    }
  }
#pragma unroll
  for (int o = 1; o < 8; o <<= 1)
#pragma unroll
    for (int c = 0; c < 16; ++c) acc[c] += __shfl_xor(acc[c], o);
  if (ok && pl == 0) {
    uint32_t o4[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int c = 0; c < 16; ++c) {
      const int v = clip_i8(zy + rescale(acc[c] - HW * zx, m));
      o4[c >> 2] |= ((uint32_t)v & 0xFFu) << (8 * (c & 3));
    }
    *(uint4*)(reinterpret_cast<int8_t*>(p.y) + (size_t)n * p.Cp + g * 16) = make_uint4(o4[0], o4[1], o4[2], o4[3]);
  }
}

// 16 codes per thread.
__global__ __launch_bounds__(kThreads) void add_i8_kernel(QAddParams p) {
  const int64_t groups = p.n / 16;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < groups; i += (int64_t)gridDim.x * kThreads) {
    const uint4 ua = *(const uint4*)(p.a + i * 16), ub = *(const uint4*)(p.b + i * 16);
    const uint32_t wa[4] = {ua.x, ua.y, ua.z, ua.w}, wb[4] = {ub.x, ub.y, ub.z, ub.w};
    uint32_t o[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int a = (int)(int8_t)(wa[j >> 2] >> (8 * (j & 3)));
      const int b = (int)(int8_t)(wb[j >> 2] >> (8 * (j & 3)));
      int v = p.zy + rescale(a - p.za, p.ma) + rescale(b - p.zb, p.mb);
      if (p.leaky) v = leaky_code(v, p.zy, p.slope);
      v = min(max(v, p.lo), p.hi);
      o[j >> 2] |= ((uint32_t)v & 0xFFu) << (8 * (j & 3));
    }
    *(uint4*)(p.y + i * 16) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

}  // namespace

hipError_t launch_quantize_i8(const void* x, bool src_bf16, int8_t* y, int N, int C, int H, int W, int Cp,
                              float inv_scale, int zp, hipStream_t s) {
  if (Cp % 16 != 0 || Cp < C) return hipErrorInvalidValue;
  quantize_kernel<<<grid_for((int64_t)N * (Cp / 16) * H * W), kThreads, 0, s>>>(x, src_bf16 ? 1 : 0, y, N, C, H, W,
                                                                                 Cp, inv_scale, zp);
  return hipGetLastError();
}

hipError_t launch_quantize_im2col_i8(const void* x, bool src_bf16, int8_t* y, const PoolParams& g, float inv_scale,
                                     int zp, hipStream_t s) {
  if (g.Cp % 16 != 0 || g.Cp < g.R * g.S * 4 || g.C > 4 || g.R * g.W * 4 > kIm2colLds) return hipErrorInvalidValue;
  quantize_im2col_kernel<<<g.N * g.P, kThreads, g.R * g.W * 4, s>>>(
      x, src_bf16 ? 1 : 0, y, g, inv_scale, zp);
  return hipGetLastError();
}

hipError_t launch_dequantize_i8(const int8_t* x, void* y, bool dst_bf16, int N, int C, int H, int W, int Cp,
                                float scale, int zp, hipStream_t s) {
  if (Cp < C) return hipErrorInvalidValue;
  dequantize_kernel<<<grid_for((int64_t)N * C * H * W), kThreads, 0, s>>>(x, y, dst_bf16 ? 1 : 0, N, C, H, W, Cp,
                                                                          scale, zp);
  return hipGetLastError();
}

hipError_t launch_depthwise_i8(const QDwParams& p, hipStream_t s) {
  if (p.Cp % 16 != 0) return hipErrorInvalidValue;
  const int per_xcd = (int)((grid_for((int64_t)p.N * p.P * p.Q * (p.Cp / 16)) + 7) / 8);
  depthwise_i8_kernel<<<8u * (unsigned)per_xcd, kThreads, 0, s>>>(p, per_xcd);
  return hipGetLastError();
}

hipError_t launch_maxpool_nhwc_i8(const PoolParams& p, hipStream_t s) {
  if (p.Cp % 16 != 0) return hipErrorInvalidValue;
  maxpool_i8_kernel<<<grid_for((int64_t)p.N * p.P * p.Q * (p.Cp / 16)), kThreads, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_avgpool_nhwc_i8(const PoolParams& p, int zx, int zy, float m, hipStream_t s) {
  if (p.Cp % 16 != 0) return hipErrorInvalidValue;
  avgpool_i8_kernel<<<dim3(p.N, (p.Cp / 16 + kThreads / 8 - 1) / (kThreads / 8)), kThreads, 0, s>>>(p, zx, zy, m);
  return hipGetLastError();
}

hipError_t launch_add_i8(const QAddParams& p, hipStream_t s) {
  if (p.n % 16 != 0) return hipErrorInvalidValue;
  add_i8_kernel<<<grid_for(p.n / 16), kThreads, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace byoc
