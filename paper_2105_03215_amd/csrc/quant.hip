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
  const int64_t total = (int64_t)N * G * HW;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < total; i += (int64_t)gridDim.x * kThreads) {
    const int hw = (int)(i % HW);
    const int64_t ng = i / HW;
    const int g = (int)(ng % G);
    const int n = (int)(ng / G);
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

// One thread per output element (n, c, h, w), w fastest.
__global__ __launch_bounds__(kThreads) void dequantize_kernel(const int8_t* x, void* y, int dst_bf16, int N, int C,
                                                              int H, int W, int Cp, float scale, int zp) {
  const int HW = H * W;
  const int64_t total = (int64_t)N * C * HW;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < total; i += (int64_t)gridDim.x * kThreads) {
    const int hw = (int)(i % HW);
    const int64_t nc = i / HW;
    const int c = (int)(nc % C);
    const int n = (int)(nc / C);
    const float v = scale * (float)((int)x[((int64_t)n * HW + hw) * Cp + c] - zp);
    if (dst_bf16) reinterpret_cast<bf16_t*>(y)[i] = f32_to_bf16(v);
    else reinterpret_cast<float*>(y)[i] = v;
  }
}

// One thread per (n, p, q, 16-channel group): bytewise maximum over the
// window's taps inside the image.
__global__ __launch_bounds__(kThreads) void maxpool_i8_kernel(PoolParams p) {
  const int G = p.Cp / 16;
  const int64_t total = (int64_t)p.N * p.P * p.Q * G;
  const int8_t* x = reinterpret_cast<const int8_t*>(p.x);
  int8_t* y = reinterpret_cast<int8_t*>(p.y);
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < total; i += (int64_t)gridDim.x * kThreads) {
    const int g = (int)(i % G);
    const int64_t pix = i / G;
    const int qq = (int)(pix % p.Q);
    const int pp = (int)((pix / p.Q) % p.P);
    const int n = (int)(pix / ((int64_t)p.P * p.Q));
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
    *(uint4*)(y + i * 16) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// One thread per (n, channel): the integer sum over the image is exact.
__global__ __launch_bounds__(kThreads) void avgpool_i8_kernel(PoolParams p, int zx, int zy, float m) {
  const int64_t total = (int64_t)p.N * p.Cp;
  const int HW = p.H * p.W;
  const int8_t* x = reinterpret_cast<const int8_t*>(p.x);
  int8_t* y = reinterpret_cast<int8_t*>(p.y);
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < total; i += (int64_t)gridDim.x * kThreads) {
    const int c = (int)(i % p.Cp);
    const int n = (int)(i / p.Cp);
    const int8_t* src = x + (int64_t)n * HW * p.Cp + c;
    int sum = 0;
    for (int j = 0; j < HW; ++j) sum += (int)src[(int64_t)j * p.Cp] - zx;
    y[i] = (int8_t)clip_i8(zy + rescale(sum, m));
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
      const int v = min(max(p.zy + rescale(a - p.za, p.ma) + rescale(b - p.zb, p.mb), p.lo), p.hi);
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

hipError_t launch_dequantize_i8(const int8_t* x, void* y, bool dst_bf16, int N, int C, int H, int W, int Cp,
                                float scale, int zp, hipStream_t s) {
  if (Cp < C) return hipErrorInvalidValue;
  dequantize_kernel<<<grid_for((int64_t)N * C * H * W), kThreads, 0, s>>>(x, y, dst_bf16 ? 1 : 0, N, C, H, W, Cp,
                                                                          scale, zp);
  return hipGetLastError();
}

hipError_t launch_maxpool_nhwc_i8(const PoolParams& p, hipStream_t s) {
  if (p.Cp % 16 != 0) return hipErrorInvalidValue;
  maxpool_i8_kernel<<<grid_for((int64_t)p.N * p.P * p.Q * (p.Cp / 16)), kThreads, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_avgpool_nhwc_i8(const PoolParams& p, int zx, int zy, float m, hipStream_t s) {
  avgpool_i8_kernel<<<grid_for((int64_t)p.N * p.Cp), kThreads, 0, s>>>(p, zx, zy, m);
  return hipGetLastError();
}

hipError_t launch_add_i8(const QAddParams& p, hipStream_t s) {
  if (p.n % 16 != 0) return hipErrorInvalidValue;
  add_i8_kernel<<<grid_for(p.n / 16), kThreads, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace byoc
