// fp32 convolution for fp32 graphs: direct NCHW evaluation of the conv
// composite, one thread per output, fused multiply-adds in fp32 over the
// reduction in (c, r, s) order, then bias, residual, activation.  Dense runs
// as the 1x1 case on [M, K, 1, 1].  These graphs are small (the fp32 path
// exists for exactness, not throughput); consecutive threads take
// consecutive output columns so input rows are read contiguously.
#include "device_common.h"

namespace byoc {
namespace {

__global__ __launch_bounds__(256) void conv_f32_kernel(ConvF32Params p) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t total = (int64_t)p.N * p.K * p.P * p.Q;
  if (idx >= total) return;
  const int q = (int)(idx % p.Q);
  int64_t t = idx / p.Q;
  const int pp = (int)(t % p.P);
  t /= p.P;
  const int k = (int)(t % p.K);
  const int n = (int)(t / p.K);
  const int cg = p.C / p.groups;
  const int kg = p.K / p.groups;
  const int g = k / kg;
  const int ih0 = pp * p.sh - p.pt;
  const int iw0 = q * p.sw - p.pl;
  float acc = 0.f;
  for (int c = 0; c < cg; ++c) {
    const float* xc = p.x + ((size_t)n * p.C + g * cg + c) * p.H * p.W;
    const float* wc = p.w + ((size_t)k * cg + c) * p.R * p.S;
    for (int r = 0; r < p.R; ++r) {
      const int ih = ih0 + r;
      if ((unsigned)ih >= (unsigned)p.H) continue;
      for (int s = 0; s < p.S; ++s) {
        const int iw = iw0 + s;
        if ((unsigned)iw >= (unsigned)p.W) continue;
        acc = fmaf(xc[ih * p.W + iw], wc[r * p.S + s], acc);
      }
    }
  }
  if (p.bias) acc += p.bias[k];
  if (p.res) acc += p.res[idx];
  p.y[idx] = apply_act(acc, p.act, p.alpha);
}

// Register-blocked form for groups == 1 and RxS taps known at compile
// time: one thread per output pixel computes KB output channels; the
// channel block is uniform over the workgroup (grid y), so its weights come
// through scalar loads shared by the wave, and the taps of two input
// channels are loaded at once.  Each output sums its terms in the order of
// the kernel above - channel, kernel row, column - from zero (a tap outside
// the image adds an exact zero), then bias, residual and activation.
constexpr int kKB = 4;

template <int R, int S>
__global__ __launch_bounds__(64) void conv_f32_regs_kernel(ConvF32Params p) {
  const int nkb = (p.K + kKB - 1) / kKB;
  const int n = blockIdx.y / nkb;
  const int k0 = (blockIdx.y - n * nkb) * kKB;
  const int pix = blockIdx.x * 64 + threadIdx.x;
  const bool live = pix < p.P * p.Q;
  const int pp = live ? pix / p.Q : 0;
  const int q = live ? pix - pp * p.Q : 0;
  const int ih0 = pp * p.sh - p.pt, iw0 = q * p.sw - p.pl;
  const int HW = p.H * p.W;
  // taps inside the image (offsets within a channel plane)
  int off[R * S];
  bool in[R * S];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int t = 0; t < S; ++t) {
      const int ih = ih0 + r, iw = iw0 + t;
      in[r * S + t] = live && (unsigned)ih < (unsigned)p.H && (unsigned)iw < (unsigned)p.W;
      off[r * S + t] = in[r * S + t] ? ih * p.W + iw : 0;
    }
  const float* xn = p.x + (size_t)n * p.C * HW;
  const float* wk[kKB];
#pragma unroll
  for (int j = 0; j < kKB; ++j) wk[j] = p.w + (size_t)min(k0 + j, p.K - 1) * p.C * R * S;
  float acc[kKB];
#pragma unroll
  for (int j = 0; j < kKB; ++j) acc[j] = 0.f;
  auto tap_sum = [&](int c, const float* xv) {
#pragma unroll
    for (int t = 0; t < R * S; ++t)
#pragma unroll
      for (int j = 0; j < kKB; ++j) acc[j] = fmaf(xv[t], wk[j][c * R * S + t], acc[j]);
  };
  int c = 0;
  for (; c + 2 <= p.C; c += 2) {
    float xa[R * S], xb[R * S];
    const float* xc = xn + (size_t)c * HW;
#pragma unroll
    for (int t = 0; t < R * S; ++t) {
      xa[t] = in[t] ? xc[off[t]] : 0.f;
      xb[t] = in[t] ? xc[HW + off[t]] : 0.f;
    }
    tap_sum(c, xa);
    tap_sum(c + 1, xb);
  }
  if (c < p.C) {
    float xa[R * S];
    const float* xc = xn + (size_t)c * HW;
#pragma unroll
    for (int t = 0; t < R * S; ++t) xa[t] = in[t] ? xc[off[t]] : 0.f;
    tap_sum(c, xa);
  }
  if (!live) return;
#pragma unroll
  for (int j = 0; j < kKB; ++j) {
    const int k = k0 + j;
    if (k >= p.K) break;
    const size_t o = (((size_t)n * p.K + k) * p.P + pp) * p.Q + q;
    float v = acc[j];
    if (p.bias) v += p.bias[k];
    if (p.res) v += p.res[o];
    p.y[o] = apply_act(v, p.act, p.alpha);
  }
}

}  // namespace

hipError_t launch_conv_f32(const ConvF32Params& p, hipStream_t s) {
  const int64_t total = (int64_t)p.N * p.K * p.P * p.Q;
  if (total == 0) return hipSuccess;
  const int64_t gy = (int64_t)p.N * ((p.K + kKB - 1) / kKB);
  const int64_t pix = (int64_t)p.P * p.Q;
  const bool regs = p.groups == 1 && gy <= 65535 && pix < (int64_t(1) << 30) &&
                    (int64_t)p.C * p.H * p.W < (int64_t(1) << 31);
  if (regs && p.R == 3 && p.S == 3) {
    conv_f32_regs_kernel<3, 3><<<dim3((unsigned)((pix + 63) / 64), (unsigned)gy), 64, 0, s>>>(p);
    return hipGetLastError();
  }
  if (regs && p.R == 1 && p.S == 1) {
    conv_f32_regs_kernel<1, 1><<<dim3((unsigned)((pix + 63) / 64), (unsigned)gy), 64, 0, s>>>(p);
    return hipGetLastError();
  }
  conv_f32_kernel<<<(unsigned)((total + 255) / 256), 256, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace byoc
