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

}  // namespace

hipError_t launch_conv_f32(const ConvF32Params& p, hipStream_t s) {
  const int64_t total = (int64_t)p.N * p.K * p.P * p.Q;
  conv_f32_kernel<<<(unsigned)((total + 255) / 256), 256, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace byoc
