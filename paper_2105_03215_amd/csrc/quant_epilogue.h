// The int8 conv epilogue shared by the implicit-GEMM and the windowed (halo)
// int8 kernels: 8 consecutive output channels k .. k + 7 of output pixel m
// from their int32 sums (Sec. 3.2: the requantization of a quantized conv).
#pragma once

#include "device_common.h"

namespace byoc {

// a[c] holds the sum of channel k + c over the taps inside the image of
// (x_q * w_q); qc[c] = {bias with -Z_x * sum(w) folded in, float32 factor
// bits} of channel k + c; rv the 8 residual (or folded add operand) codes.
// Returns the 8 output codes, packed little-endian.
__device__ __forceinline__ uint2 finish8_i8(int a[8], const int2* qc, uint2 rv, const QConvParams& q, int m,
                                           int k) {
  const ConvParams& p = q.g;
#pragma unroll
  for (int c8 = 0; c8 < 8; ++c8) a[c8] += qc[c8].x;
  if (q.wtap) {
    // window of this pixel: taps outside the image get Z_x * their weight sums back
    const int PQ = p.P * p.Q, RS = p.R * p.S;
    const int n = mdiv(m, p.mg_pq);
    const int pq = m - n * PQ;
    const int pp = mdiv(pq, p.mg_q);
    const int qq = pq - pp * p.Q;
    const int ih0 = pp * p.sh - p.pt, iw0 = qq * p.sw - p.pl;
    const bool inside = ih0 >= 0 && iw0 >= 0 && ih0 + p.R <= p.H && iw0 + p.S <= p.W;
    if (!inside) {
      // the table is tap-major: the 8 channels of one tap are two 16-byte loads
      int corr[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      auto add_tap = [&](int t) {
        const int4* wt = reinterpret_cast<const int4*>(q.wtap + (size_t)t * q.wtap_ld + k);
        const int4 lo = wt[0], hi = wt[1];
        corr[0] += lo.x, corr[1] += lo.y, corr[2] += lo.z, corr[3] += lo.w;
        corr[4] += hi.x, corr[5] += hi.y, corr[6] += hi.z, corr[7] += hi.w;
      };
      if (p.R == 3 && p.S == 3) {  // unrolled: the loads of all outside taps in flight together
#pragma unroll
        for (int t = 0; t < 9; ++t)
          if ((unsigned)(ih0 + t / 3) >= (unsigned)p.H || (unsigned)(iw0 + t % 3) >= (unsigned)p.W) add_tap(t);
      } else {
        for (int t = 0; t < RS; ++t) {
          const int rr = t / p.S, ss = t - rr * p.S;
          if ((unsigned)(ih0 + rr) >= (unsigned)p.H || (unsigned)(iw0 + ss) >= (unsigned)p.W) add_tap(t);
        }
      }
#pragma unroll
      for (int c8 = 0; c8 < 8; ++c8) a[c8] += q.zx * corr[c8];
    }
  }
  const uint32_t rw[2] = {rv.x, rv.y};
  uint32_t out[2] = {0u, 0u};
#pragma unroll
  for (int c8 = 0; c8 < 8; ++c8) {
    int v = q.zy + rescale(a[c8], __int_as_float(qc[c8].y));
    const int rc = (int)(int8_t)(rw[c8 >> 2] >> (8 * (c8 & 3)));
    if (p.res && !q.post) v += rescale(rc - q.zr, q.mr);
    if (q.leaky) v = leaky_code(v, q.zy, q.slope);
    v = min(max(v, q.lo), q.hi);
    if (q.post) v = clip_i8(q.pz + rescale(v - q.zy, q.pm) + rescale(rc - q.zr, q.mr));
    out[c8 >> 2] |= ((uint32_t)v & 0xFFu) << (8 * (c8 & 3));
  }
  return make_uint2(out[0], out[1]);
}

}  // namespace byoc
