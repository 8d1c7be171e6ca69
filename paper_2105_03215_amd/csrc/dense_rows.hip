// Dense composite (dense + bias + activation [+ residual], Sec. 3.1.1) for
// few rows: y[m][n] = act(sum_k x[m][k] w[n][k] + b[n] (+ r[m][n])) with
// M <= 64 rows, e.g. the classifier of an image network at small batch.
//
// The conv kernels tile rows x channels and would leave most of the chip
// idle here (a handful of tiles), or need a split-K pass with a separate
// reduction launch.  Instead one workgroup owns 16 output channels and all
// rows, and splits the reduction across its 16 waves: wave w takes the
// 32-element k-steps w, w + 16, ...; every load is issued before the
// MFMAs that use it.  The waves' partial sums meet in LDS and are added in
// wave order (run-to-run identical), then bias, residual and activation
// are applied and bf16 rows are stored.
//
// MFMA v_mfma_f32_16x16x32_bf16 with the weights as the A operand (16
// channels) and the rows as B (16 rows per MFMA tile), so a lane ends up
// with 4 consecutive channels of one row.
#include "device_common.h"

namespace byoc {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr int kWaves = 16;
constexpr int kThreads = 64 * kWaves;
constexpr int kUnroll = 8;  // k-steps per wave with loads in flight together

template <int MT>  // 16-row MFMA tiles: ceil(M / 16)
__global__ __launch_bounds__(kThreads) void dense_rows_kernel(ConvParams p) {
  __shared__ f32x4 red[kWaves][MT][64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n0 = blockIdx.x * 16;
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(p.x), (short)0, p.x_bytes, kBufferFlags);
  const __amdgpu_buffer_rsrc_t wr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(p.w), (short)0, p.w_bytes, kBufferFlags);
  const int nk = p.Kgp / 32;
  // lane l: 16 bytes (8 reduction elements, chunk l / 16) of weight row
  // n0 + l % 16 and of input row mt * 16 + l % 16; rows past M read zeros
  const uint32_t woff = (uint32_t)(((n0 + (lane & 15)) * p.Kgp + (lane >> 4) * 8) * 2);
  uint32_t xoff[MT];
  bool xin[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = mt * 16 + (lane & 15);
    xin[mt] = m < p.M;
    xoff[mt] = xin[mt] ? (uint32_t)((m * p.Cp + (lane >> 4) * 8) * 2) : 0u;
  }
  f32x4 acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int t0 = wave; t0 < nk; t0 += kWaves * kUnroll) {
    uint4 a[kUnroll], b[kUnroll][MT];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int t = t0 + u * kWaves;
      const bool live = t < nk;
      // k-step t covers elements 32 t .. 32 t + 31 (64 bytes); the weight
      // rows' padding past Kg is zero, so the input may read past its row
      // there (the last row's overrun reads zeros from the buffer range)
      a[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(wr, live ? woff + t * 64u : kOOB, 0, 0));
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        b[u][mt] = __builtin_bit_cast(
            uint4, __builtin_amdgcn_raw_buffer_load_b128(xr, live && xin[mt] ? xoff[mt] + t * 64u : kOOB, 0, 0));
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (t0 + u * kWaves >= nk) break;  // uniform per wave
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a[u]),
                                                          __builtin_bit_cast(bf16x8, b[u][mt]), acc[mt], 0, 0, 0);
    }
  }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) red[wave][mt][lane] = acc[mt];
  __syncthreads();

  // output (row m, channels n0 + 4q .. + 3) sits in lane q * 16 + m % 16 of
  // MFMA tile m / 16 of every wave
  if (tid >= MT * 16 * 4) return;
  const int m = tid >> 2, q = tid & 3;
  const int n = n0 + 4 * q;
  if (m >= p.M || n >= p.Kp) return;
  f32x4 s = red[0][m >> 4][q * 16 + (m & 15)];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) s += red[w][m >> 4][q * 16 + (m & 15)];
  float v[4] = {s[0], s[1], s[2], s[3]};
  if (p.bias) {
    const float4 bb = *reinterpret_cast<const float4*>(p.bias + n);
    v[0] += bb.x, v[1] += bb.y, v[2] += bb.z, v[3] += bb.w;
  }
  if (p.res) {
    const uint2 r = *reinterpret_cast<const uint2*>(p.res + (size_t)m * p.ldr + n);
    v[0] += bf16_to_f32((bf16_t)(r.x & 0xFFFF)), v[1] += bf16_to_f32((bf16_t)(r.x >> 16));
    v[2] += bf16_to_f32((bf16_t)(r.y & 0xFFFF)), v[3] += bf16_to_f32((bf16_t)(r.y >> 16));
  }
  const ActClamp ac = act_clamp_of(p.act, p.alpha);
  if (p.act == kActGelu) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = act_apply<true>(v[e], ac);
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = act_apply<false>(v[e], ac);
  }
  *reinterpret_cast<uint2*>(p.y + (size_t)m * p.ldy + n) = make_uint2(pack2_bf16(v[0], v[1]), pack2_bf16(v[2], v[3]));
}

}  // namespace

bool dense_rows_supported(const ConvParams& p) {
  return p.M >= 1 && p.M <= 64 && p.R == 1 && p.S == 1 && p.H == 1 && p.W == 1 && p.P == 1 && p.Q == 1 &&
         p.splits == 1 && p.Kp % 4 == 0 && p.Kgp % 64 == 0;
}

hipError_t launch_dense_rows(const ConvParams& p, hipStream_t s) {
  if (!dense_rows_supported(p)) return hipErrorInvalidValue;
  const dim3 grid((p.Kp + 15) / 16);
  switch ((p.M + 15) / 16) {
    case 1: dense_rows_kernel<1><<<grid, kThreads, 0, s>>>(p); break;
    case 2: dense_rows_kernel<2><<<grid, kThreads, 0, s>>>(p); break;
    case 3: dense_rows_kernel<3><<<grid, kThreads, 0, s>>>(p); break;
    default: dense_rows_kernel<4><<<grid, kThreads, 0, s>>>(p); break;
  }
  return hipGetLastError();
}

}  // namespace byoc
