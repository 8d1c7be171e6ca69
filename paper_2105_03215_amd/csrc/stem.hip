// Fused network stem: convolution of an NCHW graph input with few channels
// (C <= 4) + bias + activation, followed by max pooling, in one kernel.
//
// The composites are the conv2d + bias + activation and max-pool operators
// of the offloaded graph (Sec. 3.1.1); fusing them inside the codegen keeps
// the full-resolution conv output (e.g. 32x112x112x64 for a ResNet stem) out
// of HBM, and reading the NCHW input directly removes the layout transform
// (Sec. 3.2) that the input would otherwise need.  Values are those of the
// unfused chain: each conv output is rounded to bf16 before the pooling max.
//
// Workgroup: 256 threads, one 8x8 tile of pooled outputs x 64 channels.  It
// computes the (7*sp + kp)^2 conv outputs the tile's windows cover (at most
// 17x17 for a 3x3 / stride-2 pool), so neighbouring tiles recompute a border
// of one conv row and column.
//  1. The input patch those conv outputs read is staged in LDS as
//     [row][col][4 channels] bf16 (zero outside the image), the packed
//     weights as [64][R*32 + 8].
//  2. Implicit GEMM on v_mfma_f32_16x16x32_bf16: one 32-element reduction
//     step per kernel row r, ordered (tap s < 8, channel c < 4); a lane's 8
//     reduction elements are taps 2g and 2g+1 of its conv pixel, i.e. two
//     adjacent 8-byte patch cells.  Weights are the A operand, pixels B.
//  3. Bias, activation and bf16 rounding; the results go to an LDS tile
//     (conv outputs outside the image as -inf, which never win the max).
//  4. Each thread pools 8 channels of a pooled pixel and stores 16 bytes
//     of the NHWC output.
#include "device_common.h"

namespace byoc {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr int kThreads = 256;
constexpr int kPI = 8, kPJ = 8;  // pooled outputs per tile
constexpr int kCMax = 17;        // conv rows / cols per tile (7 * 2 + 3)
constexpr int kPatch = 40;       // patch rows / cols: (kCMax - 1) * 2 + 8
constexpr int kK = 64;           // output channels
constexpr int kTileLd = kK + 8;  // conv tile row (bf16): 144 bytes, 16 rows on distinct banks
constexpr int kFrags = (kCMax * kCMax + 15) / 16;  // 16-pixel MFMA tiles (19)
constexpr int kFragsPerWave = (kFrags + 3) / 4;    // 5
constexpr int kPatchBytes = kPatch * kPatch * 8;
constexpr int kWeightLdMax = 8 * 32 + 8;
constexpr int kLdsBytes = kPatchBytes + kK * kWeightLdMax * 2;  // >= conv tile bytes
static_assert(kCMax * kCMax * kTileLd * 2 <= kLdsBytes, "conv tile overlays patch + weights");

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

__device__ __forceinline__ uint16_t in_bf16(const void* x, bool bf, size_t i) {
  return bf ? ((const uint16_t*)x)[i] : f32_to_bf16(((const float*)x)[i]);
}

__global__ __launch_bounds__(kThreads) void stem_conv_maxpool_kernel(StemParams p) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[kLdsBytes];
  uint2* patch = reinterpret_cast<uint2*>(lds);                           // [kPatch][kPatch] cells
  bf16_t* wl = reinterpret_cast<bf16_t*>(lds + kPatchBytes);              // [64][wld]
  bf16_t* tile = reinterpret_cast<bf16_t*>(lds);                          // [CR*CC][kTileLd] (after the GEMM)

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tj = blockIdx.x, ti = blockIdx.y, n = blockIdx.z;
  const int g = lane >> 4;
  // bias of the 16 channels this lane finishes (fetched first: used last)
  float4 bv[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
    bv[j] = p.bias ? *reinterpret_cast<const float4*>(p.bias + j * 16 + 4 * g) : make_float4(0.f, 0.f, 0.f, 0.f);
  const int CR = (kPI - 1) * p.sph + p.kph;  // conv rows / cols of the tile
  const int CC = (kPJ - 1) * p.spw + p.kpw;
  const int cr0 = ti * kPI * p.sph - p.ppt;  // global conv row / col of local (0, 0)
  const int cc0 = tj * kPJ * p.spw - p.ppl;
  const int ir0 = cr0 * p.sh - p.pt;         // global input row / col of patch (0, 0)
  const int ic0 = cc0 * p.sw - p.pl;
  const int IR = (CR - 1) * p.sh + p.R;
  const int IC = (CC - 1) * p.sw + 8;

  // 1. weights (16-byte chunks) and input patch; every load of a thread is
  // issued before the first LDS write so their latencies overlap
  {
    constexpr int kWChunks = (kK * kWeightLdMax / 8 + kThreads - 1) / kThreads;
    const uint4* src = reinterpret_cast<const uint4*>(p.w);
    uint4* dst = reinterpret_cast<uint4*>(wl);
    const int chunks = kK * p.wld / 8;
    uint4 wv[kWChunks];
#pragma unroll
    for (int i = 0; i < kWChunks; ++i) {
      const int idx = tid + i * kThreads;
      wv[i] = src[idx < chunks ? idx : 0];
    }
#pragma unroll
    for (int i = 0; i < kWChunks; ++i) {
      const int idx = tid + i * kThreads;
      if (idx < chunks) dst[idx] = wv[i];
    }
  }
  {
    constexpr int kCells = (kPatch * kPatch + kThreads - 1) / kThreads;
    const bool bf = p.x_bf16 != 0;
    const size_t plane = (size_t)p.H * p.W;
    const size_t img = (size_t)n * p.C * plane;
    uint2 cell[kCells];
#pragma unroll
    for (int k = 0; k < kCells; ++k) {
      const int i = tid + k * kThreads;
      const int rr = i / IC, cc = i - (i / IC) * IC;
      const int ih = ir0 + rr, iw = ic0 + cc;
      const bool ok = i < IR * IC && (unsigned)ih < (unsigned)p.H && (unsigned)iw < (unsigned)p.W;
      const size_t o = img + (size_t)ih * p.W + iw;
      const uint32_t c0 = ok ? in_bf16(p.x, bf, o) : 0u;
      const uint32_t c1 = (ok && p.C > 1) ? in_bf16(p.x, bf, o + plane) : 0u;
      const uint32_t c2 = (ok && p.C > 2) ? in_bf16(p.x, bf, o + 2 * plane) : 0u;
      const uint32_t c3 = (ok && p.C > 3) ? in_bf16(p.x, bf, o + 3 * plane) : 0u;
      cell[k] = make_uint2(c0 | (c1 << 16), c2 | (c3 << 16));
    }
#pragma unroll
    for (int k = 0; k < kCells; ++k) {
      const int i = tid + k * kThreads;
      if (i >= IR * IC) break;
      const int rr = i / IC, cc = i - (i / IC) * IC;
      patch[rr * kPatch + cc] = cell[k];
    }
  }
  __syncthreads();

  // 2. implicit GEMM: this wave owns pixel tiles wave, wave + 4, ...
  const int npix = CR * CC;
  int pbase[kFragsPerWave];  // patch cell of this lane's pixel at tap (0, 0)
#pragma unroll
  for (int i = 0; i < kFragsPerWave; ++i) {
    int m = (wave + 4 * i) * 16 + (lane & 15);
    if (m >= npix) m = 0;  // padding rows of the last tile: any valid address
    const int lr = m / CC, lc = m - (m / CC) * CC;
    pbase[i] = lr * p.sh * kPatch + lc * p.sw + 2 * g;
  }
  f32x4 acc[kFragsPerWave][4];
#pragma unroll
  for (int i = 0; i < kFragsPerWave; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    if (r >= p.R) break;
    bf16x8 a[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      a[j] = as_bf16x8(*reinterpret_cast<const uint4*>(wl + (j * 16 + (lane & 15)) * p.wld + r * 32 + g * 8));
#pragma unroll
    for (int i = 0; i < kFragsPerWave; ++i) {  // a wave's surplus tile computes discarded values
      const uint2 t0 = patch[pbase[i] + r * kPatch];
      const uint2 t1 = patch[pbase[i] + r * kPatch + 1];
      const bf16x8 b = as_bf16x8(make_uint4(t0.x, t0.y, t1.x, t1.y));
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[j], b, acc[i][j], 0, 0, 0);
    }
  }
  __syncthreads();  // patch and weights are dead: the conv tile overlays them

  // 3. bias, activation, bf16; conv outputs outside the image -> -inf
  const ActClamp ac = act_clamp_of(p.act);
  auto epilogue = [&](auto gelu_tag) {
    constexpr bool G = decltype(gelu_tag)::value;
#pragma unroll
    for (int i = 0; i < kFragsPerWave; ++i) {
      if (wave + 4 * i >= kFrags) break;
      const int m = (wave + 4 * i) * 16 + (lane & 15);
      if (m >= npix) continue;
      const int lr = m / CC, lc = m - (m / CC) * CC;
      const bool inside = (unsigned)(cr0 + lr) < (unsigned)p.P && (unsigned)(cc0 + lc) < (unsigned)p.Q;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        uint2 o;
        if (inside) {
          const f32x4 v = acc[i][j];
          o = make_uint2(pack2_bf16(act_apply<G>(v[0] + bv[j].x, ac), act_apply<G>(v[1] + bv[j].y, ac)),
                         pack2_bf16(act_apply<G>(v[2] + bv[j].z, ac), act_apply<G>(v[3] + bv[j].w, ac)));
        } else {
          o = make_uint2(0xFF80FF80u, 0xFF80FF80u);  // bf16 -inf
        }
        *reinterpret_cast<uint2*>(tile + m * kTileLd + j * 16 + 4 * g) = o;
      }
    }
  };
  if (p.act == kActGelu)
    epilogue(std::true_type{});
  else
    epilogue(std::false_type{});
  __syncthreads();

  // 4. pooling: 64 pooled pixels x 8 channel groups, two per thread
  for (int it = tid; it < kPI * kPJ * (kK / 8); it += kThreads) {
    const int c8 = (it & 7) * 8;
    const int pi = (it >> 3) / kPJ, pj = (it >> 3) % kPJ;
    const int po = ti * kPI + pi, qo = tj * kPJ + pj;
    if (po >= p.PO || qo >= p.QO) continue;
    float mx[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) mx[e] = -INFINITY;
    uint4 win[3][3];  // all window reads issued before the first max
#pragma unroll
    for (int dr = 0; dr < 3; ++dr)
#pragma unroll
      for (int dc = 0; dc < 3; ++dc) {
        const int m = (pi * p.sph + (dr < p.kph ? dr : 0)) * CC + pj * p.spw + (dc < p.kpw ? dc : 0);
        win[dr][dc] = *reinterpret_cast<const uint4*>(tile + m * kTileLd + c8);
      }
#pragma unroll
    for (int dr = 0; dr < 3; ++dr)
#pragma unroll
      for (int dc = 0; dc < 3; ++dc) {
        float v[8];
        unpack8(win[dr][dc], v);  // taps past the window repeat its first one: no effect on the max
#pragma unroll
        for (int e = 0; e < 8; ++e) mx[e] = fmaxf(mx[e], v[e]);
      }
    *reinterpret_cast<uint4*>(p.y + (((size_t)n * p.PO + po) * p.QO + qo) * kK + c8) = pack8(mx);
  }
}

// Packs conv weights [64][C][R][S] (f32 or bf16) into [64][wld] bf16 with
// column r*32 + s*4 + c, zero for s >= S, c >= C and the row padding.
__global__ void pack_stem_weights_kernel(const void* src, int src_bf16, bf16_t* dst, int C, int R, int S,
                                         int wld) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= kK * wld) return;
  const int k = i / wld, col = i - (i / wld) * wld;
  const int r = col / 32, s = (col % 32) / 4, c = col % 4;
  bf16_t v = 0;
  if (r < R && s < S && c < C) {
    const size_t o = (((size_t)k * C + c) * R + r) * S + s;
    v = src_bf16 ? ((const bf16_t*)src)[o] : f32_to_bf16(((const float*)src)[o]);
  }
  dst[i] = v;
}

}  // namespace

bool stem_supported(int C, int K, int R, int S, int sh, int sw, int kph, int kpw, int sph, int spw) {
  return C >= 1 && C <= 4 && K == kK && R >= 1 && R <= 8 && S >= 1 && S <= 8 && sh >= 1 && sh <= 2 &&
         sw >= 1 && sw <= 2 && kph >= 1 && kph <= 3 && kpw >= 1 && kpw <= 3 && sph >= 1 && sph <= 2 &&
         spw >= 1 && spw <= 2;
}

int stem_weight_ld(int R) { return R * 32 + 8; }

hipError_t launch_stem_conv_maxpool(const StemParams& p, hipStream_t s) {
  dim3 grid((p.QO + kPJ - 1) / kPJ, (p.PO + kPI - 1) / kPI, p.N);
  stem_conv_maxpool_kernel<<<grid, kThreads, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_pack_stem_weights(const void* src, bool src_bf16, bf16_t* dst, int C, int R, int S, int wld,
                                    hipStream_t s) {
  const int n = kK * wld;
  pack_stem_weights_kernel<<<(n + 255) / 256, 256, 0, s>>>(src, src_bf16 ? 1 : 0, dst, C, R, S, wld);
  return hipGetLastError();
}

}  // namespace byoc
