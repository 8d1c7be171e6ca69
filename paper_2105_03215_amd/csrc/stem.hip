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
// Work unit ("tile"): one 8x8 block of pooled outputs x 64 channels of one
// image.  It needs the (7*sp + kp)^2 conv outputs its windows cover (at most
// 17x17 for a 3x3 / stride-2 pool), so neighbouring tiles recompute a border
// of one conv row and column.  Workgroups are persistent (two per CU, 256
// threads each) and stride over the tiles:
//  - the packed weights [64][R*32 + 8] are staged in LDS once;
//  - the input patch of a tile is staged in LDS as [row][col][4 channels]
//    bf16 cells (zero outside the image); the global loads of the next
//    tile's patch are issued at the end of a tile and land in registers
//    while the current tile computes;
//  - implicit GEMM on v_mfma_f32_16x16x32_bf16: one 32-element reduction
//    step per kernel row r, ordered (tap s < 8, channel c < 4); a lane's 8
//    reduction elements are taps 2g and 2g+1 of its conv pixel, i.e. two
//    adjacent patch cells.  Weights are the A operand, pixels B;
//  - bias, activation and bf16 rounding; the conv tile goes to LDS over the
//    dead patch (conv outputs outside the image as -inf, which never win
//    the max);
//  - each thread pools 8 channels of two pooled pixels; the 16-byte NHWC
//    stores go out after the next patch is in LDS.
// Barriers inside the tile loop wait on LDS only, so the patch loads in
// flight cross them.
#include "device_common.h"

#include <atomic>

namespace byoc {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr int kThreads = 256;
constexpr int kPI = 8, kPJ = 8;  // pooled outputs per tile
constexpr int kCMax = 17;        // conv rows / cols per tile (7 * 2 + 3)
constexpr int kPR = 40;          // patch rows: (kCMax - 1) * 2 + 8
constexpr int kPC = 48;          // patch cols: (kCMax - 1) * 2 + 8 + 3 (alignment offset), in 4-cell segments
constexpr int kSegs = kPC / 4;
constexpr int kUnits = (kPR * kSegs + kThreads - 1) / kThreads;  // (row, segment) units per thread
constexpr int kK = 64;           // output channels
constexpr int kTileLd = kK + 8;  // conv tile row (bf16): 144 bytes, 16 rows on distinct banks
constexpr int kFrags = (kCMax * kCMax + 15) / 16;  // 16-pixel MFMA tiles (19)
constexpr int kFragsPerWave = (kFrags + 3) / 4;    // 5
constexpr int kWeightLdMax = 8 * 32 + 8;
constexpr int kWeightBytes = kK * kWeightLdMax * 2;
constexpr int kPatchBytes = kPR * kPC * 8;
constexpr int kTileBytes = kCMax * kCMax * kTileLd * 2;
constexpr int kLdsBytes = kWeightBytes + (kPatchBytes > kTileBytes ? kPatchBytes : kTileBytes);
static_assert(2 * kLdsBytes <= 160 * 1024, "two workgroups per CU");

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

// Input values of one (patch row, 4-column segment) unit, per channel:
// 4 bf16 (XBF) or 4 f32.
template <bool XBF>
struct PatchRegs {
  using T = std::conditional_t<XBF, uint2, float4>;
  T v[kUnits][4];
};

// Issues the loads of a tile's patch (rows ir0.., columns ic0.. of image n).
// VEC: a segment is one vector load (W % 4 == 0 and ic0 % 4 == 0, so a
// segment is wholly inside or outside the image); else per-element loads.
// Every load is unconditional (out-of-image lanes read element 0 and are
// zeroed), so they all issue back to back.
template <bool VEC, bool XBF>
__device__ __forceinline__ void load_patch(PatchRegs<XBF>& r, const StemParams& p, int n, int ir0, int ic0,
                                           int tid) {
  using E = std::conditional_t<XBF, uint16_t, float>;
  const E* x = static_cast<const E*>(p.x);
#pragma unroll
  for (int u = 0; u < kUnits; ++u) {
    const int unit = tid + u * kThreads;
    const int row = unit / kSegs, seg = unit - (unit / kSegs) * kSegs;
    const int ih = ir0 + row, iw0 = ic0 + 4 * seg;
    const bool rok = unit < kPR * kSegs && (unsigned)ih < (unsigned)p.H;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const bool cok = rok && c < p.C;
      const size_t rbase = (((size_t)n * p.C + c) * p.H + ih) * p.W;
      if constexpr (VEC) {
        const bool ok = cok && iw0 >= 0 && iw0 < p.W;
        const size_t o = ok ? rbase + iw0 : 0;
        if constexpr (XBF) {
          const uint2 v = *reinterpret_cast<const uint2*>(x + o);
          r.v[u][c] = ok ? v : make_uint2(0u, 0u);
        } else {
          const float4 v = *reinterpret_cast<const float4*>(x + o);
          r.v[u][c] = ok ? v : make_float4(0.f, 0.f, 0.f, 0.f);
        }
      } else {
        E e4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bool ok = cok && (unsigned)(iw0 + e) < (unsigned)p.W;
          const E v = x[ok ? rbase + iw0 + e : 0];
          e4[e] = ok ? v : (E)0;
        }
        if constexpr (XBF)
          r.v[u][c] = make_uint2((uint32_t)e4[0] | ((uint32_t)e4[1] << 16), (uint32_t)e4[2] | ((uint32_t)e4[3] << 16));
        else
          r.v[u][c] = make_float4(e4[0], e4[1], e4[2], e4[3]);
      }
    }
  }
}

// Writes the loaded units as 4-channel cells: unit (row, seg) is cells
// [row][4 seg .. 4 seg + 3], 32 contiguous bytes.
template <bool XBF>
__device__ __forceinline__ void store_patch(const PatchRegs<XBF>& r, uint2* patch, int tid) {
#pragma unroll
  for (int u = 0; u < kUnits; ++u) {
    const int unit = tid + u * kThreads;
    if (unit >= kPR * kSegs) break;
    uint32_t h[4][4];  // [channel][pixel] bf16 bits
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if constexpr (XBF) {
        const uint2 v = r.v[u][c];
        h[c][0] = v.x & 0xFFFFu; h[c][1] = v.x >> 16; h[c][2] = v.y & 0xFFFFu; h[c][3] = v.y >> 16;
      } else {
        const float4 v = r.v[u][c];
        h[c][0] = f32_to_bf16(v.x); h[c][1] = f32_to_bf16(v.y); h[c][2] = f32_to_bf16(v.z); h[c][3] = f32_to_bf16(v.w);
      }
    }
    uint32_t w[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      w[2 * e] = h[0][e] | (h[1][e] << 16);
      w[2 * e + 1] = h[2][e] | (h[3][e] << 16);
    }
    uint4* dst = reinterpret_cast<uint4*>(patch + unit * 4);  // row * kPC + 4 * seg == 4 * unit
    dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
    dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
  }
}

template <bool VEC, bool XBF>
__global__ __launch_bounds__(kThreads, 2) void stem_conv_maxpool_kernel(StemParams p) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[kLdsBytes];
  bf16_t* wl = reinterpret_cast<bf16_t*>(lds);                    // [64][wld]
  uint2* patch = reinterpret_cast<uint2*>(lds + kWeightBytes);    // [kPR][kPC] cells
  bf16_t* tile = reinterpret_cast<bf16_t*>(lds + kWeightBytes);   // [CR*CC][kTileLd], over the patch

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4;
  const int TJ = (p.QO + kPJ - 1) / kPJ, TI = (p.PO + kPI - 1) / kPI;
  const int ntiles = p.N * TI * TJ;
  const int G = gridDim.x;
  int t = blockIdx.x;
  if (t >= ntiles) return;

  const int CR = (kPI - 1) * p.sph + p.kph;  // conv rows / cols of a tile
  const int CC = (kPJ - 1) * p.spw + p.kpw;
  const int npix = CR * CC;
  // patch column 0 sits `off` columns left of the tile's first input column,
  // so that it is 4-aligned in the image (the same for every tile: tile
  // origins step by multiples of 4 input columns)
  const int off = VEC ? (-(p.ppl * p.sw + p.pl)) & 3 : 0;
  // tile tt: image n, tile row / col ti, tj, global conv row / col of its local (0, 0)
  auto origin = [&](int tt, int& n, int& ti, int& tj, int& cr0, int& cc0) {
    tj = tt % TJ;
    const int rest = tt / TJ;
    ti = rest % TI;
    n = rest / TI;
    cr0 = ti * kPI * p.sph - p.ppt;
    cc0 = tj * kPJ * p.spw - p.ppl;
  };
  auto issue_patch = [&](PatchRegs<XBF>& r, int tt) {
    int n, ti, tj, cr0, cc0;
    origin(tt, n, ti, tj, cr0, cc0);
    load_patch<VEC, XBF>(r, p, n, cr0 * p.sh - p.pt, cc0 * p.sw - p.pl - off, tid);
  };

  // per-lane GEMM addressing, the same for every tile: patch cell of this
  // lane's pixel at tap (0, 0), and its (row, col) in the conv tile
  int pbase[kFragsPerWave], lrc[kFragsPerWave];
#pragma unroll
  for (int i = 0; i < kFragsPerWave; ++i) {
    const int m0 = (wave + 4 * i) * 16 + (lane & 15);
    const int m = m0 < npix ? m0 : 0;  // padding rows of the last tile: any valid address
    const int lr = m / CC, lc = m - (m / CC) * CC;
    pbase[i] = lr * p.sh * kPC + lc * p.sw + off + 2 * g;
    lrc[i] = m0 < npix ? (lr << 16) | lc : -1;
  }
  // bias of the 16 channels this lane finishes
  float4 bv[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
    bv[j] = p.bias ? *reinterpret_cast<const float4*>(p.bias + j * 16 + 4 * g) : make_float4(0.f, 0.f, 0.f, 0.f);

  // weights into LDS, once (16-byte chunks, all loads issued before the writes)
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
  PatchRegs<XBF> pr;
  issue_patch(pr, t);
  store_patch<XBF>(pr, patch, tid);
  if (t + G < ntiles) issue_patch(pr, t + G);
  lds_barrier();

  const ActClamp ac = act_clamp_of(p.act);
  for (;;) {
    int n, ti, tj, cr0, cc0;
    origin(t, n, ti, tj, cr0, cc0);

    // implicit GEMM: this wave owns pixel tiles wave, wave + 4, ...
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
        const uint2 t0 = patch[pbase[i] + r * kPC];
        const uint2 t1 = patch[pbase[i] + r * kPC + 1];
        const bf16x8 b = as_bf16x8(make_uint4(t0.x, t0.y, t1.x, t1.y));
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[j], b, acc[i][j], 0, 0, 0);
      }
    }
    lds_barrier();  // the patch is dead: the conv tile overlays it

    // bias, activation, bf16; conv outputs outside the image -> -inf
    auto epilogue = [&](auto gelu_tag) {
      constexpr bool GE = decltype(gelu_tag)::value;
#pragma unroll
      for (int i = 0; i < kFragsPerWave; ++i) {
        if (lrc[i] < 0) continue;
        const int lr = lrc[i] >> 16, lc = lrc[i] & 0xFFFF;
        const int m = lr * CC + lc;
        const bool inside = (unsigned)(cr0 + lr) < (unsigned)p.P && (unsigned)(cc0 + lc) < (unsigned)p.Q;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          uint2 o;
          if (inside) {
            const f32x4 v = acc[i][j];
            o = make_uint2(pack2_bf16(act_apply<GE>(v[0] + bv[j].x, ac), act_apply<GE>(v[1] + bv[j].y, ac)),
                           pack2_bf16(act_apply<GE>(v[2] + bv[j].z, ac), act_apply<GE>(v[3] + bv[j].w, ac)));
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
    lds_barrier();

    // pooling: 64 pooled pixels x 8 channel groups, two per thread
    constexpr int kItems = kPI * kPJ * (kK / 8) / kThreads;
    static_assert(kItems * kThreads == kPI * kPJ * (kK / 8), "pooling items");
    uint4 outv[kItems];
#pragma unroll
    for (int k = 0; k < kItems; ++k) {
      const int it = tid + k * kThreads;
      const int c8 = (it & 7) * 8;
      const int pi = (it >> 3) / kPJ, pj = (it >> 3) % kPJ;
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
      outv[k] = pack8(mx);
    }
    lds_barrier();  // the conv tile is dead: the next patch overlays it

    const int tn = t + G;
    if (tn < ntiles) store_patch<XBF>(pr, patch, tid);
#pragma unroll
    for (int k = 0; k < kItems; ++k) {
      const int it = tid + k * kThreads;
      const int c8 = (it & 7) * 8;
      const int po = ti * kPI + (it >> 3) / kPJ, qo = tj * kPJ + (it >> 3) % kPJ;
      if (po < p.PO && qo < p.QO)
        *reinterpret_cast<uint4*>(p.y + (((size_t)n * p.PO + po) * p.QO + qo) * kK + c8) = outv[k];
    }
    if (tn >= ntiles) break;
    if (tn + G < ntiles) issue_patch(pr, tn + G);
    lds_barrier();
    t = tn;
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
  // persistent grid: two workgroups per CU, never more than the tiles
  static std::atomic<int> cus{0};
  if (cus.load() == 0) {
    int dev = 0, n = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    cus.store(n > 0 ? n : 1);
  }
  const int64_t tiles = (int64_t)p.N * ((p.PO + kPI - 1) / kPI) * ((p.QO + kPJ - 1) / kPJ);
  if (tiles <= 0) return hipSuccess;
  if (tiles > (1ll << 30)) return hipErrorInvalidValue;
  int64_t grid = std::min<int64_t>(tiles, 2 * (int64_t)cus.load());
  if (p.grid_cap > 0) grid = std::min<int64_t>(grid, p.grid_cap);
  // vector segment loads need 4-aligned rows and an aligned base
  const size_t elem = p.x_bf16 ? 2 : 4;
  const bool vec = p.W % 4 == 0 && reinterpret_cast<uintptr_t>(p.x) % (4 * elem) == 0;
  if (p.x_bf16) {
    if (vec)
      stem_conv_maxpool_kernel<true, true><<<(int)grid, kThreads, 0, s>>>(p);
    else
      stem_conv_maxpool_kernel<false, true><<<(int)grid, kThreads, 0, s>>>(p);
  } else {
    if (vec)
      stem_conv_maxpool_kernel<true, false><<<(int)grid, kThreads, 0, s>>>(p);
    else
      stem_conv_maxpool_kernel<false, false><<<(int)grid, kThreads, 0, s>>>(p);
  }
  return hipGetLastError();
}

hipError_t launch_pack_stem_weights(const void* src, bool src_bf16, bf16_t* dst, int C, int R, int S, int wld,
                                    hipStream_t s) {
  const int n = kK * wld;
  pack_stem_weights_kernel<<<(n + 255) / 256, 256, 0, s>>>(src, src_bf16 ? 1 : 0, dst, C, R, S, wld);
  return hipGetLastError();
}

}  // namespace byoc
