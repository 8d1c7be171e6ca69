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
// Work unit ("tile"): TH = 8 rows x TW columns of pooled outputs x 64
// channels of one image, TW = (16 - pool width) / pool stride + 1 (7 for a
// 3x3 / stride-2 pool).  Each of the 4 waves computes two pooled rows: the
// conv rows their windows cover (sph + kph <= 5 rows, a row shared with the
// next wave is recomputed), each row a 16-pixel MFMA tile whose lane l holds
// conv column l.  So the pooling never leaves registers: the window's rows
// are accumulators of the same lane, its columns neighbouring lanes (DPP
// row shifts).  Workgroups are persistent (256 threads) and stride over
// the tiles:
//  - the packed weights [64][R*32 + 8] and the bias are staged in LDS once;
//  - the input patch of a tile is staged in LDS as [row][col][4 channels]
//    bf16 cells (zero outside the image); the global loads of the next
//    tile's patch are issued one tile ahead and land in registers while
//    the current tile computes;
//  - implicit GEMM on v_mfma_f32_16x16x32_bf16: one 32-element reduction
//    step per kernel row r, ordered (tap s < 8, channel c < 4); a lane's 8
//    reduction elements are taps 2g and 2g+1 of its conv pixel, i.e. two
//    adjacent patch cells.  Weights are the A operand, pixels B, and the
//    accumulators start at the bias;
//  - activation, -inf for conv outputs outside the image (they never win
//    the max), max over the window, bf16 rounding (monotone, so rounding
//    after the max equals the max of rounded values), 8-byte NHWC stores.
// Barriers inside the tile loop wait on LDS only, so the patch loads in
// flight cross them.
//
// int8 codes (a partially quantized function, Sec. 3.2): the patch holds
// the input's codes, clip(rint(x / S_x) + Z_x) as the boundary quantize
// computes them (positions outside the image read 0 and so hold Z_x, the
// padding the folded bias expects), one dword of 4 channel codes per cell;
// v_mfma_i32_16x16x64_i8 takes two kernel rows per step (lane group g: row
// 2m + g / 2, taps 4 (g % 2) .. + 3, four cells); the int32 sums start at
// the folded bias.  Requantizing (clamp(Z_y + rescale(a, m), lo, hi), m > 0)
// is monotone, so the pooling max is taken over the sums of the positions
// inside the image and the maximum requantized once: the codes of the
// unfused conv followed by the max pool of codes.
#include "device_common.h"

#include <atomic>
#include <climits>

namespace byoc {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) int i32x4;

constexpr int kThreads = 256;
constexpr int kTH = 8;        // pooled rows per tile (2 per wave)
constexpr int kRowsWave = 5;  // conv rows (MFMA tiles) per wave: sph + kph <= 5
constexpr int kPR = 40;       // patch rows: (3 * 2 * 2 + 4) * 2 + 8
constexpr int kPC = 48;       // patch cols: 15 * 2 + 8 + 3 (alignment offset), in 4-cell segments
constexpr int kSegs = kPC / 4;
constexpr int kUnits = (kPR * kSegs + kThreads - 1) / kThreads;  // (row, segment) units per thread
constexpr int kK = 64;                                           // output channels
constexpr int kWeightLdMax = 8 * 32 + 8;
constexpr int kWChunks = (kK * kWeightLdMax / 8 + kThreads - 1) / kThreads;  // 16-byte weight chunks per thread
constexpr int kWeightBytes = kWChunks * kThreads * 16;  // >= 64 rows of kWeightLdMax; every thread fills its chunks
constexpr int kBiasBytes = kK * 8;  // float bias, or {int32 bias, float32 factor} of codes
constexpr int kPatchBytes = kUnits * kThreads * 32;  // every thread writes its units, the last ones past the patch
constexpr int kLdsBytes = kWeightBytes + kBiasBytes + kPatchBytes;
static_assert(kPatchBytes >= kPR * kPC * 8, "patch");
static_assert(3 * kLdsBytes <= 160 * 1024, "three workgroups per CU");

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

// max(a, b) in one instruction (median of a, b and +inf); no NaN handling
__device__ __forceinline__ float max2(float a, float b) { return __builtin_amdgcn_fmed3f(a, b, INFINITY); }

// Lane l + k of the same 16-lane row (k = 1, 2); lanes past the row's end
// read their own value (they are never kept).
template <int K>
__device__ __forceinline__ float row_next(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0x100 + K, 0xF, 0xF, false));
}

// Input values of one (patch row, 4-column segment) unit, per channel:
// 4 bf16 (XBF) or 4 f32.
template <bool XBF>
struct PatchRegs {
  using T = std::conditional_t<XBF, uint2, float4>;
  T v[kUnits][4];
};

// Issues the loads of a tile's patch (rows ir0.., columns ic0.. of image n)
// through a buffer descriptor over the image: positions outside the image
// take an out-of-range offset and read zeros, so every load is issued
// unconditionally and back to back, and no select follows it.
// VEC: a segment is one vector load (W % 4 == 0 and ic0 % 4 == 0, so a
// segment is wholly inside or outside the image); else per-element loads.
template <bool VEC, bool XBF>
__device__ __forceinline__ void load_patch(PatchRegs<XBF>& r, const StemParams& p, int n, int ir0, int ic0,
                                           int tid) {
  constexpr int kE = XBF ? 2 : 4;       // element bytes
  const int img = p.C * p.H * p.W * kE;  // image bytes (< 2^31, checked by the launcher)
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char*>(static_cast<const char*>(p.x)) + (size_t)n * img, (short)0, img, kBufferFlags);
#pragma unroll
  for (int u = 0; u < kUnits; ++u) {
    const int unit = tid + u * kThreads;
    const int row = unit / kSegs, seg = unit - (unit / kSegs) * kSegs;
    const int ih = ir0 + row, iw0 = ic0 + 4 * seg;
    // non-short-circuit tests: the offsets are selects, not branches
    const bool rok = (unit < kPR * kSegs) & ((unsigned)ih < (unsigned)p.H);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const bool cok = rok & (c < p.C);
      const int rbase = (c * p.H + ih) * p.W;  // element offset of the row (used only when in range)
      if constexpr (VEC) {
        const uint32_t off = (cok & (iw0 >= 0) & (iw0 < p.W)) ? (uint32_t)(rbase + iw0) * kE : kOOB;
        if constexpr (XBF)
          r.v[u][c] = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0));
        else
          r.v[u][c] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
      } else {
        uint32_t e4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t off = (cok & ((unsigned)(iw0 + e) < (unsigned)p.W)) ? (uint32_t)(rbase + iw0 + e) * kE : kOOB;
          if constexpr (XBF)
            e4[e] = __builtin_amdgcn_raw_buffer_load_b16(rs, off, 0, 0);
          else
            e4[e] = __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0);
        }
        if constexpr (XBF)
          r.v[u][c] = make_uint2(e4[0] | (e4[1] << 16), e4[2] | (e4[3] << 16));
        else
          r.v[u][c] = make_float4(__uint_as_float(e4[0]), __uint_as_float(e4[1]), __uint_as_float(e4[2]),
                                  __uint_as_float(e4[3]));
      }
    }
  }
}

// Writes the loaded units as 4-channel cells: unit (row, seg) is cells
// [row][4 seg .. 4 seg + 3], 32 contiguous bytes.  Units past the patch
// (zeros) land in the padding after it; the writes are unconditional so
// that every load is waited for on every path (a skipped wait would make
// the compiler wait again inside the tile loop).
template <bool XBF>
__device__ __forceinline__ void store_patch(const PatchRegs<XBF>& r, uint2* patch, int tid) {
#pragma unroll
  for (int u = 0; u < kUnits; ++u) {
    const int unit = tid + u * kThreads;
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

// int8: the loaded units quantized to codes, 4 channel codes per cell
// (16 bytes per unit).
template <bool XBF>
__device__ __forceinline__ void store_patch_i8(const PatchRegs<XBF>& r, uint32_t* patch, int tid, float inv,
                                               int zp) {
#pragma unroll
  for (int u = 0; u < kUnits; ++u) {
    const int unit = tid + u * kThreads;
    uint32_t w[4] = {0u, 0u, 0u, 0u};  // cells (pixels) of the unit
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      float f[4];
      if constexpr (XBF) {
        const uint2 v = r.v[u][c];
        f[0] = __uint_as_float(v.x << 16), f[1] = __uint_as_float(v.x & 0xFFFF0000u);
        f[2] = __uint_as_float(v.y << 16), f[3] = __uint_as_float(v.y & 0xFFFF0000u);
      } else {
        const float4 v = r.v[u][c];
        f[0] = v.x, f[1] = v.y, f[2] = v.z, f[3] = v.w;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float t = fminf(fmaxf(rintf(f[e] * inv), -512.0f), 512.0f);
        w[e] |= ((uint32_t)clip_i8((int)t + zp) & 0xFFu) << (8 * c);
      }
    }
    *reinterpret_cast<uint4*>(patch + unit * 4) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// lane l + k of the same 16-lane row, as row_next, on int32
template <int K>
__device__ __forceinline__ int row_next_i(int v) {
  return __builtin_amdgcn_update_dpp(v, v, 0x100 + K, 0xF, 0xF, false);
}

template <bool VEC, bool XBF, bool I8>
__global__ __launch_bounds__(kThreads, 2) void stem_conv_maxpool_kernel(StemParams p) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[kLdsBytes];
  bf16_t* wl = reinterpret_cast<bf16_t*>(lds);                               // [64][wld]
  const unsigned char* wl8 = lds;                                            // int8: [64][wld] bytes
  float* sbias = reinterpret_cast<float*>(lds + kWeightBytes);               // [64] (int8: [64][2])
  uint2* patch = reinterpret_cast<uint2*>(lds + kWeightBytes + kBiasBytes);  // [kPR][kPC] cells
  uint32_t* patch8 = reinterpret_cast<uint32_t*>(patch);                     // int8 cells

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, l16 = lane & 15;
  const int TW = (16 - p.kpw) / p.spw + 1;  // pooled columns per tile
  const int TJ = (p.QO + TW - 1) / TW, TI = (p.PO + kTH - 1) / kTH;
  const int ntiles = p.N * TI * TJ;
  const int G = gridDim.x;
  int t = blockIdx.x;
  if (t >= ntiles) return;

  // tile tt: image n, tile row / col ti, tj, global conv row / col of the
  // tile's first conv row / column (lane 0 of wave 0's first MFMA tile)
  auto origin = [&](int tt, int& n, int& ti, int& tj, int& cr0, int& cc0) {
    tj = tt % TJ;
    const int rest = tt / TJ;
    ti = rest % TI;
    n = rest / TI;
    cr0 = ti * kTH * p.sph - p.ppt;
    cc0 = tj * TW * p.spw - p.ppl;
  };
  // patch column 0 is the tile's first input column rounded down to a
  // multiple of 4 (vector loads); `off` is the difference
  auto col_off = [&](int cc0) { return VEC ? (cc0 * p.sw - p.pl) & 3 : 0; };
  auto issue_patch = [&](PatchRegs<XBF>& r, int tt) {
    int n, ti, tj, cr0, cc0;
    origin(tt, n, ti, tj, cr0, cc0);
    load_patch<VEC, XBF>(r, p, n, cr0 * p.sh - p.pt, cc0 * p.sw - p.pl - col_off(cc0), tid);
  };

  // this wave's conv rows: local rows wave * 2 * sph + f, f < kRowsWave;
  // patch cell of lane (row f, column l16) at tap (0, 0), before `off`
  const int lrow0 = wave * 2 * p.sph;
  int pbase[kRowsWave];
#pragma unroll
  for (int f = 0; f < kRowsWave; ++f)
    pbase[f] = I8 ? (lrow0 + f) * p.sh * kPC + l16 * p.sw + (g >> 1) * kPC + 4 * (g & 1)
                  : (lrow0 + f) * p.sh * kPC + l16 * p.sw + 2 * g;

  // weights, bias and the first patch: every load is issued before the
  // first LDS write, and all are unconditional (buffer loads past the end
  // read zeros), so their latencies overlap.  Values the tile loop uses
  // never come straight from a global load: the compiler's wait tracking
  // would then stall the loop on the patch loads in flight.
  {
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p.w), (short)0,
                                                                         kK * p.wld * (I8 ? 1 : 2), kBufferFlags);
    uint4 wv[kWChunks];
#pragma unroll
    for (int i = 0; i < kWChunks; ++i)
      wv[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(wr, (uint32_t)(tid + i * kThreads) * 16u, 0, 0));
    constexpr int kBiasLoads = kK * (I8 ? 8 : 4) / 16;  // 16-byte loads of the bias (table)
    const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p.bias), (short)0,
                                                                         p.bias ? kBiasLoads * 16 : 0, kBufferFlags);
    float4 b = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(br, tid < kBiasLoads ? tid * 16u : kOOB, 0, 0));
    PatchRegs<XBF> first;
    issue_patch(first, t);
    asm volatile("" : "+v"(b.x), "+v"(b.y), "+v"(b.z), "+v"(b.w));  // keeps the bias load ahead of the writes
    uint4* dst = reinterpret_cast<uint4*>(wl);
#pragma unroll
    for (int i = 0; i < kWChunks; ++i) dst[tid + i * kThreads] = wv[i];
    if (tid < kBiasLoads) reinterpret_cast<float4*>(sbias)[tid] = b;
    if constexpr (I8) store_patch_i8<XBF>(first, patch8, tid, p.inv_scale, p.zx);
    else store_patch<XBF>(first, patch, tid);
  }
  PatchRegs<XBF> pr;
  if (t + G < ntiles) issue_patch(pr, t + G);
  lds_barrier();

  for (;;) {
    int n, ti, tj, cr0, cc0;
    origin(t, n, ti, tj, cr0, cc0);
    const int off = col_off(cc0);

    if constexpr (I8) {
      // implicit GEMM on codes: the sums start at the folded bias
      i32x4 acc[kRowsWave][4];
      const int* sq = reinterpret_cast<const int*>(sbias);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int4 lo = *reinterpret_cast<const int4*>(sq + 2 * (j * 16 + 4 * g));
        const int4 hi = *reinterpret_cast<const int4*>(sq + 2 * (j * 16 + 4 * g) + 4);
#pragma unroll
        for (int f = 0; f < kRowsWave; ++f) acc[f][j] = i32x4{lo.x, lo.z, hi.x, hi.z};
      }
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        if (2 * m >= p.R) break;
        i32x4 a[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          a[j] = *reinterpret_cast<const i32x4*>(wl8 + (j * 16 + l16) * p.wld + m * 64 + g * 16);
#pragma unroll
        for (int f = 0; f < kRowsWave; ++f) {
          const uint32_t* c = patch8 + pbase[f] + off + 2 * m * kPC;  // four cells, 4-byte aligned
          const i32x4 b = i32x4{(int)c[0], (int)c[1], (int)c[2], (int)c[3]};
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[f][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[j], b, acc[f][j], 0, 0, 0);
        }
      }
      lds_barrier();  // every wave is done with the patch
      const int tn = t + G;
      if (tn < ntiles) store_patch_i8<XBF>(pr, patch8, tid, p.inv_scale, p.zx);
      if (tn + G < ntiles) issue_patch(pr, tn + G);
      // conv positions outside the image never win the max
      const bool colok = (unsigned)(cc0 + l16) < (unsigned)p.Q;
#pragma unroll
      for (int f = 0; f < kRowsWave; ++f) {
        const bool ok = colok & ((unsigned)(cr0 + lrow0 + f) < (unsigned)p.P);
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[f][j][e] = ok ? acc[f][j][e] : INT_MIN;
      }
      const bool lane_out = (l16 % p.spw == 0) & (l16 / p.spw < TW);
      const int qo = tj * TW + l16 / p.spw;
      const bool r1 = p.kph > 1, r2 = p.kph > 2, c1 = p.kpw > 1, c2 = p.kpw > 2;
      int8_t* y8 = reinterpret_cast<int8_t*>(p.y);
      auto pool = [&](auto sph_tag) {
        constexpr int SPH = decltype(sph_tag)::value;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int po = ti * kTH + 2 * wave + q;
          const bool st = lane_out & (po < p.PO) & (qo < p.QO);
          int8_t* dst = y8 + (((size_t)n * p.PO + po) * p.QO + qo) * kK + 4 * g;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int4 lo = *reinterpret_cast<const int4*>(sq + 2 * (j * 16 + 4 * g));
            const int4 hi = *reinterpret_cast<const int4*>(sq + 2 * (j * 16 + 4 * g) + 4);
            const int fs[4] = {lo.y, lo.w, hi.y, hi.w};
            uint32_t w = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              int v = acc[SPH * q][j][e];
              v = max(v, r1 ? acc[SPH * q + 1][j][e] : INT_MIN);
              v = max(v, r2 ? acc[SPH * q + 2][j][e] : INT_MIN);
              const int h1 = row_next_i<1>(v), h2 = row_next_i<2>(v);
              int h = max(v, c1 ? h1 : INT_MIN);
              h = max(h, c2 ? h2 : INT_MIN);
              const int code = min(max(p.zy + rescale(h, __int_as_float(fs[e])), p.lo), p.hi);
              w |= ((uint32_t)code & 0xFFu) << (8 * e);
            }
            if (st) *reinterpret_cast<uint32_t*>(dst + j * 16) = w;
          }
        }
      };
      if (p.sph == 2) pool(std::integral_constant<int, 2>{});
      else pool(std::integral_constant<int, 1>{});
      if (tn >= ntiles) break;
      lds_barrier();  // the next patch is in LDS
      t = tn;
      continue;
    }
    if constexpr (!I8) {
    // implicit GEMM.  Accumulators start at the bias of their channels, or
    // at -inf for conv positions outside the image (then they stay -inf:
    // the products added are finite), which excludes those positions from
    // the pooling max.
    const bool colok = (unsigned)(cc0 + l16) < (unsigned)p.Q;
    f32x4 acc[kRowsWave][4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float4 b = reinterpret_cast<const float4*>(sbias)[j * 4 + g];
#pragma unroll
      for (int f = 0; f < kRowsWave; ++f) {
        const bool ok = colok & ((unsigned)(cr0 + lrow0 + f) < (unsigned)p.P);
        acc[f][j] = ok ? f32x4{b.x, b.y, b.z, b.w} : f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      }
    }
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      if (r >= p.R) break;
      bf16x8 a[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        a[j] = as_bf16x8(*reinterpret_cast<const uint4*>(wl + (j * 16 + l16) * p.wld + r * 32 + g * 8));
#pragma unroll
      for (int f = 0; f < kRowsWave; ++f) {
        const uint2 t0 = patch[pbase[f] + off + r * kPC];
        const uint2 t1 = patch[pbase[f] + off + r * kPC + 1];
        const bf16x8 b = as_bf16x8(make_uint4(t0.x, t0.y, t1.x, t1.y));
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[f][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[j], b, acc[f][j], 0, 0, 0);
      }
    }
    lds_barrier();  // every wave is done with the patch

    // the next tile's patch (its loads were issued a tile ago), then the
    // loads of the one after
    const int tn = t + G;
    if (tn < ntiles) store_patch<XBF>(pr, patch, tid);
    if (tn + G < ntiles) issue_patch(pr, tn + G);

    // GELU is not monotone: it goes before the max (outside positions stay
    // -inf).  The clamps (none, ReLU, ReLU6) are, as is bf16 rounding: they
    // go after it, once per pooled value.
    if (p.act == kActGelu) {
#pragma unroll
      for (int f = 0; f < kRowsWave; ++f)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float x = acc[f][j][e];
            acc[f][j][e] = x == -INFINITY ? x : gelu(x);
          }
    }
    const ActClamp ac = p.act == kActGelu ? act_clamp_of(kActNone, 0.f) : act_clamp_of(p.act, p.alpha);

    // pooled rows 2 wave + q (q < 2): window rows SPH * q + dr of this
    // wave's conv rows, window columns lanes spw * c + dc.  FULL: a 3x3
    // window; else rows / columns past the window are masked to -inf.
    const bool lane_out = (l16 % p.spw == 0) & (l16 / p.spw < TW);
    const int qo = tj * TW + l16 / p.spw;
    auto pool = [&](auto sph_tag, auto full_tag) {
      constexpr int SPH = decltype(sph_tag)::value;
      constexpr bool FULL = decltype(full_tag)::value;
      const bool r1 = FULL || p.kph > 1, r2 = FULL || p.kph > 2, c1 = FULL || p.kpw > 1, c2 = FULL || p.kpw > 2;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int po = ti * kTH + 2 * wave + q;
        const bool st = lane_out & (po < p.PO) & (qo < p.QO);
        bf16_t* dst = reinterpret_cast<bf16_t*>(p.y) + (((size_t)n * p.PO + po) * p.QO + qo) * kK + 4 * g;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float m[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float v = acc[SPH * q][j][e];
            v = max2(v, r1 ? acc[SPH * q + 1][j][e] : -INFINITY);
            v = max2(v, r2 ? acc[SPH * q + 2][j][e] : -INFINITY);
            const float h1 = row_next<1>(v), h2 = row_next<2>(v);
            float h = max2(v, c1 ? h1 : -INFINITY);
            h = max2(h, c2 ? h2 : -INFINITY);
            m[e] = act_apply<false>(h, ac);
          }
          if (st) *reinterpret_cast<uint2*>(dst + j * 16) = make_uint2(pack2_bf16(m[0], m[1]), pack2_bf16(m[2], m[3]));
        }
      }
    };
    const bool full = p.kph == 3 && p.kpw == 3;
    if (p.sph == 2) {
      if (full) pool(std::integral_constant<int, 2>{}, std::true_type{});
      else pool(std::integral_constant<int, 2>{}, std::false_type{});
    } else {
      if (full) pool(std::integral_constant<int, 1>{}, std::true_type{});
      else pool(std::integral_constant<int, 1>{}, std::false_type{});
    }
    if (tn >= ntiles) break;
    lds_barrier();  // the next patch is in LDS
    t = tn;
    }
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

int stem_weight_ld_i8(int R) { return (R + 1) / 2 * 64 + 16; }

hipError_t launch_stem_conv_maxpool(const StemParams& p, hipStream_t s) {
  // persistent grid: two workgroups per CU of the current device, never
  // more than the tiles (CU counts cached per device)
  constexpr int kMaxDev = 64;
  static std::atomic<int> cu_of[kMaxDev] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  int ncu = dev >= 0 && dev < kMaxDev ? cu_of[dev].load() : 0;
  if (ncu == 0) {
    int n = 0;
    e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    ncu = n > 0 ? n : 1;
    if (dev >= 0 && dev < kMaxDev) cu_of[dev].store(ncu);
  }
  const int tw = (16 - p.kpw) / p.spw + 1;
  const int64_t tiles = (int64_t)p.N * ((p.PO + kTH - 1) / kTH) * ((p.QO + tw - 1) / tw);
  if (tiles <= 0) return hipSuccess;
  // tile indices are int; one image is addressed by 32-bit buffer offsets
  if (tiles > (1ll << 30) || (int64_t)p.C * p.H * p.W * (p.x_bf16 ? 2 : 4) >= (1ll << 31))
    return hipErrorInvalidValue;
  int64_t grid = std::min<int64_t>(tiles, 2 * (int64_t)ncu);
  if (p.grid_cap > 0) grid = std::min<int64_t>(grid, p.grid_cap);
  // vector segment loads need 4-aligned rows and an aligned base
  const size_t elem = p.x_bf16 ? 2 : 4;
  const bool vec = p.W % 4 == 0 && reinterpret_cast<uintptr_t>(p.x) % (4 * elem) == 0;
  if (p.i8 && (p.wld % 16 != 0 || p.wld < (p.R + 1) / 2 * 64)) return hipErrorInvalidValue;
  auto go = [&](auto i8_tag) {
    constexpr bool Q = decltype(i8_tag)::value;
    if (p.x_bf16) {
      if (vec)
        stem_conv_maxpool_kernel<true, true, Q><<<(int)grid, kThreads, 0, s>>>(p);
      else
        stem_conv_maxpool_kernel<false, true, Q><<<(int)grid, kThreads, 0, s>>>(p);
    } else {
      if (vec)
        stem_conv_maxpool_kernel<true, false, Q><<<(int)grid, kThreads, 0, s>>>(p);
      else
        stem_conv_maxpool_kernel<false, false, Q><<<(int)grid, kThreads, 0, s>>>(p);
    }
  };
  if (p.i8) go(std::true_type{});
  else go(std::false_type{});
  return hipGetLastError();
}

hipError_t launch_pack_stem_weights(const void* src, bool src_bf16, bf16_t* dst, int C, int R, int S, int wld,
                                    hipStream_t s) {
  const int n = kK * wld;
  pack_stem_weights_kernel<<<(n + 255) / 256, 256, 0, s>>>(src, src_bf16 ? 1 : 0, dst, C, R, S, wld);
  return hipGetLastError();
}

}  // namespace byoc
