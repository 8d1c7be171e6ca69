// 3x3 stride-1 convolution with the input window of a tile staged in LDS.
//
// The implicit-GEMM kernel reads every activation once per tap: a tile of
// BM output pixels fetches BM rows of 64 channels for each of the nine taps.
// Here the tile's input window - the rows its output pixels touch plus a
// one-pixel halo, zero padded - is loaded into LDS once per 64-channel
// slice, and the nine taps are nine shifted views of it: output pixel
// (n, p, q) reads patch pixel base(n, p, q) + r * (W + 2) + s for tap (r, s).
// The activation bytes fetched per tile drop from 9 * BM rows to about
// (BM / W + 2 + 2 * images) * (W + 2) rows per slice; the weights stream as
// before, one tap (BN rows of 64 channels) per stage.
//
// Patch geometry.  Stack the images with a zero row above and below each:
// input row h of image n is virtual row n * (H + 2) + h + 1.  The output
// pixels of a tile (a run of BM consecutive pixels of the N*P*Q order) need
// the virtual rows from that of input row p_first - 1 of the first pixel's
// image to that of input row p_last + 1 of the last pixel's image; every
// row between them is part of some output pixel's window or a zero row.
// Each virtual row is W + 2 pixels wide (zero columns left and right).  The
// host checks that the largest tile's patch fits the kernel's capacity.
//
// Pipeline.  A stage is TPS taps (1, or 3 = one kernel row) of one 64-channel
// slice; a slice has 9 / TPS stages, unrolled.  Per stage: wait for its
// weights - and at the slice's first stage for the slice's patch, which is
// older - then one barrier; issue the weights NSW - 1 stages ahead (into the
// ring slot of the stage computed last) and, at a slice's first stage, the
// next slice's patch into the other patch buffer; then 2 * TPS k-steps of
// the 16x16x32 MFMA.  Larger stages amortize the barrier and the LDS read
// latency that every stage exposes.  Loads past the end read zeros
// (out-of-range buffer offsets) so every step issues the same loads and the
// wait counts are compile-time constants.
//
// LDS rows are 128 bytes (64 channels); a load instruction fills 8
// consecutive rows (lane l -> row l / 8, slot l % 8), each lane fetching the
// logical chunk that belongs in its slot.  Weight row rw keeps chunk ch at
// slot ch ^ (rw & 7), the implicit-GEMM kernel's layout.  Patch pixel pp of
// virtual row v uses the key (pp - 2 v) & 7 instead: pp - 2 v = v W + col
// is the pixel's index with the zero columns left out, which runs on by one
// from pixel to pixel of consecutive output pixels also where they cross
// an image row (pp itself jumps by 3 there).  So any 8 consecutive output
// pixels read 8 distinct slots for every tap: no bank conflicts.
//
// Weights are the MFMA A operand and pixels the B operand, so each lane
// holds 4 consecutive output channels of one pixel; the epilogue (bias,
// residual, activation, bf16 rounding, 16-byte stores through an LDS
// staging tile) is the implicit-GEMM kernel's.
//
// int8 codes (I8): a 128-byte row holds 128 channels, the same two k-steps
// of v_mfma_i32_16x16x64_i8 per row, exact int32 sums; the zero rows and
// columns of the patch read as code 0, and the epilogue is the int8
// implicit-GEMM kernel's (folded bias, border correction for the taps
// outside the image, rescaling, residual, clamp).
#include <algorithm>
#include <type_traits>

#include "lds_dma.h"
#include "quant_epilogue.h"

namespace byoc {
namespace {

using namespace dma;

constexpr int kSlice = 64;  // bf16 channels per reduction slice (one 128-byte LDS row per pixel)
constexpr int kTaps = 9;

__device__ __forceinline__ f32x4 mma(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}
__device__ __forceinline__ i32x4 mma(uint4 a, uint4 b, i32x4 c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, a), __builtin_bit_cast(i32x4, b), c, 0,
                                               0, 0);
}

template <int BM, int BN, int WM, int WN, int TPS, int NSW, int LP, int NPB, bool I8>
__global__ __launch_bounds__(64 * WM * WN) void conv_halo_kernel(QConvParams q) {
  const ConvParams& p = q.g;
  constexpr int ES = I8 ? 1 : 2;   // bytes per element
  constexpr int CS = 128 / ES;     // channels per slice
  using Acc = std::conditional_t<I8, i32x4, f32x4>;
  constexpr int kWaves = WM * WN;
  constexpr int kNT = 64 * kWaves;
  constexpr int WTM = BM / WM, WTN = BN / WN;  // wave tile
  constexpr int TM = WTM / 16, TN = WTN / 16;  // 16x16 MFMA tiles per wave
  constexpr int kRowsPerPass = kNT / 8;        // weight rows one load of every wave covers
  constexpr int BR = BN / kRowsPerPass;        // weight loads per thread per stage
  static_assert(TM >= 1 && TN >= 1 && BR >= 1, "tile");
  static_assert(TPS == 1 || TPS == 3, "taps per stage");
  constexpr int SPS = kTaps / TPS;  // stages per slice
  // the next slice's patch (issued at a slice's first stage, after the
  // weights NSW - 1 stages ahead) must be older than the next slice's
  // first weights
  static_assert(NSW >= 2 && NSW <= SPS, "weight ring depth");
  static_assert(NPB == 1 || NPB == 2, "patch buffers");
  constexpr int PPX = LP * kWaves * 8;  // patch capacity (pixels)
  constexpr int PSTAGE = PPX * 8;       // uint4 per patch buffer
  constexpr int WTAP = BN * 8;          // uint4 per tap of a weight stage
  constexpr int WSTAGE = TPS * WTAP;    // uint4 per weight stage
  constexpr int LW = TPS * BR;          // weight loads per thread per stage
  static_assert((NSW - 2) * LW + LP <= 63, "vmcnt immediate");

  __shared__ uint4 lds[NPB * PSTAGE + NSW * WSTAGE];
  uint4* const patch = lds;                 // NPB patch buffers
  uint4* const wring = lds + NPB * PSTAGE;  // NSW weight stages
  __shared__ float4 sbias[64];  // bias of the tile's channels (a whole wave's 16-byte fill)
  materialize_args(p);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int cv = (lane & 7) ^ ((lane >> 3) & 7);  // logical chunk this lane fetches (weights)

  int tm, tn;
  if (!place_tile<BM, BN>(p, &tm, &tn)) return;
  const int m0 = tm * BM;
  const int n0 = tn * BN;
  const int PQ = p.P * p.Q;
  const int HP = p.H + 2, WP = p.W + 2;

  // virtual rows of the tile's patch: first = input row p_first - 1 of the
  // first pixel's image, last = input row p_last + 1 of the last one's
  const int mlast = min(m0 + BM, p.M) - 1;
  const int nf = mdiv(m0, p.mg_pq);
  const int pf = mdiv(m0 - nf * PQ, p.mg_q);
  const int nl = mdiv(mlast, p.mg_pq);
  const int pl = mdiv(mlast - nl * PQ, p.mg_q);
  const int vr0 = nf * HP + pf;
  const int npx = (nl * HP + pl + 2 - vr0 + 1) * WP;  // patch pixels (<= PPX, checked by the host)

  // Patch pixels this thread fetches: load i of wave w fills pixels
  // [(i * kWaves + w) * 8, +8), lane l pixel (l / 8).  Offsets are those of
  // slice 0; slice c adds 128 c bytes.  Zero rows and columns, and pixels
  // past the patch, read from an out-of-range offset.
  uint32_t poff[LP];
#pragma unroll
  for (int i = 0; i < LP; ++i) {
    const int pp = (i * kWaves + wave) * 8 + (lane >> 3);
    uint32_t off = kOOB;
    if (pp < npx) {
      const int vrow = mdiv(pp, p.mg_wp);
      const int col = pp - vrow * WP;
      const int ch = (lane & 7) ^ ((pp - 2 * vrow) & 7);  // logical chunk of this lane's slot
      const int vr = vr0 + vrow;
      const int n = mdiv(vr, p.mg_hp);
      const int h = vr - n * HP - 1;
      const int w = col - 1;
      if ((unsigned)h < (unsigned)p.H && (unsigned)w < (unsigned)p.W)
        off = (uint32_t)(((n * p.H + h) * p.W + w) * p.Cp * ES + ch * 16);
    }
    poff[i] = off;
  }
  // Patch pixel of the window's top-left corner for this lane's output
  // pixels (MFMA column lane % 16 of each of the wave's TM pixel tiles) and
  // its swizzle index (the pixel index without zero columns); rows past M
  // read pixel 0 and are never stored.
  int pbase[TM], cbase[TM];
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    const int m = m0 + wm * WTM + j * 16 + (lane & 15);
    int b = 0;
    if (m < p.M) {
      const int n = mdiv(m, p.mg_pq);
      const int pq = m - n * PQ;
      const int pp = mdiv(pq, p.mg_q);
      const int q = pq - pp * p.Q;
      b = (n * HP + pp - vr0) * WP + q;
    }
    pbase[j] = b;
    cbase[j] = b - 2 * mdiv(b, p.mg_wp);
  }

  const i32x4 xr = buffer_rsrc(p.x, p.x_bytes);
  const i32x4 wr = buffer_rsrc(p.w, p.w_bytes);
  uint32_t wvoff[BR];  // byte offset of this thread's weight rows and chunk
#pragma unroll
  for (int i = 0; i < BR; ++i) wvoff[i] = (uint32_t)((n0 + (tid >> 3) + i * kRowsPerPass) * p.Kgp * ES + cv * 16);

  const int nslices = p.Cp / CS;
  const int nst = SPS * nslices;  // weight stages
  // next weight stage to issue: its index, stage within the slice, slice and ring slot
  int wg = 0, wt = 0, wc = 0, wslot = 0;
  auto issue_w = [&]() {
    uint4* dst = wring + wslot * WSTAGE;
    const bool live = wg < nst;
#pragma unroll
    for (int u = 0; u < TPS; ++u) {
      const uint32_t col = (uint32_t)((wt * TPS + u) * p.Cp + wc * CS) * ES;
#pragma unroll
      for (int i = 0; i < BR; ++i)
        lds_fill16(wr,
                   __builtin_amdgcn_readfirstlane(lds_addr(dst + u * WTAP + (i * kRowsPerPass + wave * 8) * 8)),
                   live ? wvoff[i] + col : kOOB);
    }
    ++wg;
    if (++wt == SPS) {
      wt = 0;
      ++wc;
    }
    if (++wslot == NSW) wslot = 0;
  };
  auto issue_patch = [&](int c, int buf) {
    uint4* dst = patch + buf * PSTAGE;
    const bool live = c < nslices;
    const uint32_t add = (uint32_t)c * 128u;
#pragma unroll
    for (int i = 0; i < LP; ++i)
      lds_fill16(xr, __builtin_amdgcn_readfirstlane(lds_addr(dst + (i * kWaves + wave) * 64)),
                 live ? poff[i] + add : kOOB);
  };

  Acc acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = Acc{0, 0, 0, 0};

  // One tap: 2 k-steps of the MFMA (64 bytes each).  Lane l reads 16 bytes
  // of row l % 16 at chunk (k-step, l / 16).
  auto compute = [&](const uint4* sP, const uint4* sW, int toff, int tkey) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int chunk = ks * 4 + (lane >> 4);
      uint4 af[TN], bfr[TM];
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int row = wn * WTN + i * 16 + (lane & 15);
        af[i] = sW[row * 8 + (chunk ^ (row & 7))];
      }
#pragma unroll
      for (int j = 0; j < TM; ++j) {
        const int pp = pbase[j] + toff;
        bfr[j] = sP[pp * 8 + (chunk ^ ((cbase[j] + tkey) & 7))];
      }
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j) acc[i][j] = mma(af[i], bfr[j], acc[i][j]);
    }
  };

  // Epilogue operands (bias and residual of the 8 channels this thread
  // finishes per pass) are fetched before the main loop.
  constexpr int kEC = 32;  // channels per epilogue pass
  constexpr int NPASS = BN / kEC;
  constexpr int TPP = kEC / 8;  // threads per pixel
  constexpr int EPV = (BM * TPP + kNT - 1) / kNT;  // pixels per thread per pass
  const int ec8 = (tid % TPP) * 8;
  using RT = std::conditional_t<I8, uint2, uint4>;  // the residual of 8 channels
  RT resv[NPASS][EPV];
  {
    const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16_t*>(p.res), (short)0, p.res ? p.res_bytes : 0, kBufferFlags);
#pragma unroll
    for (int pass = 0; pass < NPASS; ++pass) {
      const int k = n0 + pass * kEC + ec8;
#pragma unroll
      for (int e = 0; e < EPV; ++e) {
        const int px = (tid + e * kNT) / TPP;
        const int m = m0 + px;
        const uint32_t off = (px < BM && m < p.M && k < p.Kp) ? (uint32_t)(m * p.ldr + k) * ES : kOOB;
        if constexpr (I8)
          resv[pass][e] = p.res ? __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rr, off, 0, 0))
                                : make_uint2(0u, 0u);
        else
          resv[pass][e] = p.res ? __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rr, off, 0, 0))
                                : make_uint4(0u, 0u, 0u, 0u);
      }
    }
  }
  // the tile's bias (codes: {bias, factor} table), straight into LDS (zeros without a bias)
  if (tid < 64) {
    if constexpr (I8) {
      const i32x4 br = buffer_rsrc(q.qch, ((p.Kp + 255) / 256) * 256 * 8);
      const uint32_t off = lane < BN / 2 ? (uint32_t)(n0 + 2 * lane) * 8u : kOOB;
      lds_fill16(br, __builtin_amdgcn_readfirstlane(lds_addr(sbias)), off);
    } else {
      const i32x4 br = buffer_rsrc(p.bias, p.bias ? ((p.Kp + 255) / 256) * 256 * 4 : 0);
      const uint32_t off = lane < BN / 4 ? (uint32_t)(n0 + 4 * lane) * 4u : kOOB;
      lds_fill16(br, __builtin_amdgcn_readfirstlane(lds_addr(sbias)), off);
    }
  }
  issue_patch(0, 0);
  static_for<0, NSW - 1>([&](auto) { issue_w(); });

  int cslot = 0;  // ring slot of the stage computed next
  for (int c = 0; c < nslices; ++c) {
    const int pb = NPB == 2 ? (c & 1) : 0;
    const uint4* sP = patch + pb * PSTAGE;
    static_for<0, SPS>([&](auto tt) {
      constexpr int t = decltype(tt)::value;
      // loads younger than this stage's weights: the NSW - 2 weight stages
      // after it, and the next slice's patch while it was issued after them
      constexpr int vm = (NSW - 2) * LW + ((NPB == 2 && t >= 1 && t <= NSW - 1) ? LP : 0);
      asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(vm) : "memory");
      issue_w();
      if constexpr (t == 0 && NPB == 2) issue_patch(c + 1, pb ^ 1);
      const uint4* sW = wring + cslot * WSTAGE;
      static_for<0, TPS>([&](auto uu) {
        constexpr int tap = t * TPS + decltype(uu)::value;
        compute(sP, sW + decltype(uu)::value * WTAP, (tap / 3) * WP + (tap % 3), (tap / 3) * p.W + (tap % 3));
      });
      if (++cslot == NSW) cslot = 0;
    });
  }
  // all fills (including the zero fills past the end) landed, all waves
  // done reading the operand buffers
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");

  // Epilogue through LDS: the fp32 sums of a 32-channel slice are parked in
  // a [BM][kEC + 4] tile in the operand buffers; every thread then takes 8
  // consecutive channels of one pixel, adds bias and residual, applies the
  // activation and stores 16 bytes.
  constexpr int kLd = kEC + 4;
  static_assert(BM * kLd * 4 <= (NPB * PSTAGE + NSW * WSTAGE) * 16, "staging tile");
  if constexpr (I8) {
    int* stage = reinterpret_cast<int*>(lds);
#pragma unroll
    for (int pass = 0; pass < NPASS; ++pass) {
      if (pass > 0) lds_barrier();
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int ch = wn * WTN + i * 16 + 4 * (lane >> 4) - pass * kEC;
        if (ch < 0 || ch >= kEC) continue;
#pragma unroll
        for (int j = 0; j < TM; ++j) {
          const int px = wm * WTM + j * 16 + (lane & 15);
          *(i32x4*)(stage + px * kLd + ch) = acc[i][j];
        }
      }
      lds_barrier();
      const int k = n0 + pass * kEC + ec8;
#pragma unroll
      for (int e = 0; e < EPV; ++e) {
        const int px = (tid + e * kNT) / TPP;
        const int m = m0 + px;
        if (px >= BM || m >= p.M || k >= p.Kp) continue;
        const int* st = stage + px * kLd + ec8;
        const int4 lo4 = *(const int4*)st, hi4 = *(const int4*)(st + 4);
        int a[8] = {lo4.x, lo4.y, lo4.z, lo4.w, hi4.x, hi4.y, hi4.z, hi4.w};
        *(uint2*)(reinterpret_cast<int8_t*>(p.y) + (size_t)m * p.ldy + k) =
            finish8_i8(a, reinterpret_cast<const int2*>(sbias) + pass * kEC + ec8, resv[pass][e], q, m, k);
      }
    }
    return;
  } else {
  float* stage = reinterpret_cast<float*>(lds);
  const ActClamp ac = act_clamp_of(p.act, p.alpha);
  auto epilogue = [&](auto mode_tag) {
    constexpr int G = decltype(mode_tag)::value;
#pragma unroll
    for (int pass = 0; pass < NPASS; ++pass) {
      if (pass > 0) lds_barrier();
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int ch = wn * WTN + i * 16 + 4 * (lane >> 4) - pass * kEC;
        if (ch < 0 || ch >= kEC) continue;
#pragma unroll
        for (int j = 0; j < TM; ++j) {
          const int px = wm * WTM + j * 16 + (lane & 15);
          const f32x4 a = acc[i][j];
          *(float4*)(stage + px * kLd + ch) = make_float4(a[0], a[1], a[2], a[3]);
        }
      }
      lds_barrier();
      const int k = n0 + pass * kEC + ec8;
#pragma unroll
      for (int e = 0; e < EPV; ++e) {
        const int px = (tid + e * kNT) / TPP;
        const int m = m0 + px;
        if (px >= BM || m >= p.M || k >= p.Kp) continue;
        const float* st0 = stage + px * kLd + ec8;
        const float4 lo = *(const float4*)st0;
        const float4 hi = *(const float4*)(st0 + 4);
        float f[8], rv[8];
        const float4 b0 = sbias[(pass * kEC + ec8) / 4], b1 = sbias[(pass * kEC + ec8) / 4 + 1];
        unpack8(resv[pass][e], rv);
        f[0] = lo.x + b0.x; f[1] = lo.y + b0.y; f[2] = lo.z + b0.z; f[3] = lo.w + b0.w;
        f[4] = hi.x + b1.x; f[5] = hi.y + b1.y; f[6] = hi.z + b1.z; f[7] = hi.w + b1.w;
#pragma unroll
        for (int e = 0; e < 8; ++e) f[e] = epilogue_value<G>(f[e], rv[e], ac);
        *(uint4*)(p.y + (size_t)m * p.ldy + k) = pack8(f);
      }
    }
  };
  if (p.res_post)
    epilogue(std::integral_constant<int, 3>{});
  else if (act_mode(p.act) == 1)
    epilogue(std::integral_constant<int, 1>{});
  else if (act_mode(p.act) == 0)
    epilogue(std::integral_constant<int, 0>{});
  else
    epilogue(std::integral_constant<int, 2>{});
  }
}

// A weight-ring setting `stages` of the launchers: 2 or 3 are rings of
// whole kernel rows (three taps per stage), 4, 6 or 8 rings of single taps.
constexpr int taps_per_stage(int stages) { return stages <= 3 ? 3 : 1; }

// LDS bytes of one instantiation.
constexpr int halo_lds(int bn, int tps, int nsw, int lp, int npb, int waves) {
  return npb * lp * waves * 8 * 128 + nsw * tps * bn * 128 + 64 * 16;  // + the bias table (one wave's fill)
}

// Patch pixels of the largest tile of a BM-pixel tiling.
int max_patch_pixels(const ConvParams& p, int bm) {
  const int PQ = p.P * p.Q, HP = p.H + 2, WP = p.W + 2;
  int best = 0;
  for (int m0 = 0; m0 < p.M; m0 += bm) {
    const int ml = std::min(m0 + bm, p.M) - 1;
    const int nf = m0 / PQ, pf = (m0 - nf * PQ) / p.Q;
    const int nl = ml / PQ, pl = (ml - nl * PQ) / p.Q;
    best = std::max(best, (nl * HP + pl + 2 - (nf * HP + pf) + 1) * WP);
  }
  return best;
}

constexpr int kHaloWaves = 8;
constexpr int kLPs[] = {4, 5, 6, 8};  // 128-pixel tiles
constexpr int kLPs64[] = {3, 4};      // 64-pixel tiles

// Smallest patch capacity (loads per thread) that holds every tile's patch
// and fits the LDS with `nsw` weight stages; 0 if none.
int choose_lp(const ConvParams& p, int bm, int bn, int stages, int* npb, int cs) {
  *npb = p.Cp / cs > 1 ? 2 : 1;
  const int need = max_patch_pixels(p, bm);
  auto fits = [&](int lp) {
    return lp * kHaloWaves * 8 >= need &&
           halo_lds(bn, taps_per_stage(stages), stages, lp, *npb, kHaloWaves) <= kLdsLimit;
  };
  if (bm == 64) {
    for (int lp : kLPs64)
      if (fits(lp)) return lp;
    return 0;
  }
  for (int lp : kLPs)
    if (fits(lp)) return lp;
  return 0;
}

bool shape_ok(const ConvParams& p, int cs) {
  return p.R == 3 && p.S == 3 && p.sh == 1 && p.sw == 1 && p.pt == 1 && p.pl == 1 && p.P == p.H &&
         p.Q == p.W && p.Cp % cs == 0 && p.splits == 1 && p.Kg == 9 * p.Cp;
}

template <int BM, int BN, int WM, int WN, int TPS, int NSW, int LP, int NPB, bool I8>
hipError_t launch_one(const QConvParams& q_in, hipStream_t s) {
  if constexpr (halo_lds(BN, TPS, NSW, LP, NPB, WM * WN) > kLdsLimit) {
    return hipErrorInvalidValue;
  } else {
    QConvParams q = q_in;
    ConvParams& p = q.g;
    p.mg_wp = magic40(p.W + 2);
    p.mg_hp = magic40(p.H + 2);
    const int blocks = placed_blocks(p, BM, BN);
    conv_halo_kernel<BM, BN, WM, WN, TPS, NSW, LP, NPB, I8><<<blocks, 64 * WM * WN, 0, s>>>(q);
    return hipGetLastError();
  }
}

template <int STAGES, bool I8>
hipError_t launch_stages(const QConvParams& q, int bm, int lp, int npb, hipStream_t s) {
  constexpr int T = taps_per_stage(STAGES);
  if (bm == 64) {  // 64-pixel tiles (8 waves of 16 pixels x 32 channels): rings of kernel rows only
    if constexpr (STAGES == 2 || STAGES == 3) {
      if (npb == 2) {
        if (lp == 3) return launch_one<64, 64, 4, 2, T, STAGES, 3, 2, I8>(q, s);
        if (lp == 4) return launch_one<64, 64, 4, 2, T, STAGES, 4, 2, I8>(q, s);
      } else {
        if (lp == 3) return launch_one<64, 64, 4, 2, T, STAGES, 3, 1, I8>(q, s);
        if (lp == 4) return launch_one<64, 64, 4, 2, T, STAGES, 4, 1, I8>(q, s);
      }
    }
    return hipErrorInvalidValue;
  }
  if (npb == 2) {
    if (lp == 4) return launch_one<128, 64, 4, 2, T, STAGES, 4, 2, I8>(q, s);
    if (lp == 5) return launch_one<128, 64, 4, 2, T, STAGES, 5, 2, I8>(q, s);
    if (lp == 6) return launch_one<128, 64, 4, 2, T, STAGES, 6, 2, I8>(q, s);
    return hipErrorInvalidValue;
  }
  if (lp == 4) return launch_one<128, 64, 4, 2, T, STAGES, 4, 1, I8>(q, s);
  if (lp == 5) return launch_one<128, 64, 4, 2, T, STAGES, 5, 1, I8>(q, s);
  if (lp == 6) return launch_one<128, 64, 4, 2, T, STAGES, 6, 1, I8>(q, s);
  if (lp == 8) return launch_one<128, 64, 4, 2, T, STAGES, 8, 1, I8>(q, s);
  return hipErrorInvalidValue;
}

template <bool I8>
hipError_t launch_any(const QConvParams& q, int bm, int bn, int stages, int lp, int npb, hipStream_t s) {
  if ((bm != 128 && bm != 64) || bn != 64 || !shape_ok(q.g, I8 ? 128 : kSlice)) return hipErrorInvalidValue;
  if (stages == 2) return launch_stages<2, I8>(q, bm, lp, npb, s);
  if (stages == 3) return launch_stages<3, I8>(q, bm, lp, npb, s);
  if (stages == 4) return launch_stages<4, I8>(q, bm, lp, npb, s);
  if (stages == 6) return launch_stages<6, I8>(q, bm, lp, npb, s);
  if (stages == 8) return launch_stages<8, I8>(q, bm, lp, npb, s);
  return hipErrorInvalidValue;
}

}  // namespace

bool conv_halo_plan(const ConvParams& p, int bm, int bn, int stages, int* lp, int* npb, bool i8) {
  const int cs = i8 ? 128 : kSlice;
  // 128 x 64 tiles at every ring depth; 64 x 64 tiles with rings of kernel rows
  if (!(bm == 128 || (bm == 64 && (stages == 2 || stages == 3))) || bn != 64 || !shape_ok(p, cs)) return false;
  if (stages != 2 && stages != 3 && stages != 4 && stages != 6 && stages != 8) return false;
  // index math: patch offsets and pixel bases stay within int32
  if ((int64_t)p.N * (p.H + 2) * (p.W + 2) >= (int64_t(1) << 30)) return false;
  *lp = choose_lp(p, bm, bn, stages, npb, cs);
  return *lp > 0;
}

hipError_t launch_conv_halo(const ConvParams& p, int bm, int bn, int stages, int lp, int npb, hipStream_t s) {
  QConvParams q{};
  q.g = p;
  return launch_any<false>(q, bm, bn, stages, lp, npb, s);
}

hipError_t launch_conv_halo_i8(const QConvParams& q, int bm, int bn, int stages, int lp, int npb, hipStream_t s) {
  return launch_any<true>(q, bm, bn, stages, lp, npb, s);
}

}  // namespace byoc
