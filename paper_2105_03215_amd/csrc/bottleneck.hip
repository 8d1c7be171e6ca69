// Fused ResNet bottleneck block: 1x1 reduce, 3x3, 1x1 expand with the
// block input (or a 1x1 projection of it) added back, as one kernel.
//
// The composites of a bottleneck block are planned as separate launches
// elsewhere; here they run in one workgroup per tile of output pixels, and
// the narrow intermediates and the projection live only in LDS and
// registers (the engine owns an offloaded subgraph's intermediates, Sec.
// 3.4, so they need not exist in memory).  Of the HBM traffic of the
// separate launches - x read two or three times, the intermediates written
// and read back, y written - one read of x (plus the halo) and the write of
// y remain.
//
// A workgroup owns a TH x TW tile of output pixels of one image.  The first
// 1x1 and the projection may have stride S (2: a downsampling block); the
// rest runs on the output grid.
//
// Phase A (1x1 reduce): the tile's halo - (TH + 2) x (TW + 2) positions of
// the output grid, i.e. input pixels S apart - times W1, streamed one
// 64-channel slice of x at a time through a ring of LDS stages (x slice and
// W1 slice per stage, HBM -> LDS loads).  The sums are finished (bias,
// activation, bf16 rounding) into M1 in LDS; positions outside the image
// are stored as zeros, the 3x3's zero padding.  While each x slice is
// staged, the threads copy the tile's own pixels of it into registers: the
// residual of phase C (identity shortcut), or the MFMA operand fragments of
// the projection (projection shortcut).
//
// Phase B (3x3): nine shifted views of M1 times W2, streamed through a ring
// of stages of TPS taps x SPB 64-channel slices (tap by tap, then slice);
// the output tile is finished into M2 in LDS.
//
// Phase C (1x1 expand): M2 times W3, F output channels per chunk, the
// weights streamed one 64-channel slice (of M2, then of x for the
// projection) per stage; with the projection shortcut the chunk's
// projection is summed from the registers of phase A and finished (bias,
// bf16 rounding) as the projection composite stores it; then bias, the
// residual, activation, bf16 stores to y.
//
// Operands of every product: weights are the MFMA A operand (16 output
// channels), pixels the B operand, so each lane ends with 4 consecutive
// channels of one pixel.  A wave owns one 64-channel group of the output
// channels of each product and a set of 16-pixel tiles.  Every LDS row is
// 128 bytes (64 channels) with its 16-byte chunks permuted by a per-row key
// so that the 16 rows one MFMA operand read touches spread over the banks.
//
// Reduction order of each output: phase A and the projection slice by slice of x (32
// channels per MFMA step), phase B tap by tap then channel, phase C channel -
// the order of the single-group implicit-GEMM kernel on the same composites.
#include <cstdio>

#include "lds_dma.h"

namespace byoc {
namespace {

using namespace dma;

typedef __attribute__((ext_vector_type(2))) unsigned int u32x2;

constexpr int cmin(int a, int b) { return a < b ? a : b; }
constexpr int cmax(int a, int b) { return a > b ? a : b; }

template <int F_, int CIN_, int COUT_, int S_, int TH_, int TW_, int NW_, int NSA_, int TPS_, int SPB_, int NSB_>
struct Bn {
  static constexpr int F = F_, CIN = CIN_, COUT = COUT_, S = S_, TH = TH_, TW = TW_, NW = NW_;
  static constexpr int NSA = NSA_, TPS = TPS_, SPB = SPB_, NSB = NSB_;  // rings and stages
  static constexpr bool PROJ = COUT != CIN || S != 1;  // projection shortcut
  static constexpr int NT = 64 * NW;
  static constexpr int WGC = F / 64;   // 64-channel groups of the mid width (a wave owns one)
  static constexpr int WP = NW / WGC;  // waves per group
  static constexpr int HC = TW + 2, HR = TH + 2;
  static constexpr int HPX = HR * HC;  // halo positions
  static constexpr int HPXP = (HPX + 15) / 16 * 16;
  static constexpr int OPX = TH * TW;  // output pixels
  static constexpr int OPXP = (OPX + 15) / 16 * 16;
  static constexpr int NTA = HPXP / 16, NTB = OPXP / 16;  // 16-pixel tiles
  static constexpr int TA = (NTA + WP - 1) / WP;          // pixel tiles per wave, phase A
  static constexpr int TB = (NTB + WP - 1) / WP;          // phases B and C
  static constexpr int SA = CIN / 64;                     // phase A stages (x slices)
  static constexpr int PFA = NSA >= 2 ? NSA - 1 : 1;      // phase A stages issued ahead
  static constexpr int NQ = COUT / F;                     // phase C chunks (F output channels each)
  static constexpr int CSL = PROJ ? 1 : WGC;              // 64-channel slices per phase C stage
  static constexpr int UQ = (WGC + (PROJ ? SA : 0)) / CSL;  // phase C stages per chunk: W3, then Wp slices
  static constexpr int SC = NQ * UQ;                      // phase C stages
  static constexpr int GB = WGC / SPB;                    // slice groups of a tap
  static constexpr int SB = 9 / TPS * GB;                 // phase B stages
  static constexpr int XF = PROJ ? 2 * SA : 1;            // projection fragments per pixel tile
  static constexpr int ROW = 128;
  // LDS plan (bytes)
  static constexpr int M1B = WGC * HPXP * ROW;
  static constexpr int XB = HPXP * ROW;
  static constexpr int W1B = F * ROW;
  static constexpr int ASTG = XB + W1B;
  static constexpr int W2B = TPS * SPB * F * ROW;
  static constexpr int M2B = WGC * OPXP * ROW;
  static constexpr int CB = CSL * F * ROW;  // phase C stage: F rows of a chunk x CSL x 64 input channels
  static constexpr int OFF_R2 = M1B;  // the phase A ring, then the W2 ring and M2
  static constexpr int OFF_M2 = OFF_R2 + NSB * W2B;
  static constexpr int END_A = OFF_R2 + NSA * ASTG;
  static constexpr int END_B = OFF_M2 + M2B;
  static constexpr int NSC = cmin(OFF_M2 / CB, SC);  // phase C ring, over M1 and the W2 ring
  static constexpr int OFF_BIAS = cmax(END_A, END_B);
  static constexpr int B3BLK = (COUT * 4 + 1023) / 1024;
  static constexpr int BBLK = 2 + (PROJ ? 2 : 1) * B3BLK;  // 1 KB blocks: b1, b2, b3 (, bp)
  static constexpr int OFF_JUNK = OFF_BIAS + BBLK * 1024;
  static constexpr int LDS = OFF_JUNK + 1024;
  // 1 KB fills (8 rows of 128 bytes) per stage and per thread
  static constexpr int XBLK = HPXP / 8, W1BLK = F / 8, W2BLK = TPS * SPB * F / 8, CBLK = CSL * F / 8;
  static constexpr int LXA = (XBLK + NW - 1) / NW, LW1 = (W1BLK + NW - 1) / NW;
  static constexpr int LA = LXA + LW1;
  static constexpr int LB = (W2BLK + NW - 1) / NW;
  static constexpr int LC = (CBLK + NW - 1) / NW;
  static constexpr int ST = TB * 4;  // y stores per chunk per thread
  // Identity blocks finish a chunk after the next chunk's first stage
  // (DEFER), projection blocks at the chunk's last stage; does stage i
  // store a chunk?
  static constexpr bool DEFER = !PROJ;
  static constexpr bool stores_at(int i) { return DEFER ? (i % UQ == 0 && i >= UQ) : (i % UQ == UQ - 1); }
  // Vector memory operations a thread may have outstanding after phase C
  // stage k's loads: the loads of the stages issued ahead of it, and the
  // y stores of the chunks finished since it was issued (stage i issues
  // stage i + NSC - 1 after its wait, then computes, then stores).
  static constexpr int c_younger(int k) {
    int stores = 0;
    for (int i = cmax(0, k - NSC + 1); i < k; ++i) stores += stores_at(i) ? ST : 0;
    return cmin(NSC - 2, SC - 1 - k) * LC + stores;
  }
  static constexpr int c_younger_max() {
    int m = 0;
    for (int k = 0; k < SC; ++k) m = cmax(m, c_younger(k));
    return m;
  }

  static_assert(F % 64 == 0 && CIN % 64 == 0 && COUT % F == 0 && NW % WGC == 0, "shape");
  static_assert(PROJ || CIN % F == 0, "identity shortcut: chunks of F channels");
  static_assert(9 % TPS == 0 && ((NSA >= 2 && NSA <= SA) || (NSA == 1 && SA == 1)), "phase A stages");
  static_assert(NSB >= 2 && NSB <= SB, "phase B stages");
  static_assert(WGC % SPB == 0 && (TPS == 1 || SPB == WGC), "phase B stages run tap by tap, then slice");
  static_assert(NSC >= 2, "phase C ring");
  static_assert(BBLK <= NW, "one bias fill per wave");
  static_assert(LDS <= kLdsLimit, "LDS");
  static_assert((PFA - 1) * LA <= 63 && (NSB - 2) * LB <= 63 && c_younger_max() <= 63, "vmcnt immediate");
};

// rows r of a 128-byte-row buffer keep logical 16-byte chunk c at slot c ^ key
__device__ __forceinline__ uint32_t slot_off(int row, int chunk, int key) {
  return (uint32_t)(row * 128 + ((chunk ^ (key & 7)) << 4));
}

// A ring stage is complete for this thread and - after the barrier - for
// the whole workgroup, once at most `YOUNGER` of the thread's later vector
// memory operations are outstanding.
template <int YOUNGER>
__device__ __forceinline__ void stage_barrier() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(YOUNGER) : "memory");
}

template <class B>
__global__ __launch_bounds__(B::NT) void bottleneck_kernel(BottleneckParams p) {
  constexpr int F = B::F, CIN = B::CIN, TW = B::TW, HC = B::HC, NW = B::NW, WP = B::WP;
  __shared__ __attribute__((aligned(1024))) char lds[B::LDS];
  asm volatile("" ::"s"(p.x), "s"(p.y), "s"(p.w1), "s"(p.w2), "s"(p.w3), "s"(p.b1), "s"(p.b2), "s"(p.b3));
  asm volatile("" ::"s"(p.N), "s"(p.H), "s"(p.W), "s"(p.P), "s"(p.Q), "s"(p.ld1), "s"(p.ld2), "s"(p.ld3),
               "s"(p.x_bytes), "s"(p.y_bytes), "s"(p.w1_bytes), "s"(p.w2_bytes), "s"(p.w3_bytes));
  if constexpr (B::PROJ) asm volatile("" ::"s"(p.wp), "s"(p.bp), "s"(p.ldp), "s"(p.wp_bytes), "s"(p.bp_bytes));
  asm volatile("" ::"s"(p.b1_bytes), "s"(p.b2_bytes), "s"(p.b3_bytes), "s"(p.act1), "s"(p.act2), "s"(p.act3),
               "s"(p.alpha1), "s"(p.alpha2), "s"(p.alpha3), "s"(p.tiles_w), "s"(p.tiles_hw), "s"(p.mg_tw),
               "s"(p.mg_thw), "s"(p.tiles), "s"(p.per_xcd));

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int l16 = lane & 15, lk = lane & 7, lq = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int cg = wave % B::WGC, wp = wave / B::WGC;

  // the tile: the hardware deals workgroups round-robin to the 8 XCDs, so
  // XCD x takes the contiguous run of tiles [x * per_xcd, (x + 1) * per_xcd):
  // neighbouring tiles, which read each other's halo rows, share an L2
  const int tile = (blockIdx.x & 7) * p.per_xcd + (blockIdx.x >> 3);
  if (tile >= p.tiles) return;
  const int n = mdiv(tile, p.mg_thw);
  const int tr = tile - n * p.tiles_hw;
  const int th = mdiv(tr, p.mg_tw);
  const int h0 = th * B::TH, w0 = (tr - th * p.tiles_w) * TW;  // on the output grid
  const int H = p.H, W = p.W, P = p.P, Q = p.Q;

  const uint32_t base = lds_addr(lds);
  const uint32_t junk = base + B::OFF_JUNK;
  const float* sb1 = reinterpret_cast<const float*>(lds + B::OFF_BIAS);
  const float* sb2 = sb1 + 256;
  const float* sb3 = sb1 + 512;
  const float* sbp = sb3 + 256 * B::B3BLK;  // projection bias

  // ---- load plans: per-thread source offsets, wave-uniform destinations ----
  const i32x4 xr = buffer_rsrc(p.x, p.x_bytes);
  const i32x4 w1r = buffer_rsrc(p.w1, p.w1_bytes);
  const i32x4 w2r = buffer_rsrc(p.w2, p.w2_bytes);
  const i32x4 w3r = buffer_rsrc(p.w3, p.w3_bytes);
  const i32x4 wpr = buffer_rsrc(p.wp, B::PROJ ? p.wp_bytes : 0);
  uint32_t xoff[B::LXA], w1off[B::LW1], w2off[B::LB], w3off[B::LC], wpoff[B::LC];
#pragma unroll
  for (int u = 0; u < B::LXA; ++u) {
    const int blk = wave + NW * u;
    const int px = 8 * blk + (lane >> 3);
    uint32_t off = kOOB;
    if (blk < B::XBLK && px < B::HPX) {
      const int hr = px / HC, hc = px - (px / HC) * HC;
      const int mh = h0 - 1 + hr, mw = w0 - 1 + hc;  // position on the output grid
      if ((unsigned)mh < (unsigned)P && (unsigned)mw < (unsigned)Q)
        off = (uint32_t)((((n * H + B::S * mh) * W + B::S * mw) * CIN + ((lk ^ (px & 7)) * 8)) * 2);
    }
    xoff[u] = off;
  }
  // rows 8 * blk + lane / 8 of a weight block, chunk lk at slot lk ^ (row & 7)
  auto row_off = [&](int blk, int nblk, int ld, int col) {
    const int row = 8 * blk + (lane >> 3);
    return blk < nblk ? (uint32_t)((row * ld + col + ((lk ^ (row & 7)) * 8)) * 2) : kOOB;
  };
#pragma unroll
  for (int u = 0; u < B::LW1; ++u) w1off[u] = row_off(wave + NW * u, B::W1BLK, p.ld1, 0);
#pragma unroll
  for (int u = 0; u < B::LB; ++u) {
    const int blk = wave + NW * u;  // [tap u][slice sl][F rows]
    const int tap = blk / (B::SPB * F / 8), rem = blk - tap * (B::SPB * F / 8);
    const int sl = rem / (F / 8);
    w2off[u] = blk < B::W2BLK ? row_off(rem - sl * (F / 8), F / 8, p.ld2, tap * F + sl * 64) : kOOB;
  }
#pragma unroll
  for (int u = 0; u < B::LC; ++u) {  // [slice sl][F rows of a chunk] of W3 (of Wp: one slice)
    const int blk = wave + NW * u;
    const int sl = blk / (F / 8);
    w3off[u] = blk < B::CBLK ? row_off(blk - sl * (F / 8), F / 8, p.ld3, sl * 64) : kOOB;
    wpoff[u] = B::PROJ ? row_off(blk, B::CBLK, p.ldp, 0) : kOOB;
  }
  auto dst = [&](uint32_t region, int blk, int nblk) {
    return __builtin_amdgcn_readfirstlane(blk < nblk ? region + blk * 1024 : junk);
  };
  auto live = [](uint32_t off, uint32_t add) { return off == kOOB ? kOOB : off + add; };
  auto issue_a = [&](int s) {
    const uint32_t slot = base + B::OFF_R2 + (s % B::NSA) * B::ASTG;
#pragma unroll
    for (int u = 0; u < B::LXA; ++u) lds_fill16(xr, dst(slot, wave + NW * u, B::XBLK), live(xoff[u], s * 128));
#pragma unroll
    for (int u = 0; u < B::LW1; ++u)
      lds_fill16(w1r, dst(slot + B::XB, wave + NW * u, B::W1BLK), live(w1off[u], s * 128));
  };
  auto issue_b = [&](int s) {
    const uint32_t slot = base + B::OFF_R2 + (s % B::NSB) * B::W2B;
#pragma unroll
    for (int u = 0; u < B::LB; ++u)
      lds_fill16(w2r, dst(slot, wave + NW * u, B::W2BLK),
                 live(w2off[u], ((s / B::GB) * B::TPS * F + (s % B::GB) * B::SPB * 64) * 2));
  };
  auto issue_c = [&](int k) {  // chunk k / UQ: stage j = k % UQ, W3 slices j * CSL .. (j < WGC / CSL), else Wp
    const uint32_t slot = base + (k % B::NSC) * B::CB;
    const int q = k / B::UQ, j = k % B::UQ;
    if (j * B::CSL < B::WGC) {
#pragma unroll
      for (int u = 0; u < B::LC; ++u)
        lds_fill16(w3r, dst(slot, wave + NW * u, B::CBLK),
                   live(w3off[u], (q * F * p.ld3 + j * B::CSL * 64) * 2));
    } else {
#pragma unroll
      for (int u = 0; u < B::LC; ++u)
        lds_fill16(wpr, dst(slot, wave + NW * u, B::CBLK),
                   live(wpoff[u], (q * F * p.ldp + (j - B::WGC) * 64) * 2));
    }
  };

  // biases: wave w < BBLK fills one 1 KB block (b1, b2, the blocks of b3, then those of bp)
  {
    const bool pb = wave >= 2 + B::B3BLK;
    const void* src = wave == 0 ? (const void*)p.b1
                      : wave == 1 ? (const void*)p.b2
                      : pb        ? (const void*)p.bp
                                  : (const void*)p.b3;
    const int bytes = wave == 0 ? p.b1_bytes : wave == 1 ? p.b2_bytes : pb ? p.bp_bytes : p.b3_bytes;
    const int blk = wave < 2 ? 0 : pb ? wave - 2 - B::B3BLK : wave - 2;
    const uint32_t off = wave < B::BBLK ? (uint32_t)(blk * 1024 + lane * 16) : kOOB;
    lds_fill16(buffer_rsrc(src, bytes), dst(base + B::OFF_BIAS, wave, B::BBLK), off);
  }

  const ActClamp ac1 = act_clamp_of(p.act1, p.alpha1);
  const ActClamp ac2 = act_clamp_of(p.act2, p.alpha2);
  const ActClamp ac3 = act_clamp_of(p.act3, p.alpha3);

  // this lane's output pixel in each of the wave's pixel tiles (phases B and
  // C): its halo row (0 past the tile)
  int hrow[B::TB];
#pragma unroll
  for (int t = 0; t < B::TB; ++t) {
    const int o = 16 * (wp + WP * t) + l16;
    hrow[t] = o < B::OPX ? (o / TW + 1) * HC + (o % TW) + 1 : 0;
  }

  // ---- phase A: M1 = act1(halo x W1 + b1) -----------------------------------
  f32x4 accA[B::TA][4];
#pragma unroll
  for (int t = 0; t < B::TA; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) accA[t][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  // identity shortcut: the residual of phase C per chunk, 4 bf16 channels of
  // one pixel per (chunk, pixel tile, channel tile)
  uint2 resv[B::PROJ ? 1 : B::NQ][B::TB][4];
  uint4 xf[B::TB][B::XF];  // projection: x at the tile's pixels as MFMA B fragments, per 32-channel step

  static_for<0, B::PFA>([&](auto s) {
    if constexpr (decltype(s)::value < B::SA) issue_a(decltype(s)::value);
  });
  static_for<0, B::SA>([&](auto ss) {
    constexpr int s = decltype(ss)::value;
    stage_barrier<cmin(B::PFA - 1, B::SA - 1 - s) * B::LA>();
    if constexpr (B::NSA >= 2 && s + B::PFA < B::SA) issue_a(s + B::PFA);
    const char* xs = lds + B::OFF_R2 + (s % B::NSA) * B::ASTG;
    const char* ws = xs + B::XB;
    if constexpr (B::PROJ) {
#pragma unroll
      for (int t = 0; t < B::TB; ++t)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) xf[t][2 * s + ks] = *(const uint4*)(xs + slot_off(hrow[t], ks * 4 + lq, hrow[t]));
    } else if (cg == s % B::WGC) {  // this slice is the residual of the wave's channel group in chunk s / WGC
#pragma unroll
      for (int t = 0; t < B::TB; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          resv[B::PROJ ? 0 : s / B::WGC][t][i] =
              *(const uint2*)(xs + slot_off(hrow[t], 2 * i + (lane >> 5), hrow[t]) + (lq & 1) * 8);
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int c = ks * 4 + lq;
      bf16x8 a[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = as_bf16x8(*(const uint4*)(ws + slot_off(cg * 64 + 16 * i + l16, c, lk)));
#pragma unroll
      for (int t = 0; t < B::TA; ++t) {
        const int j = wp + WP * t;
        if (j < B::NTA) {
          const bf16x8 b = as_bf16x8(*(const uint4*)(xs + slot_off(16 * j + l16, c, lk)));
#pragma unroll
          for (int i = 0; i < 4; ++i) accA[t][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b, accA[t][i], 0, 0, 0);
        }
      }
    }
  });
  // every wave is done with the phase A ring: the next ring may overwrite it
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  static_for<0, B::NSB - 1>([&](auto s) { issue_b(decltype(s)::value); });
  // biases into registers before the first M1 store (a later LDS read could
  // not move above a store the compiler cannot tell apart from it)
  float4 bias[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) bias[i] = *(const float4*)(sb1 + cg * 64 + 16 * i + 4 * lq);
#pragma unroll
  for (int t = 0; t < B::TA; ++t) {
    const int j = wp + WP * t;
    if (j >= B::NTA) continue;
    const int px = 16 * j + l16;
    const int hr = px / HC, hc = px - (px / HC) * HC;
    const int mh = h0 - 1 + hr, mw = w0 - 1 + hc;
    const bool inside = px < B::HPX && (unsigned)mh < (unsigned)P && (unsigned)mw < (unsigned)Q;
    const int key = hr * TW + hc;
    char* m1 = lds + cg * B::HPXP * 128;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float4 bb = bias[i];
      const f32x4 v = accA[t][i];
      // (+ 0: the unfused epilogue adds its zero residual, which turns a -0 into +0)
      float f0 = act_apply<2>((v[0] + bb.x) + 0.f, ac1), f1 = act_apply<2>((v[1] + bb.y) + 0.f, ac1);
      float f2 = act_apply<2>((v[2] + bb.z) + 0.f, ac1), f3 = act_apply<2>((v[3] + bb.w) + 0.f, ac1);
      if (!inside) f0 = f1 = f2 = f3 = 0.f;
      *(uint2*)(m1 + slot_off(px, 2 * i + (lane >> 5), key) + (lq & 1) * 8) =
          make_uint2(pack2_bf16(f0, f1), pack2_bf16(f2, f3));
    }
  }

  // ---- phase B: M2 = act2(conv3x3(M1) W2 + b2) -------------------------------
  // Phases B and C run every one of a wave's TB pixel tiles (a tile past the
  // last reads row 0 and is never stored): no branches between the LDS reads
  // of a step and its MFMAs.
  int pbase[B::TB], obase[B::TB];
#pragma unroll
  for (int t = 0; t < B::TB; ++t) {
    const int o = 16 * (wp + WP * t) + l16;
    const bool ok = o < B::OPX;
    pbase[t] = ok ? (o / TW) * HC + (o % TW) : 0;
    obase[t] = ok ? o : 0;
  }
  f32x4 accB[B::TB][4];
#pragma unroll
  for (int t = 0; t < B::TB; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) accB[t][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  static_for<0, B::SB>([&](auto ss) {
    constexpr int s = decltype(ss)::value;
    stage_barrier<cmin(B::NSB - 2, B::SB - 1 - s) * B::LB>();
    if constexpr (s + B::NSB - 1 < B::SB) issue_b(s + B::NSB - 1);
    const char* wst = lds + B::OFF_R2 + (s % B::NSB) * B::W2B;
    static_for<0, B::TPS>([&](auto uu) {
      constexpr int u = decltype(uu)::value;
      constexpr int tap = (s / B::GB) * B::TPS + u;
      constexpr int r = tap / 3, sx = tap % 3;
#pragma unroll
      for (int sl = 0; sl < B::SPB; ++sl) {
        const char* m1 = lds + ((s % B::GB) * B::SPB + sl) * B::HPXP * 128;
        const char* wt = wst + (u * B::SPB + sl) * F * 128;
        bf16x8 a[2][4], b[2][B::TB];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const int c = ks * 4 + lq;
#pragma unroll
          for (int i = 0; i < 4; ++i)
            a[ks][i] = as_bf16x8(*(const uint4*)(wt + slot_off(cg * 64 + 16 * i + l16, c, lk)));
#pragma unroll
          for (int t = 0; t < B::TB; ++t)
            b[ks][t] = as_bf16x8(
                *(const uint4*)(m1 + slot_off(pbase[t] + r * HC + sx, c, obase[t] + r * TW + sx)));
        }
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int t = 0; t < B::TB; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              accB[t][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks][i], b[ks][t], accB[t][i], 0, 0, 0);
      }
    });
  });
  // every wave is done with M1 and the W2 ring: the W3 ring may overwrite them
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  static_for<0, B::NSC - 1>([&](auto k) { issue_c(decltype(k)::value); });
#pragma unroll
  for (int i = 0; i < 4; ++i) bias[i] = *(const float4*)(sb2 + cg * 64 + 16 * i + 4 * lq);
#pragma unroll
  for (int t = 0; t < B::TB; ++t) {
    const int jb = wp + WP * t;
    if (jb >= B::NTB) continue;
    const int o = 16 * jb + l16;
    char* m2 = lds + B::OFF_M2 + cg * B::OPXP * 128;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float4 bb = bias[i];
      const f32x4 v = accB[t][i];
      const float f0 = act_apply<2>((v[0] + bb.x) + 0.f, ac2), f1 = act_apply<2>((v[1] + bb.y) + 0.f, ac2);
      const float f2 = act_apply<2>((v[2] + bb.z) + 0.f, ac2), f3 = act_apply<2>((v[3] + bb.w) + 0.f, ac2);
      *(uint2*)(m2 + slot_off(o, 2 * i + (lane >> 5), o) + (lq & 1) * 8) =
          make_uint2(pack2_bf16(f0, f1), pack2_bf16(f2, f3));
    }
  }

  // ---- phase C: y = act3(M2 W3 + b3 + residual) -----------------------------
  // output offsets of this thread's pixels (kOOB: not stored) and their M2 rows
  uint32_t yoff[B::TB];
  int crow[B::TB];
#pragma unroll
  for (int t = 0; t < B::TB; ++t) {
    const int o = 16 * (wp + WP * t) + l16;
    const int oh = h0 + o / TW, ow = w0 + o % TW;
    const bool tile_ok = wp + WP * t < B::NTB;
    const bool ok = tile_ok && o < B::OPX && oh < P && ow < Q;
    yoff[t] = ok ? (uint32_t)((((n * P + oh) * Q + ow) * B::COUT + cg * 64 + 4 * lq) * 2) : kOOB;
    crow[t] = tile_ok ? o : l16;
  }
  const __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(p.y, (short)0, p.y_bytes, kBufferFlags);
  // Identity blocks defer a chunk's epilogue past the next chunk's MFMAs
  // (two accumulator sets), so its ALU work and stores overlap them.
  f32x4 acc[B::DEFER ? 2 : 1][B::TB][4], accp[B::TB][4];
  // the chunk's epilogue; every thread issues all ST stores (out-of-range
  // offsets for pixels it does not own), so the wait counts are exact
  auto finish = [&](auto qq) {
    constexpr int q = decltype(qq)::value;
    constexpr int set = B::DEFER ? q % 2 : 0;
    float4 bp[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      bias[i] = *(const float4*)(sb3 + q * F + cg * 64 + 16 * i + 4 * lq);
      if constexpr (B::PROJ) bp[i] = *(const float4*)(sbp + q * F + cg * 64 + 16 * i + 4 * lq);
    }
#pragma unroll
    for (int t = 0; t < B::TB; ++t) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float4 bb = bias[i];
        uint2 rv;
        if constexpr (B::PROJ) {  // the projection composite's output: bias, no activation, bf16
          const f32x4 u = accp[t][i];
          rv = make_uint2(pack2_bf16((u[0] + bp[i].x) + 0.f, (u[1] + bp[i].y) + 0.f),
                          pack2_bf16((u[2] + bp[i].z) + 0.f, (u[3] + bp[i].w) + 0.f));
        } else {
          rv = resv[q][t][i];
        }
        const f32x4 v = acc[set][t][i];
        const float r0 = __uint_as_float(rv.x << 16), r1 = __uint_as_float(rv.x & 0xFFFF0000u);
        const float r2 = __uint_as_float(rv.y << 16), r3 = __uint_as_float(rv.y & 0xFFFF0000u);
        const float f0 = act_apply<2>((v[0] + bb.x) + r0, ac3), f1 = act_apply<2>((v[1] + bb.y) + r1, ac3);
        const float f2 = act_apply<2>((v[2] + bb.z) + r2, ac3), f3 = act_apply<2>((v[3] + bb.w) + r3, ac3);
        const uint32_t off = yoff[t] == kOOB ? kOOB : yoff[t] + (uint32_t)((q * F + 16 * i) * 2);
        __builtin_amdgcn_raw_buffer_store_b64(u32x2{pack2_bf16(f0, f1), pack2_bf16(f2, f3)}, yr, (int)off, 0, 0);
      }
    }
  };
  static_for<0, B::SC>([&](auto kk) {
    constexpr int k = decltype(kk)::value;
    constexpr int q = k / B::UQ, j = k % B::UQ;
    constexpr int set = B::DEFER ? q % 2 : 0;
    stage_barrier<B::c_younger(k)>();
    if constexpr (k + B::NSC - 1 < B::SC) issue_c(k + B::NSC - 1);
    const char* wt = lds + (k % B::NSC) * B::CB;
    if constexpr (j == 0) {
#pragma unroll
      for (int t = 0; t < B::TB; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[set][t][i] = accp[t][i] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int sl = 0; sl < B::CSL; ++sl) {
      constexpr bool w3 = j * B::CSL < B::WGC;  // W3: slice j * CSL + sl of M2; else Wp: slice j - WGC of x
      bf16x8 a[2][4], b[2][B::TB];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int c = ks * 4 + lq;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          a[ks][i] = as_bf16x8(*(const uint4*)(wt + sl * F * 128 + slot_off(cg * 64 + 16 * i + l16, c, lk)));
        if constexpr (w3) {
          const char* m2 = lds + B::OFF_M2 + (j * B::CSL + sl) * B::OPXP * 128;
#pragma unroll
          for (int t = 0; t < B::TB; ++t) b[ks][t] = as_bf16x8(*(const uint4*)(m2 + slot_off(crow[t], c, lk)));
        } else {
#pragma unroll
          for (int t = 0; t < B::TB; ++t) b[ks][t] = as_bf16x8(xf[t][2 * (j - B::WGC) + ks]);
        }
      }
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int t = 0; t < B::TB; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if constexpr (w3)
              acc[set][t][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks][i], b[ks][t], acc[set][t][i], 0, 0, 0);
            else
              accp[t][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks][i], b[ks][t], accp[t][i], 0, 0, 0);
          }
    }
    if constexpr (B::DEFER) {
      if constexpr (j == 0 && q >= 1) finish(std::integral_constant<int, q - 1>{});
    } else if constexpr (j == B::UQ - 1) {
      finish(std::integral_constant<int, q>{});
    }
  });
  if constexpr (B::DEFER) finish(std::integral_constant<int, B::NQ - 1>{});
}

template <class B>
hipError_t launch_one(const BottleneckParams& p_in, hipStream_t s) {
  BottleneckParams p = p_in;
  p.tiles_w = (p.Q + B::TW - 1) / B::TW;
  p.tiles_hw = p.tiles_w * ((p.P + B::TH - 1) / B::TH);
  p.mg_tw = magic40(p.tiles_w);
  p.mg_thw = magic40(p.tiles_hw);
  p.tiles = p.N * p.tiles_hw;
  p.per_xcd = (p.tiles + 7) / 8;
  bottleneck_kernel<B><<<8 * p.per_xcd, B::NT, 0, s>>>(p);
  return hipGetLastError();
}

// Kinds (F, CIN, COUT, stride) and their variants: <F, CIN, COUT, S, TH, TW,
// waves, phase A ring, phase B taps x slices per stage, phase B ring>
using V64a = Bn<64, 256, 256, 1, 8, 28, 7, 2, 1, 1, 6>;    // 134 KB LDS
using V64b = Bn<64, 256, 256, 1, 8, 14, 7, 2, 1, 1, 5>;    // 80 KB: two workgroups per CU
using V64c = Bn<64, 256, 256, 1, 8, 14, 7, 4, 1, 1, 8>;    // 136 KB, deeper rings
using V128a = Bn<128, 512, 512, 1, 4, 28, 8, 2, 1, 1, 4>;  // 145 KB
using V128b = Bn<128, 512, 512, 1, 7, 14, 8, 3, 1, 1, 4>;  // 143 KB
using V128c = Bn<128, 512, 512, 1, 7, 14, 8, 2, 1, 1, 5>;  // 149 KB
using P64a = Bn<64, 64, 256, 1, 8, 28, 7, 1, 1, 1, 6>;     // projection, 64 input channels
using P64b = Bn<64, 64, 256, 1, 8, 14, 7, 1, 1, 1, 2>;     //   (57 KB: two workgroups per CU)
using P64c = Bn<64, 64, 256, 1, 8, 14, 7, 1, 1, 1, 5>;
using D128a = Bn<128, 256, 512, 2, 7, 14, 8, 2, 1, 1, 5>;  // projection, stride 2
using D128b = Bn<128, 256, 512, 2, 4, 28, 8, 2, 1, 1, 4>;
using D128c = Bn<128, 256, 512, 2, 7, 14, 8, 2, 1, 1, 3>;

// f(Bn{}) on variant v of a kind, or `none` for an unknown one
template <class R, class Fn>
R with_variant(int F, int CIN, int COUT, int S, int v, R none, Fn&& f) {
  if (v < 0 || v > 2) return none;
  if (S == 1 && F == 64 && CIN == 256 && COUT == 256) return v == 0 ? f(V64a{}) : v == 1 ? f(V64b{}) : f(V64c{});
  if (S == 1 && F == 128 && CIN == 512 && COUT == 512)
    return v == 0 ? f(V128a{}) : v == 1 ? f(V128b{}) : f(V128c{});
  if (S == 1 && F == 64 && CIN == 64 && COUT == 256) return v == 0 ? f(P64a{}) : v == 1 ? f(P64b{}) : f(P64c{});
  if (S == 2 && F == 128 && CIN == 256 && COUT == 512)
    return v == 0 ? f(D128a{}) : v == 1 ? f(D128b{}) : f(D128c{});
  return none;
}

template <class B>
const char* variant_name() {
  static char buf[64];
  static const int once =
      std::snprintf(buf, sizeof(buf), "bottleneck_f%d_%s%dx%d_w%d_a%d_b%d", B::F,
                    !B::PROJ ? "" : B::S == 1 ? "proj_" : "proj_s2_", B::TH, B::TW, B::NW, B::NSA, B::NSB);
  (void)once;
  return buf;
}

}  // namespace

int bottleneck_variants(int F, int CIN, int COUT, int S) {
  return with_variant(F, CIN, COUT, S, 0, 0, [](auto) { return 3; });
}

const char* bottleneck_variant_name(int F, int CIN, int COUT, int S, int v) {
  return with_variant(F, CIN, COUT, S, v, (const char*)"bottleneck_unsupported",
                      [](auto cfg) { return variant_name<decltype(cfg)>(); });
}

int bottleneck_tiles(int F, int CIN, int COUT, int S, int v, int N, int P, int Q) {
  return with_variant(F, CIN, COUT, S, v, 0, [&](auto cfg) {
    using B = decltype(cfg);
    return N * ((P + B::TH - 1) / B::TH) * ((Q + B::TW - 1) / B::TW);
  });
}

hipError_t launch_bottleneck(const BottleneckParams& p, int F, int CIN, int COUT, int S, int v, hipStream_t s) {
  return with_variant(F, CIN, COUT, S, v, hipErrorInvalidValue,
                      [&](auto cfg) { return launch_one<decltype(cfg)>(p, s); });
}

}  // namespace byoc
