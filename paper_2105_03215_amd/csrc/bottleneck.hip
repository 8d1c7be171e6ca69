// Fused ResNet bottleneck block: 1x1 reduce, 3x3, 1x1 expand with the
// block input (or a 1x1 projection of it) added back, as one kernel, on
// bf16 activations (fp32 sums) or on the int8 codes of a partially
// quantized function (int32 sums, Sec. 3.2).
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
// 128-byte slice of x at a time through a ring of LDS stages (x slice and
// W1 slice per stage, HBM -> LDS loads).  The sums are finished into M1 in
// LDS; positions outside the image are stored as the 3x3's padding: zeros,
// or for codes M1's zero point, so that the padded taps contribute exactly
// what the unfused int8 conv's border correction adds back.  While each x
// slice is staged, the threads copy the tile's own pixels of it into
// registers: the residual of phase C (identity shortcut), or the MFMA
// operand fragments of the projection (projection shortcut).
//
// Phase B (3x3): nine shifted views of M1 times W2, streamed through a ring
// of stages of TPS taps x SPB slices (tap by tap, then slice); the output
// tile is finished into M2 in LDS.
//
// Phase C (1x1 expand): M2 times W3, F output channels per chunk, the
// weights streamed one slice (of M2, then of x for the projection) per
// stage; with the projection shortcut the chunk's projection is summed from
// the registers of phase A and finished as the projection composite stores
// it; then the residual is added and y stored.
//
// Finishing a sum: bf16 - bias, activation, bf16 rounding; int8 - the
// folded bias, the float32 rescaling (one rounding per term), the output
// zero point, the residual's own rescaling, the activation clamp in code
// space: the arithmetic of the unfused int8 conv.
//
// Operands of every product: weights are the MFMA A operand (16 output
// channels), pixels the B operand, so each lane ends with 4 consecutive
// channels of one pixel.  A wave owns one 64-channel group of the output
// channels of each product and a set of 16-pixel tiles.  Every LDS row is
// 128 bytes (a "slice": 64 bf16 or 128 int8 channels of a pixel; an int8
// tensor of 64 channels uses half of it) with its 16-byte chunks permuted by
// a per-row key so that the 16 rows one MFMA operand read touches spread
// over the banks.  Both MFMAs (16x16x32 bf16, 16x16x64 int8) take 16 bytes
// per lane per operand, so one step consumes 64 bytes of a slice.
//
// Reduction order of each output: phase A and the projection slice by slice of x (64
// bytes per MFMA step), phase B tap by tap then channel, phase C channel -
// the order of the single-group implicit-GEMM kernel on the same composites
// (int32 sums are exact in any order).
#include <cstdio>
#include <type_traits>

#include "lds_dma.h"

namespace byoc {
namespace {

using namespace dma;

typedef __attribute__((ext_vector_type(2))) unsigned int u32x2;

constexpr int cmin(int a, int b) { return a < b ? a : b; }
constexpr int cmax(int a, int b) { return a > b ? a : b; }

// one MFMA step on 16-byte operand fragments
__device__ __forceinline__ f32x4 mma(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}
__device__ __forceinline__ i32x4 mma(uint4 a, uint4 b, i32x4 c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, a), __builtin_bit_cast(i32x4, b), c, 0,
                                               0, 0);
}

// Codes.  The int8 conv finishes an output as clamp(z + c(rint(fl32(a * m)))
// [+ c(rint(fl32((r - zr) * mr)))], lo, hi) with c() a clamp to +-2^20 and
// int32 sums.  Here the rounded terms stay float32 - integer-valued, so
// their sums are exact below 2^24 - and only the final clamp is applied:
// the same code whenever the residual term is below 2^19 in magnitude (the
// planner bounds its factor), since a term beyond 2^20 then puts the sum
// past the same end of [lo, hi] either way.  Codes are formed biased by
// +128 (v_cvt_pk_u8_f32 into byte e), the bias removed by one XOR per 4.
__device__ __forceinline__ float qterm(int a, int factor_bits) {
  return __builtin_rintf((float)a * __int_as_float(factor_bits));
}
__device__ __forceinline__ uint32_t pack_biased(float v, int e, uint32_t w) {
  return __builtin_amdgcn_cvt_pk_u8_f32(v, e, w);
}

template <int F_, int CIN_, int COUT_, int S_, int TH_, int TW_, int NW_, int NSA_, int TPS_, int SPB_, int NSB_,
          bool I8_ = false>
struct Bn {
  static constexpr int F = F_, CIN = CIN_, COUT = COUT_, S = S_, TH = TH_, TW = TW_, NW = NW_;
  static constexpr int NSA = NSA_, TPS = TPS_, SPB = SPB_, NSB = NSB_;  // rings and stages
  static constexpr bool I8 = I8_;                       // int8 codes, int32 sums
  static constexpr bool PROJ = COUT != CIN || S != 1;  // projection shortcut
  static constexpr int ES = I8 ? 1 : 2;                 // bytes per element
  static constexpr int XPB = CIN * ES, MPB = F * ES;    // bytes per pixel of x and of M1 / M2
  static constexpr int VX = cmin(128, XPB), VM = cmin(128, MPB);  // bytes of a slice in use
  static constexpr int KSA = VX / 64, KSM = VM / 64;  // MFMA steps per slice
  static constexpr int SA = (XPB + 127) / 128;        // x slices (phase A stages)
  static constexpr int MS = (MPB + 127) / 128;        // slices of M1 and M2
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
  static constexpr int PFA = NSA >= 2 ? NSA - 1 : 1;      // phase A stages issued ahead
  static constexpr int NQ = COUT / F;                     // phase C chunks (F output channels each)
  static constexpr int CSL = PROJ ? 1 : MS;               // slices per phase C stage
  static constexpr int UQ = (MS + (PROJ ? SA : 0)) / CSL;  // phase C stages per chunk: W3, then Wp slices
  static constexpr int SC = NQ * UQ;                      // phase C stages
  static constexpr int GB = MS / SPB;                     // slice groups of a tap
  static constexpr int SB = 9 / TPS * GB;                 // phase B stages
  static constexpr int XF = PROJ ? KSA * SA : 1;          // projection fragments per pixel tile
  static constexpr int MREG = 128 / (64 * ES);            // 64-channel groups per slice
  static constexpr int ROW = 128;
  // LDS plan (bytes)
  static constexpr int M1B = MS * HPXP * ROW;
  static constexpr int XB = HPXP * ROW;
  static constexpr int W1B = F * ROW;
  static constexpr int ASTG = XB + W1B;
  static constexpr int W2B = TPS * SPB * F * ROW;
  static constexpr int M2B = MS * OPXP * ROW;
  static constexpr int CB = CSL * F * ROW;  // phase C stage: F rows of a chunk x CSL slices
  static constexpr int OFF_R2 = M1B;        // the phase A ring, then the W2 ring and M2
  static constexpr int OFF_M2 = OFF_R2 + NSB * W2B;
  static constexpr int END_A = OFF_R2 + NSA * ASTG;
  static constexpr int END_B = OFF_M2 + M2B;
  static constexpr int NSC = cmin(OFF_M2 / CB, SC);  // phase C ring, over M1 and the W2 ring
  static constexpr int OFF_BIAS = cmax(END_A, END_B);
  // epilogue constants per channel: a float32 bias; for codes the folded
  // int32 bias and the float32 rescaling factor
  static constexpr int QB = I8 ? 8 : 4;
  static constexpr int B3BLK = (COUT * QB + 1023) / 1024;
  static constexpr int BBLK = 2 + (PROJ ? 2 : 1) * B3BLK;  // 1 KB blocks: b1, b2, b3 (, bp)
  static constexpr int LBB = (BBLK + NW - 1) / NW;         // bias fills per thread
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

  static_assert((XPB == 64 || XPB % 128 == 0) && (MPB == 64 || MPB % 128 == 0), "slices");
  static_assert(F % 64 == 0 && COUT % F == 0 && NW % WGC == 0 && F * QB <= 1024, "shape");
  static_assert(PROJ || CIN % F == 0, "identity shortcut: chunks of F channels");
  static_assert(9 % TPS == 0 && ((NSA >= 2 && NSA <= SA) || (NSA == 1 && SA == 1)), "phase A stages");
  static_assert(NSB >= 2 && NSB <= SB, "phase B stages");
  static_assert(MS % SPB == 0 && (TPS == 1 || SPB == MS), "phase B stages run tap by tap, then slice");
  static_assert(NSC >= 2, "phase C ring");
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
  constexpr int F = B::F, TW = B::TW, HC = B::HC, NW = B::NW, WP = B::WP, ES = B::ES;
  using Acc = std::conditional_t<B::I8, i32x4, f32x4>;
  using RT = std::conditional_t<B::I8, uint32_t, uint2>;  // 4 channels of the identity residual
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
  // epilogue constants, 256 words per 1 KB block: b1, b2, b3, bp (bf16:
  // the float bias of channel c at word c; codes: {bias, factor} at words
  // 2c, 2c + 1)
  const float* sb1 = reinterpret_cast<const float*>(lds + B::OFF_BIAS);
  const float* sb2 = sb1 + 256;
  const float* sb3 = sb1 + 512;
  const float* sbp = sb3 + 256 * B::B3BLK;  // projection bias
  const int* sq1 = reinterpret_cast<const int*>(sb1);
  const int* sq2 = reinterpret_cast<const int*>(sb2);
  const int* sq3 = reinterpret_cast<const int*>(sb3);
  const int* sqp = reinterpret_cast<const int*>(sbp);
  // codes: the folded int32 biases of channels ch .. ch + 3, the starting
  // value of their sums (int32 addition is exact in any order)
  auto bias_codes = [](const int* sq, int ch) {
    const int4 lo = *(const int4*)(sq + 2 * ch), hi = *(const int4*)(sq + 2 * ch + 4);
    return i32x4{lo.x, lo.z, hi.x, hi.z};
  };

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
    const int xc = lk ^ (px & 7);  // the logical chunk of slot lk
    uint32_t off = kOOB;
    if (blk < B::XBLK && px < B::HPX && xc * 16 < B::VX) {
      const int hr = px / HC, hc = px - (px / HC) * HC;
      const int mh = h0 - 1 + hr, mw = w0 - 1 + hc;  // position on the output grid
      if ((unsigned)mh < (unsigned)P && (unsigned)mw < (unsigned)Q)
        off = (uint32_t)(((n * H + B::S * mh) * W + B::S * mw) * B::XPB + xc * 16);
    }
    xoff[u] = off;
  }
  // rows 8 * blk + lane / 8 of a weight block (row stride ldb bytes, from
  // byte colb of a row, vb bytes in use), chunk lk at slot lk ^ (row & 7)
  auto row_off = [&](int blk, int nblk, int ldb, int colb, int vb) {
    const int row = 8 * blk + (lane >> 3);
    const int c = lk ^ (row & 7);
    return blk < nblk && c * 16 < vb ? (uint32_t)(row * ldb + colb + c * 16) : kOOB;
  };
#pragma unroll
  for (int u = 0; u < B::LW1; ++u) w1off[u] = row_off(wave + NW * u, B::W1BLK, p.ld1 * ES, 0, B::VX);
#pragma unroll
  for (int u = 0; u < B::LB; ++u) {
    const int blk = wave + NW * u;  // [tap u][slice sl][F rows]
    const int tap = blk / (B::SPB * F / 8), rem = blk - tap * (B::SPB * F / 8);
    const int sl = rem / (F / 8);
    w2off[u] = blk < B::W2BLK ? row_off(rem - sl * (F / 8), F / 8, p.ld2 * ES, tap * B::MPB + sl * 128, B::VM)
                              : kOOB;
  }
#pragma unroll
  for (int u = 0; u < B::LC; ++u) {  // [slice sl][F rows of a chunk] of W3 (of Wp: one slice)
    const int blk = wave + NW * u;
    const int sl = blk / (F / 8);
    w3off[u] = blk < B::CBLK ? row_off(blk - sl * (F / 8), F / 8, p.ld3 * ES, sl * 128, B::VM) : kOOB;
    wpoff[u] = B::PROJ ? row_off(blk, B::CBLK, p.ldp * ES, 0, B::VX) : kOOB;
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
                 live(w2off[u], (s / B::GB) * B::TPS * B::MPB + (s % B::GB) * B::SPB * 128));
  };
  auto issue_c = [&](int k) {  // chunk k / UQ: stage j = k % UQ, W3 slices j * CSL .. (j < MS / CSL), else Wp
    const uint32_t slot = base + (k % B::NSC) * B::CB;
    const int q = k / B::UQ, j = k % B::UQ;
    if (j * B::CSL < B::MS) {
#pragma unroll
      for (int u = 0; u < B::LC; ++u)
        lds_fill16(w3r, dst(slot, wave + NW * u, B::CBLK), live(w3off[u], q * F * p.ld3 * ES + j * B::CSL * 128));
    } else {
#pragma unroll
      for (int u = 0; u < B::LC; ++u)
        lds_fill16(wpr, dst(slot, wave + NW * u, B::CBLK), live(wpoff[u], q * F * p.ldp * ES + (j - B::MS) * 128));
    }
  };

  // epilogue constants: block blk < BBLK (b1, b2, the blocks of b3, then
  // those of bp) is filled by wave blk % NW
#pragma unroll
  for (int u = 0; u < B::LBB; ++u) {
    const int blk = wave + NW * u;
    const bool pb = blk >= 2 + B::B3BLK;
    const void* src = blk == 0 ? p.b1 : blk == 1 ? p.b2 : pb ? p.bp : p.b3;
    const int bytes = blk == 0 ? p.b1_bytes : blk == 1 ? p.b2_bytes : pb ? p.bp_bytes : p.b3_bytes;
    const int sub = blk < 2 ? 0 : pb ? blk - 2 - B::B3BLK : blk - 2;
    const uint32_t off = blk < B::BBLK ? (uint32_t)(sub * 1024 + lane * 16) : kOOB;
    lds_fill16(buffer_rsrc(src, bytes), dst(base + B::OFF_BIAS, blk, B::BBLK), off);
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
  Acc accA[B::TA][4];
#pragma unroll
  for (int t = 0; t < B::TA; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) accA[t][i] = Acc{0, 0, 0, 0};
  // identity shortcut: the residual of phase C per chunk, 4 channels of one
  // pixel per (chunk, pixel tile, channel tile)
  RT resv[B::PROJ ? 1 : B::NQ][B::TB][4];
  uint4 xf[B::TB][B::XF];  // projection: x at the tile's pixels as MFMA B fragments, per 64-byte step

  static_for<0, B::PFA>([&](auto s) {
    if constexpr (decltype(s)::value < B::SA) issue_a(decltype(s)::value);
  });
  static_for<0, B::SA>([&](auto ss) {
    constexpr int s = decltype(ss)::value;
    stage_barrier<cmin(B::PFA - 1, B::SA - 1 - s) * B::LA>();
    if constexpr (B::NSA >= 2 && s + B::PFA < B::SA) issue_a(s + B::PFA);
    if constexpr (B::I8 && s == 0) {  // (the epilogue constants are in, with the first stage)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const Acc b = __builtin_bit_cast(Acc, bias_codes(sq1, cg * 64 + 16 * i + 4 * lq));
#pragma unroll
        for (int t = 0; t < B::TA; ++t) accA[t][i] = b;
      }
    }
    const char* xs = lds + B::OFF_R2 + (s % B::NSA) * B::ASTG;
    const char* ws = xs + B::XB;
    if constexpr (B::PROJ) {
#pragma unroll
      for (int t = 0; t < B::TB; ++t)
#pragma unroll
        for (int ks = 0; ks < B::KSA; ++ks)
          xf[t][B::KSA * s + ks] = *(const uint4*)(xs + slot_off(hrow[t], ks * 4 + lq, hrow[t]));
    } else if constexpr (!B::I8) {
      if (cg == s % B::WGC) {  // this slice is the residual of the wave's channel group in chunk s / WGC
#pragma unroll
        for (int t = 0; t < B::TB; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            resv[B::PROJ ? 0 : s / B::WGC][t][i] =
                *(const uint2*)(xs + slot_off(hrow[t], 2 * i + (lane >> 5), hrow[t]) + (lq & 1) * 8);
      }
    } else {
      // codes: the wave's 64 channels of chunk q are bytes q * F + cg * 64 .. + 63 of a pixel
      static_for<0, B::PROJ ? 0 : B::NQ>([&](auto qq) {
        constexpr int q = decltype(qq)::value;
        const int b0 = q * F + cg * 64;
        if ((b0 >> 7) == s) {
#pragma unroll
          for (int t = 0; t < B::TB; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              resv[q][t][i] =
                  *(const uint32_t*)(xs + slot_off(hrow[t], ((b0 & 127) >> 4) + i, hrow[t]) + 4 * lq);
        }
      });
    }
#pragma unroll
    for (int ks = 0; ks < B::KSA; ++ks) {
      const int c = ks * 4 + lq;
      uint4 a[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = *(const uint4*)(ws + slot_off(cg * 64 + 16 * i + l16, c, lk));
#pragma unroll
      for (int t = 0; t < B::TA; ++t) {
        const int j = wp + WP * t;
        if (j < B::NTA) {
          const uint4 b = *(const uint4*)(xs + slot_off(16 * j + l16, c, lk));
#pragma unroll
          for (int i = 0; i < 4; ++i) accA[t][i] = mma(a[i], b, accA[t][i]);
        }
      }
    }
  });
  // every wave is done with the phase A ring: the next ring may overwrite it
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  static_for<0, B::NSB - 1>([&](auto s) { issue_b(decltype(s)::value); });
  // Where a lane's 4 channels of channel tile i of an F-wide intermediate
  // go in its pixel's row: bytes (cg * 64 + 16 i + 4 lq) * ES of the pixel,
  // in slice cg / MREG.
  auto mid_slot = [&](int px, int i, int key) -> uint32_t {
    if constexpr (B::I8) return slot_off(px, (cg & 1) * 4 + i, key) + 4 * lq;
    else return slot_off(px, 2 * i + (lane >> 5), key) + (lq & 1) * 8;
  };
  // epilogue constants into registers before the first M1 store (a later LDS
  // read could not move above a store the compiler cannot tell apart from it)
  float4 bias[4];
  int4 qlo[4], qhi[4];  // codes: {bias, factor} of channels 4 lq, 4 lq + 1 and 4 lq + 2, 4 lq + 3 of tile i
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ch = cg * 64 + 16 * i + 4 * lq;
    if constexpr (B::I8) {
      qlo[i] = *(const int4*)(sq1 + 2 * ch);
      qhi[i] = *(const int4*)(sq1 + 2 * ch + 4);
    } else {
      bias[i] = *(const float4*)(sb1 + ch);
    }
  }
#pragma unroll
  for (int t = 0; t < B::TA; ++t) {
    const int j = wp + WP * t;
    if (j >= B::NTA) continue;
    const int px = 16 * j + l16;
    const int hr = px / HC, hc = px - (px / HC) * HC;
    const int mh = h0 - 1 + hr, mw = w0 - 1 + hc;
    const bool inside = px < B::HPX && (unsigned)mh < (unsigned)P && (unsigned)mw < (unsigned)Q;
    const int key = hr * TW + hc;
    char* m1 = lds + (cg / B::MREG) * B::HPXP * 128;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const Acc v = accA[t][i];
      if constexpr (B::I8) {
        const float zb = (float)(p.qz[0] + 128), lob = (float)(p.qlo[0] + 128), hib = (float)(p.qhi[0] + 128);
        uint32_t w = 0;
        w = pack_biased(__builtin_amdgcn_fmed3f(zb + qterm(v[0], qlo[i].y), lob, hib), 0, w);
        w = pack_biased(__builtin_amdgcn_fmed3f(zb + qterm(v[1], qlo[i].w), lob, hib), 1, w);
        w = pack_biased(__builtin_amdgcn_fmed3f(zb + qterm(v[2], qhi[i].y), lob, hib), 2, w);
        w = pack_biased(__builtin_amdgcn_fmed3f(zb + qterm(v[3], qhi[i].w), lob, hib), 3, w);
        w ^= 0x80808080u;
        if (!inside) w = ((uint32_t)p.qz[0] & 0xFFu) * 0x01010101u;  // the 3x3's padding: the zero point
        *(uint32_t*)(m1 + mid_slot(px, i, key)) = w;
      } else {
        const float4 bb = bias[i];
        // (+ 0: the unfused epilogue adds its zero residual, which turns a -0 into +0)
        float f0 = act_apply<2>((v[0] + bb.x) + 0.f, ac1), f1 = act_apply<2>((v[1] + bb.y) + 0.f, ac1);
        float f2 = act_apply<2>((v[2] + bb.z) + 0.f, ac1), f3 = act_apply<2>((v[3] + bb.w) + 0.f, ac1);
        if (!inside) f0 = f1 = f2 = f3 = 0.f;
        *(uint2*)(m1 + mid_slot(px, i, key)) = make_uint2(pack2_bf16(f0, f1), pack2_bf16(f2, f3));
      }
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
  Acc accB[B::TB][4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    Acc b = Acc{0, 0, 0, 0};
    if constexpr (B::I8) b = __builtin_bit_cast(Acc, bias_codes(sq2, cg * 64 + 16 * i + 4 * lq));
#pragma unroll
    for (int t = 0; t < B::TB; ++t) accB[t][i] = b;
  }
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
        uint4 a[B::KSM][4], b[B::KSM][B::TB];
#pragma unroll
        for (int ks = 0; ks < B::KSM; ++ks) {
          const int c = ks * 4 + lq;
#pragma unroll
          for (int i = 0; i < 4; ++i) a[ks][i] = *(const uint4*)(wt + slot_off(cg * 64 + 16 * i + l16, c, lk));
#pragma unroll
          for (int t = 0; t < B::TB; ++t)
            b[ks][t] = *(const uint4*)(m1 + slot_off(pbase[t] + r * HC + sx, c, obase[t] + r * TW + sx));
        }
#pragma unroll
        for (int ks = 0; ks < B::KSM; ++ks)
#pragma unroll
          for (int t = 0; t < B::TB; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) accB[t][i] = mma(a[ks][i], b[ks][t], accB[t][i]);
      }
    });
  });
  // every wave is done with M1 and the W2 ring: the W3 ring may overwrite them
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  static_for<0, B::NSC - 1>([&](auto k) { issue_c(decltype(k)::value); });
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ch = cg * 64 + 16 * i + 4 * lq;
    if constexpr (B::I8) {
      qlo[i] = *(const int4*)(sq2 + 2 * ch);
      qhi[i] = *(const int4*)(sq2 + 2 * ch + 4);
    } else {
      bias[i] = *(const float4*)(sb2 + ch);
    }
  }
#pragma unroll
  for (int t = 0; t < B::TB; ++t) {
    const int jb = wp + WP * t;
    if (jb >= B::NTB) continue;
    const int o = 16 * jb + l16;
    char* m2 = lds + B::OFF_M2 + (cg / B::MREG) * B::OPXP * 128;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const Acc v = accB[t][i];
      if constexpr (B::I8) {
        const float zb = (float)(p.qz[1] + 128), lob = (float)(p.qlo[1] + 128), hib = (float)(p.qhi[1] + 128);
        uint32_t w = 0;
        w = pack_biased(__builtin_amdgcn_fmed3f(zb + qterm(v[0], qlo[i].y), lob, hib), 0, w);
        w = pack_biased(__builtin_amdgcn_fmed3f(zb + qterm(v[1], qlo[i].w), lob, hib), 1, w);
        w = pack_biased(__builtin_amdgcn_fmed3f(zb + qterm(v[2], qhi[i].y), lob, hib), 2, w);
        w = pack_biased(__builtin_amdgcn_fmed3f(zb + qterm(v[3], qhi[i].w), lob, hib), 3, w);
        *(uint32_t*)(m2 + mid_slot(o, i, o)) = w ^ 0x80808080u;
      } else {
        const float4 bb = bias[i];
        const float f0 = act_apply<2>((v[0] + bb.x) + 0.f, ac2), f1 = act_apply<2>((v[1] + bb.y) + 0.f, ac2);
        const float f2 = act_apply<2>((v[2] + bb.z) + 0.f, ac2), f3 = act_apply<2>((v[3] + bb.w) + 0.f, ac2);
        *(uint2*)(m2 + mid_slot(o, i, o)) = make_uint2(pack2_bf16(f0, f1), pack2_bf16(f2, f3));
      }
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
    yoff[t] = ok ? (uint32_t)((((n * P + oh) * Q + ow) * B::COUT + cg * 64 + 4 * lq) * ES) : kOOB;
    crow[t] = tile_ok ? o : l16;
  }
  const __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(p.y, (short)0, p.y_bytes, kBufferFlags);
  // Identity blocks defer a chunk's epilogue past the next chunk's MFMAs
  // (two accumulator sets), so its ALU work and stores overlap them.
  Acc acc[B::DEFER ? 2 : 1][B::TB][4], accp[B::TB][4];
  // the chunk's epilogue; every thread issues all ST stores (out-of-range
  // offsets for pixels it does not own), so the wait counts are exact
  auto finish = [&](auto qq) {
    constexpr int q = decltype(qq)::value;
    constexpr int set = B::DEFER ? q % 2 : 0;
    if constexpr (B::I8) {
      const float zb = (float)(p.qz[2] + 128), lob = (float)(p.qlo[2] + 128), hib = (float)(p.qhi[2] + 128);
      const float zrb = (float)(p.zr + 128), mr = p.mr;
      const float zpb = (float)(p.qz[3] + 128), plob = (float)(p.qlo[3] + 128), phib = (float)(p.qhi[3] + 128);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int ch = q * F + cg * 64 + 16 * i + 4 * lq;
        const int4 ql = *(const int4*)(sq3 + 2 * ch), qh = *(const int4*)(sq3 + 2 * ch + 4);
        const int fs[4] = {ql.y, ql.w, qh.y, qh.w};
        int fp[4] = {0, 0, 0, 0};
        if constexpr (B::PROJ) {
          const int4 pl = *(const int4*)(sqp + 2 * ch), ph = *(const int4*)(sqp + 2 * ch + 4);
          fp[0] = pl.y, fp[1] = pl.w, fp[2] = ph.y, fp[3] = ph.w;
        }
#pragma unroll
        for (int t = 0; t < B::TB; ++t) {
          const Acc v = acc[set][t][i];
          uint32_t rb = 0;
          if constexpr (!B::PROJ) rb = resv[q][t][i] ^ 0x80808080u;  // residual codes + 128
          uint32_t w = 0;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float d;  // residual code minus its zero point (exact)
            if constexpr (B::PROJ)  // the projection composite's output code (no activation), biased
              d = __builtin_amdgcn_fmed3f(zpb + qterm(accp[t][i][e], fp[e]), plob, phib) - zpb;
            else
              d = (float)((rb >> (8 * e)) & 0xFFu) - zrb;
            w = pack_biased(__builtin_amdgcn_fmed3f((zb + qterm(v[e], fs[e])) + __builtin_rintf(d * mr), lob, hib), e, w);
          }
          const uint32_t off = yoff[t] == kOOB ? kOOB : yoff[t] + (uint32_t)(q * F + 16 * i);
          __builtin_amdgcn_raw_buffer_store_b32(w ^ 0x80808080u, yr, (int)off, 0, 0);
        }
      }
    } else {
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
      for (int i = 0; i < 4; ++i) {
        Acc b = Acc{0, 0, 0, 0}, bp = Acc{0, 0, 0, 0};
        if constexpr (B::I8) {
          b = __builtin_bit_cast(Acc, bias_codes(sq3, q * F + cg * 64 + 16 * i + 4 * lq));
          if constexpr (B::PROJ) bp = __builtin_bit_cast(Acc, bias_codes(sqp, q * F + cg * 64 + 16 * i + 4 * lq));
        }
#pragma unroll
        for (int t = 0; t < B::TB; ++t) {
          acc[set][t][i] = b;
          accp[t][i] = bp;
        }
      }
    }
#pragma unroll
    for (int sl = 0; sl < B::CSL; ++sl) {
      constexpr bool w3 = j * B::CSL < B::MS;  // W3: slice j * CSL + sl of M2; else Wp: slice j - MS of x
      constexpr int KS = w3 ? B::KSM : B::KSA;
      uint4 a[KS][4], b[KS][B::TB];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int c = ks * 4 + lq;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          a[ks][i] = *(const uint4*)(wt + sl * F * 128 + slot_off(cg * 64 + 16 * i + l16, c, lk));
        if constexpr (w3) {
          const char* m2 = lds + B::OFF_M2 + (j * B::CSL + sl) * B::OPXP * 128;
#pragma unroll
          for (int t = 0; t < B::TB; ++t) b[ks][t] = *(const uint4*)(m2 + slot_off(crow[t], c, lk));
        } else {
#pragma unroll
          for (int t = 0; t < B::TB; ++t) b[ks][t] = xf[t][B::KSA * (j - B::MS) + ks];
        }
      }
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int t = 0; t < B::TB; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if constexpr (w3)
              acc[set][t][i] = mma(a[ks][i], b[ks][t], acc[set][t][i]);
            else
              accp[t][i] = mma(a[ks][i], b[ks][t], accp[t][i]);
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
// small tiles for small batches (4 x 7 output pixels, 4 waves): at batch 1
// the block's grids are a few dozen workgroups, so a workgroup's own
// latency sets the time
using V64d = Bn<64, 256, 256, 1, 4, 7, 4, 2, 1, 1, 4>;
using V128d = Bn<128, 512, 512, 1, 4, 7, 4, 2, 1, 1, 4>;
using P64d = Bn<64, 64, 256, 1, 4, 7, 4, 1, 1, 1, 4>;
using D128d = Bn<128, 256, 512, 2, 4, 7, 4, 2, 1, 1, 4>;
// int8 codes: the 64 mid channels of a pixel fill half a slice (one MFMA
// step per tap), so three taps fit a phase B stage
using Q64a = Bn<64, 256, 256, 1, 8, 28, 7, 2, 1, 1, 6, true>;
using Q64b = Bn<64, 256, 256, 1, 7, 14, 7, 2, 1, 1, 5, true>;  // 77 KB: two workgroups per CU
using Q64c = Bn<64, 256, 256, 1, 8, 14, 7, 2, 3, 1, 3, true>;
using Q128a = Bn<128, 512, 512, 1, 4, 28, 8, 2, 1, 1, 4, true>;
using Q128b = Bn<128, 512, 512, 1, 7, 14, 8, 3, 1, 1, 4, true>;
using Q128c = Bn<128, 512, 512, 1, 7, 14, 8, 2, 1, 1, 6, true>;
using R64a = Bn<64, 64, 256, 1, 8, 28, 7, 1, 1, 1, 6, true>;  // projection, 64 input channels
using R64b = Bn<64, 64, 256, 1, 8, 14, 7, 1, 1, 1, 2, true>;
using R64c = Bn<64, 64, 256, 1, 8, 14, 7, 1, 3, 1, 3, true>;
using E128a = Bn<128, 256, 512, 2, 7, 14, 8, 2, 1, 1, 5, true>;  // projection, stride 2
using E128b = Bn<128, 256, 512, 2, 4, 28, 8, 2, 1, 1, 4, true>;
using E128c = Bn<128, 256, 512, 2, 7, 14, 8, 2, 1, 1, 6, true>;

// f(Bn{}) on variant v of a kind, or `none` for an unknown one
// (bf16 kinds: 4 variants, the last the small-batch tile; int8: 3)
template <class R, class Fn>
R with_variant(bool i8, int F, int CIN, int COUT, int S, int v, R none, Fn&& f) {
  if (v < 0 || v > (i8 ? 2 : 3)) return none;
  if (S == 1 && F == 64 && CIN == 256 && COUT == 256) {
    if (i8) return v == 0 ? f(Q64a{}) : v == 1 ? f(Q64b{}) : f(Q64c{});
    return v == 0 ? f(V64a{}) : v == 1 ? f(V64b{}) : v == 2 ? f(V64c{}) : f(V64d{});
  }
  if (S == 1 && F == 128 && CIN == 512 && COUT == 512) {
    if (i8) return v == 0 ? f(Q128a{}) : v == 1 ? f(Q128b{}) : f(Q128c{});
    return v == 0 ? f(V128a{}) : v == 1 ? f(V128b{}) : v == 2 ? f(V128c{}) : f(V128d{});
  }
  if (S == 1 && F == 64 && CIN == 64 && COUT == 256) {
    if (i8) return v == 0 ? f(R64a{}) : v == 1 ? f(R64b{}) : f(R64c{});
    return v == 0 ? f(P64a{}) : v == 1 ? f(P64b{}) : v == 2 ? f(P64c{}) : f(P64d{});
  }
  if (S == 2 && F == 128 && CIN == 256 && COUT == 512) {
    if (i8) return v == 0 ? f(E128a{}) : v == 1 ? f(E128b{}) : f(E128c{});
    return v == 0 ? f(D128a{}) : v == 1 ? f(D128b{}) : v == 2 ? f(D128c{}) : f(D128d{});
  }
  return none;
}

template <class B>
const char* variant_name() {
  static char buf[64];
  static const int once = std::snprintf(buf, sizeof(buf), "bottleneck_%sf%d_%s%dx%d_w%d_a%d_b%d%s",
                                        B::I8 ? "i8_" : "", B::F, !B::PROJ ? "" : B::S == 1 ? "proj_" : "proj_s2_",
                                        B::TH, B::TW, B::NW, B::NSA, B::NSB, B::TPS == 3 ? "x3" : "");
  (void)once;
  return buf;
}

}  // namespace

int bottleneck_variants(bool i8, int F, int CIN, int COUT, int S) {
  return with_variant(i8, F, CIN, COUT, S, 0, 0, [i8](auto) { return i8 ? 3 : 4; });
}

const char* bottleneck_variant_name(bool i8, int F, int CIN, int COUT, int S, int v) {
  return with_variant(i8, F, CIN, COUT, S, v, (const char*)"bottleneck_unsupported",
                      [](auto cfg) { return variant_name<decltype(cfg)>(); });
}

int bottleneck_tiles(bool i8, int F, int CIN, int COUT, int S, int v, int N, int P, int Q) {
  return with_variant(i8, F, CIN, COUT, S, v, 0, [&](auto cfg) {
    using B = decltype(cfg);
    return N * ((P + B::TH - 1) / B::TH) * ((Q + B::TW - 1) / B::TW);
  });
}

hipError_t launch_bottleneck(const BottleneckParams& p, bool i8, int F, int CIN, int COUT, int S, int v,
                             hipStream_t s) {
  return with_variant(i8, F, CIN, COUT, S, v, hipErrorInvalidValue,
                      [&](auto cfg) { return launch_one<decltype(cfg)>(p, s); });
}

}  // namespace byoc
