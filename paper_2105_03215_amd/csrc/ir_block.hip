// Fused MobileNetV2 inverted-residual block: 1x1 expand (+bias, ReLU6),
// depthwise 3x3 (stride S, pad 1, +bias, ReLU6), 1x1 project (+bias) and,
// when the block keeps its shape, the block input added back - one kernel.
//
// The three composites of a block are planned as separate launches
// elsewhere; the expanded tensor (6x the block's width) and the depthwise
// output then make a round trip through HBM each, and the depthwise pass is
// a launch of its own.  Here a workgroup owns a TH x TW tile of output
// pixels; the tile's input window - (TH - 1) S + 3 by (TW - 1) S + 3 input
// pixels, the depthwise halo - is staged in LDS once, and the expanded width
// F is walked in slices of 64 channels:
//   phase A: the slice of the expanded tensor over the whole window (MFMA,
//            the expand weights' 64 rows times the window's pixels), finished
//            (bias, activation, bf16) into LDS; window positions outside the
//            image hold 0, the depthwise padding;
//   phase B: the depthwise taps of the slice (vector ALU, 8 channels of a
//            strip of output pixels per thread, the fused multiply-adds from
//            the bias in tap order (row, column) - the unfused depthwise
//            kernel's arithmetic), finished into LDS;
//   phase C: the project product accumulates the slice's 64-channel step of
//            its reduction (MFMA) in registers.
// After the last slice the project sums are finished (bias, the block input
// read from the staged window, bf16) and stored.  The intermediates never
// leave the workgroup (the engine owns an offloaded subgraph's
// intermediates, Sec. 3.4): of the separate launches' HBM traffic, one read
// of x (plus the halo) and one write of y remain.  A block without expand
// (expansion 1) runs phases B and C on the staged window itself.
//
// Reduction orders are those of the single-group implicit-GEMM kernel:
// phase A over the input channels in 32-channel MFMA steps, phase C over the
// expanded channels slice by slice - so the fused block equals the unfused
// launches bit for bit.
//
// Weights are the MFMA A operand (16 output channels), pixels the B operand.
// Every LDS row is 128 bytes (64 bf16 channels) with its 16-byte chunks
// permuted by the row index (slot = chunk ^ (row & 7)).  The weights of the
// next slice stream in while the current one computes: the expand and
// depthwise weights after phase A, the project weights after phase C, each
// into its own buffer (the depthwise slice double-buffered); every thread
// issues the same loads (out-of-range ones fill a junk block), so the wait
// counts are compile-time constants.
#include <cstdio>

#include "lds_dma.h"

namespace byoc {
namespace {

using namespace dma;

typedef __attribute__((ext_vector_type(2))) unsigned int u32x2;

template <int CT_, int S_, int TH_, int TW_, bool EXP_, int V_, int MINW_, int XS_ = 1, int FMAX_ = 512>
struct Ir {
  static constexpr int CT = CT_, S = S_, TH = TH_, TW = TW_;  // CT: 16-channel tiles of the output
  static constexpr bool EXP = EXP_;                           // expand conv present
  static constexpr int XS = XS_;      // 64-channel slices of the block input (the window's rows per pixel)
  static constexpr int FMAX = FMAX_;  // the largest expanded width (bias tables)
  static constexpr int NW = 8, NT = 64 * NW;
  static constexpr int IH = (TH - 1) * S + 3, IW = (TW - 1) * S + 3;  // input window
  static constexpr int HPX = IH * IW, HPXP = (HPX + 15) / 16 * 16;
  static constexpr int OPX = TH * TW, OPXP = (OPX + 15) / 16 * 16;
  static constexpr int NTA = HPXP / 16, NTB = OPXP / 16;  // 16-pixel tiles
  static constexpr int TA = (NTA + NW - 1) / NW;          // phase A pixel tiles per wave
  static constexpr int V = V_;                            // phase B: output rows per thread
  static constexpr int NSTRIP = TH / V * TW;              //   strips of V rows of one column
  // phase B: channels per thread (8, 4 or 2), so that the strips x channel
  // groups cover the workgroup's threads
  static constexpr int CPT = NSTRIP * 8 >= NT ? 8 : NSTRIP * 16 >= NT ? 4 : 2;
  static constexpr int NG = 64 / CPT;  // channel groups of a slice
  static constexpr int NPC = CT * NTB;                    // phase C (channel tile, pixel tile) pairs
  static constexpr int TC = (NPC + NW - 1) / NW;          // pairs per wave
  static constexpr int ROW = 128;
  // LDS plan (bytes)
  // the window: slice j of pixel px in row j * HPXP + px
  static constexpr int OFF_X = 0, XB = XS * HPXP * ROW;
  static constexpr int OFF_E = OFF_X + XB, EB = EXP ? HPXP * ROW : 0;
  static constexpr int OFF_D = OFF_E + EB, DB = OPXP * ROW;
  // expand weights of a slice of F: input slice j of row r in row j * 64 + r
  static constexpr int OFF_WE = OFF_D + DB, WEB = EXP ? XS * 64 * ROW : 0;
  // depthwise slice: 9 taps x 64 float32 channels, tap t in rows 2t, 2t + 1 (x 2 buffers)
  static constexpr int OFF_WD = OFF_WE + WEB, WDB = 3 * 1024;
  static constexpr int OFF_WP = OFF_WD + 2 * WDB, WPB = CT * 16 * ROW;
  // 1 KB blocks of float32 biases: [be (FB),] bd (FB), bp (PB)
  static constexpr int FB = FMAX * 4 / 1024, PB = (CT * 16 * 4 + 1023) / 1024;
  static constexpr int BBLK = (EXP ? FB : 0) + FB + PB, LBB = (BBLK + NW - 1) / NW;
  static constexpr int OFF_B = OFF_WP + WPB;
  static constexpr int OFF_JUNK = OFF_B + BBLK * 1024;
  static constexpr int MINW = MINW_;  // waves per SIMD the registers are held to
  static constexpr int LDS = OFF_JUNK + 1024;
  // 1 KB fills (8 rows of 128 bytes) per thread
  static constexpr int XBLK = XS * HPXP / 8, LX = (XBLK + NW - 1) / NW;
  static constexpr int LWE = EXP ? XS : 0;  // 8 blocks per input slice: one per wave
  static constexpr int LWD = 1;            // 3 blocks
  static constexpr int WPBLK = CT * 2, LWP = (WPBLK + NW - 1) / NW;
  static_assert(CT * 16 <= 320 && FMAX % 256 == 0 && LDS <= kLdsLimit && TH % V == 0 && (V == 1 || S == 1),
                "shape");
  static_assert(LWE + LWD <= 63 && LWP <= 63, "vmcnt immediate");
};

__device__ __forceinline__ uint32_t slot_off(int row, int chunk) {
  return (uint32_t)(row * 128 + ((chunk ^ (row & 7)) << 4));
}

// N (8, 4 or 2) consecutive bf16 values from LDS as floats, and back
template <int N>
__device__ __forceinline__ void load_bf16(const char* p, float* f) {
  if constexpr (N == 8) {
    unpack8(*(const uint4*)p, f);
  } else {
    uint32_t w[N / 2];
    if constexpr (N == 4) {
      const uint2 u = *(const uint2*)p;
      w[0] = u.x, w[1] = u.y;
    } else {
      w[0] = *(const uint32_t*)p;
    }
#pragma unroll
    for (int i = 0; i < N / 2; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
}
template <int N>
__device__ __forceinline__ void store_bf16(char* p, const float* f) {
  if constexpr (N == 8) {
    *(uint4*)p = pack8(f);
  } else if constexpr (N == 4) {
    *(uint2*)p = make_uint2(pack2_bf16(f[0], f[1]), pack2_bf16(f[2], f[3]));
  } else {
    *(uint32_t*)p = pack2_bf16(f[0], f[1]);
  }
}
template <int N>
__device__ __forceinline__ void load_f32(const float* p, float* f) {
  if constexpr (N == 2) {
    const float2 a = *(const float2*)p;
    f[0] = a.x, f[1] = a.y;
  } else {
#pragma unroll
    for (int i = 0; i < N / 4; ++i) {
      const float4 a = *(const float4*)(p + 4 * i);
      f[4 * i] = a.x, f[4 * i + 1] = a.y, f[4 * i + 2] = a.z, f[4 * i + 3] = a.w;
    }
  }
}

template <int YOUNGER>
__device__ __forceinline__ void wait_barrier() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(YOUNGER) : "memory");
}

template <class B>
__global__ __launch_bounds__(B::NT, B::MINW) void ir_block_kernel(IrParams p) {
  constexpr int NW = B::NW, IW = B::IW, TW = B::TW, S = B::S;
  __shared__ __attribute__((aligned(1024))) char lds[B::LDS];
  asm volatile("" ::"s"(p.x), "s"(p.y), "s"(p.we), "s"(p.be), "s"(p.wd), "s"(p.bd), "s"(p.wp), "s"(p.bp));
  asm volatile("" ::"s"(p.N), "s"(p.H), "s"(p.W), "s"(p.P), "s"(p.Q), "s"(p.CIN), "s"(p.F), "s"(p.COUT),
               "s"(p.ldE), "s"(p.ldP), "s"(p.x_bytes), "s"(p.y_bytes), "s"(p.tiles_w), "s"(p.tiles_hw),
               "s"(p.mg_tw), "s"(p.mg_thw), "s"(p.tiles), "s"(p.per_xcd));

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int l16 = lane & 15, lk = lane & 7, lq = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // the tile; XCD x takes the contiguous run [x * per_xcd, (x + 1) * per_xcd)
  // of the tile order, so neighbouring tiles share an L2
  const int tile = (blockIdx.x & 7) * p.per_xcd + (blockIdx.x >> 3);
  if (tile >= p.tiles) return;
  const int n = mdiv(tile, p.mg_thw);
  const int tr = tile - n * p.tiles_hw;
  const int th = mdiv(tr, p.mg_tw);
  const int h0 = th * B::TH, w0 = (tr - th * p.tiles_w) * TW;  // output grid
  const int ih0 = h0 * S - 1, iw0 = w0 * S - 1;                // window origin (input grid)
  const int H = p.H, W = p.W, CIN = p.CIN, F = p.F, COUT = p.COUT;
  const int FS = (F + 63) / 64;  // slices of the expanded width

  const uint32_t base = lds_addr(lds);
  const uint32_t junk = base + B::OFF_JUNK;
  const float* sbe = reinterpret_cast<const float*>(lds + B::OFF_B);
  const float* sbd = sbe + (B::EXP ? B::FMAX : 0);
  const float* sbp = sbd + B::FMAX;

  // ---- load plans ----------------------------------------------------------
  const i32x4 xr = buffer_rsrc(p.x, p.x_bytes);
  const i32x4 wer = buffer_rsrc(p.we, B::EXP ? p.we_bytes : 0);
  const i32x4 wdr = buffer_rsrc(p.wd, p.wd_bytes);
  const i32x4 wpr = buffer_rsrc(p.wp, p.wp_bytes);
  auto dst = [&](uint32_t region, int blk, int nblk) {
    return __builtin_amdgcn_readfirstlane(blk < nblk ? region + blk * 1024 : junk);
  };
  // the window: slice j of position px (px / IW, px % IW) in row
  // j * HPXP + px, logical chunk lk ^ (px & 7)
  uint32_t xoff[B::LX];
#pragma unroll
  for (int u = 0; u < B::LX; ++u) {
    const int blk = wave + NW * u;
    const int j = blk / (B::HPXP / 8);
    const int px = 8 * (blk - j * (B::HPXP / 8)) + (lane >> 3);
    const int xc = lk ^ (px & 7);
    const int ch = j * 64 + xc * 8;
    uint32_t off = kOOB;
    if (blk < B::XBLK && px < B::HPX && ch < CIN) {
      const int ih = ih0 + px / IW, iw = iw0 + px % IW;
      if ((unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)W)
        off = (uint32_t)((((n * H + ih) * W + iw) * CIN + ch) * 2);
    }
    xoff[u] = off;
  }
  // weight rows 8 * blk + lane / 8, logical chunk lk ^ (row & 7)
  const int wrow = 8 * wave + (lane >> 3);
  const int wch = lk ^ (wrow & 7);
  auto issue_we = [&](int f) {  // expand rows f*64 + wrow, input slice j's 64 channels
    if constexpr (B::EXP) {
#pragma unroll
      for (int j = 0; j < B::XS; ++j) {
        const uint32_t off = f < FS ? (uint32_t)(((f * 64 + wrow) * p.ldE + j * 64 + wch * 8) * 2) : kOOB;
        lds_fill16(wer, dst(base + B::OFF_WE + j * 64 * B::ROW, wave, 8), off);
      }
    }
  };
  auto issue_wd = [&](int f) {  // row r: tap r / 2, channels f*64 + 32 (r % 2) + 4 lk (no permutation)
    const int row = 8 * wave + (lane >> 3);
    const int tap = row >> 1, ch = f * 64 + (row & 1) * 32 + lk * 4;
    const bool ok = f < FS && wave < 3 && tap < 9 && ch < F;
    const uint32_t off = ok ? (uint32_t)((tap * F + ch) * 4) : kOOB;
    lds_fill16(wdr, dst(base + B::OFF_WD + (f & 1) * B::WDB, wave, 3), off);
  };
  auto issue_wp = [&](int f) {  // project rows (output channels), reduction slice f
#pragma unroll
    for (int u = 0; u < B::LWP; ++u) {
      const int blk = wave + NW * u;
      const int row = 8 * blk + (lane >> 3);
      const int c = lk ^ (row & 7);
      const uint32_t off = f < FS && blk < B::WPBLK ? (uint32_t)((row * p.ldP + f * 64 + c * 8) * 2) : kOOB;
      lds_fill16(wpr, dst(base + B::OFF_WP, blk, B::WPBLK), off);
    }
  };

  // ---- prologue: the window, the biases, the first slice's weights ----------
#pragma unroll
  for (int u = 0; u < B::LX; ++u) lds_fill16(xr, dst(base + B::OFF_X, wave + NW * u, B::XBLK), xoff[u]);
#pragma unroll
  for (int u = 0; u < B::LBB; ++u) {
    // blocks [FB of be,] then FB of bd, PB of bp (fp32, zero past their ends)
    const int blk = wave + NW * u;
    const int k = blk - (B::EXP ? B::FB : 0);  // index past the be blocks
    const void* src = k < 0 ? p.be : k < B::FB ? p.bd : p.bp;
    const int bytes = k < 0 ? p.be_bytes : k < B::FB ? p.bd_bytes : p.bp_bytes;
    const int sub = k < 0 ? blk : k < B::FB ? k : k - B::FB;
    const uint32_t off = blk < B::BBLK ? (uint32_t)(sub * 1024 + lane * 16) : kOOB;
    lds_fill16(buffer_rsrc(src, bytes), dst(base + B::OFF_B, blk, B::BBLK), off);
  }
  issue_we(0);
  issue_wd(0);
  issue_wp(0);
  wait_barrier<0>();

  const ActClamp ace = act_clamp_of(p.act_e, p.alpha_e);
  const ActClamp acd = act_clamp_of(p.act_d, p.alpha_d);
  const ActClamp acp = act_clamp_of(p.act_p, p.alpha_p);
  const int ka = (CIN + 31) / 32;  // phase A MFMA steps

  f32x4 accC[B::TC];
#pragma unroll
  for (int u = 0; u < B::TC; ++u) accC[u] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int f = 0; f < FS; ++f) {
    // ---- phase A: the slice of the expanded tensor over the window -----------
    if constexpr (B::EXP) {
      f32x4 accA[B::TA][4];
#pragma unroll
      for (int t = 0; t < B::TA; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) accA[t][i] = f32x4{0.f, 0.f, 0.f, 0.f};
      const char* we = lds + B::OFF_WE;
      const char* xs = lds + B::OFF_X;
      for (int ks = 0; ks < ka; ++ks) {
        const int sl = ks >> 1, c = (ks & 1) * 4 + lq;  // input slice, chunk in it
        const char* wes = we + sl * 64 * B::ROW;
        const char* xss = xs + sl * B::HPXP * B::ROW;
        uint4 a[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) a[i] = *(const uint4*)(wes + slot_off(16 * i + l16, c));
#pragma unroll
        for (int t = 0; t < B::TA; ++t) {
          const int j = wave + NW * t;
          if (j < B::NTA) {
            const bf16x8 b = as_bf16x8(*(const uint4*)(xss + slot_off(16 * j + l16, c)));
#pragma unroll
            for (int i = 0; i < 4; ++i)
              accA[t][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a[i]), b, accA[t][i], 0, 0, 0);
          }
        }
      }
      char* es = lds + B::OFF_E;
#pragma unroll
      for (int t = 0; t < B::TA; ++t) {
        const int j = wave + NW * t;
        if (j >= B::NTA) continue;
        const int px = 16 * j + l16;
        const int ih = ih0 + px / IW, iw = iw0 + px % IW;
        const bool inside = px < B::HPX && (unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)W;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float4 bb = *(const float4*)(sbe + f * 64 + 16 * i + 4 * lq);
          const f32x4 v = accA[t][i];
          // (+ 0: the unfused epilogue adds its zero residual, which turns a -0 into +0)
          float f0 = act_apply<2>((v[0] + bb.x) + 0.f, ace), f1 = act_apply<2>((v[1] + bb.y) + 0.f, ace);
          float f2 = act_apply<2>((v[2] + bb.z) + 0.f, ace), f3 = act_apply<2>((v[3] + bb.w) + 0.f, ace);
          if (!inside) f0 = f1 = f2 = f3 = 0.f;  // the depthwise padding
          *(uint2*)(es + slot_off(px, 2 * i + (lq >> 1)) + (lq & 1) * 8) =
              make_uint2(pack2_bf16(f0, f1), pack2_bf16(f2, f3));
        }
      }
      // the slice is in LDS, the expand weights are free
      asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    }
    issue_we(f + 1);
    issue_wd(f + 1);

    // ---- phase B: depthwise taps of the slice --------------------------------
    // A thread keeps CPT channels (a fixed group: NT is a multiple of the
    // group count) - their taps are float32 in LDS - and finishes a vertical
    // strip of V output pixels of one column: each input value of the
    // strip's window is unpacked once and feeds every output whose window
    // holds it, in each output's tap order (row, column) from its bias.
    {
      constexpr int CPT = B::CPT, NG = B::NG, V = B::V;
      const char* es = B::EXP ? lds + B::OFF_E : lds + B::OFF_X;
      const char* wd = lds + B::OFF_WD + (f & 1) * B::WDB;
      char* ds = lds + B::OFF_D;
      const int g = tid % NG;
      const int cb = g * CPT;                      // first channel of the group in the slice
      const int chunk = cb >> 3, inner = (cb & 7) * 2;  // its 16-byte chunk, byte offset in it
      const float* wg = reinterpret_cast<const float*>(wd) + cb;  // tap t: wg[64 t .. 64 t + CPT - 1]
      float bias[CPT];
#pragma unroll
      for (int e = 0; e < CPT; ++e) bias[e] = sbd[f * 64 + cb + e];
      for (int item = tid; item < B::NSTRIP * NG; item += B::NT) {
        const int st = item / NG;
        const int sr = st / TW, ow = st - (st / TW) * TW;
        const int oh0 = sr * V;
        float acc[V][CPT];
#pragma unroll
        for (int v = 0; v < V; ++v)
#pragma unroll
          for (int e = 0; e < CPT; ++e) acc[v][e] = bias[e];
#pragma unroll
        for (int rr = 0; rr < (V - 1) * S + 3; ++rr)
#pragma unroll
          for (int c = 0; c < 3; ++c) {
            const int row = (oh0 * S + rr) * IW + ow * S + c;
            float xf[CPT];
            load_bf16<CPT>(es + slot_off(row, chunk) + inner, xf);
#pragma unroll
            for (int v = 0; v < V; ++v) {
              const int r = rr - v * S;  // the tap row of output v
              if (r < 0 || r > 2) continue;
              float wv[CPT];
              load_f32<CPT>(wg + 64 * (r * 3 + c), wv);
#pragma unroll
              for (int e = 0; e < CPT; ++e) acc[v][e] = fmaf(xf[e], wv[e], acc[v][e]);
            }
          }
#pragma unroll
        for (int v = 0; v < V; ++v) {
#pragma unroll
          for (int e = 0; e < CPT; ++e) acc[v][e] = act_apply<2>(acc[v][e] + 0.f, acd);
          store_bf16<CPT>(ds + slot_off((oh0 + v) * TW + ow, chunk) + inner, acc[v]);
        }
      }
    }
    // the depthwise slice is in LDS; this slice's project weights have landed
    // (the next expand and depthwise weights, issued after them, may not)
    wait_barrier<B::LWE + B::LWD>();

    // ---- phase C: the slice's step of the project reduction -------------------
    {
      const char* wp = lds + B::OFF_WP;
      const char* ds = lds + B::OFF_D;
#pragma unroll
      for (int u = 0; u < B::TC; ++u) {
        const int pr = wave + NW * u;
        if (pr >= B::NPC) continue;
        const int ct = pr % B::CT, pt = pr / B::CT;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const int c = ks * 4 + lq;
          const bf16x8 a = as_bf16x8(*(const uint4*)(wp + slot_off(16 * ct + l16, c)));
          const bf16x8 b = as_bf16x8(*(const uint4*)(ds + slot_off(16 * pt + l16, c)));
          accC[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, accC[u], 0, 0, 0);
        }
      }
    }
    // every wave is done with the project weights and the depthwise slice
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    issue_wp(f + 1);
    // the next expand and depthwise weights have landed
    wait_barrier<B::LWP>();
  }

  // ---- epilogue: bias, the block input, bf16 --------------------------------
  const __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(p.y, (short)0, p.y_bytes, kBufferFlags);
  const char* xs = lds + B::OFF_X;
#pragma unroll
  for (int u = 0; u < B::TC; ++u) {
    const int pr = wave + NW * u;
    const int ct = pr % B::CT, pt = pr / B::CT;
    const int o = 16 * pt + l16;
    const int oh = o / TW, ow = o - (o / TW) * TW;
    const int ch = 16 * ct + 4 * lq;
    const bool ok = pr < B::NPC && o < B::OPX && h0 + oh < p.P && w0 + ow < p.Q && ch < COUT;
    const float4 bb = *(const float4*)(sbp + (ch < B::CT * 16 ? ch : 0));
    float r[4] = {0.f, 0.f, 0.f, 0.f};
    if (p.res && ok) {  // the block input at this output pixel (stride 1: window position (oh + 1, ow + 1))
      const int row = (ch >> 6) * B::HPXP + (oh + 1) * IW + ow + 1;
      const uint2 rv = *(const uint2*)(xs + slot_off(row, (ch & 63) >> 3) + (ch & 7) * 2);
      r[0] = __uint_as_float(rv.x << 16), r[1] = __uint_as_float(rv.x & 0xFFFF0000u);
      r[2] = __uint_as_float(rv.y << 16), r[3] = __uint_as_float(rv.y & 0xFFFF0000u);
    }
    const f32x4 v = accC[u];
    const float f0 = act_apply<2>((v[0] + bb.x) + r[0], acp), f1 = act_apply<2>((v[1] + bb.y) + r[1], acp);
    const float f2 = act_apply<2>((v[2] + bb.z) + r[2], acp), f3 = act_apply<2>((v[3] + bb.w) + r[3], acp);
    const uint32_t off = ok ? (uint32_t)((((n * p.P + h0 + oh) * p.Q + w0 + ow) * COUT + ch) * 2) : kOOB;
    __builtin_amdgcn_raw_buffer_store_b64(u32x2{pack2_bf16(f0, f1), pack2_bf16(f2, f3)}, yr, (int)off, 0, 0);
  }
}

template <class B>
hipError_t launch_one(const IrParams& p_in, hipStream_t s) {
  IrParams p = p_in;
  p.tiles_w = (p.Q + B::TW - 1) / B::TW;
  p.tiles_hw = p.tiles_w * ((p.P + B::TH - 1) / B::TH);
  p.mg_tw = magic40(p.tiles_w);
  p.mg_thw = magic40(p.tiles_hw);
  p.tiles = p.N * p.tiles_hw;
  p.per_xcd = (p.tiles + 7) / 8;
  ir_block_kernel<B><<<8 * p.per_xcd, B::NT, 0, s>>>(p);
  return hipGetLastError();
}

// Kinds (output channel tiles, stride, expand) and their variants: <CT, S,
// tile height, tile width, expand, output rows per phase-B thread, waves per
// SIMD the registers are held to>.  Every variant sums each output in the
// same order, so all of a kind's variants give the same bits.
template <int CT, int S, bool EXP>
struct Variants;
template <>
struct Variants<1, 1, false> {  // expansion 1 (32 -> 16 at 112x112)
  using V0 = Ir<1, 1, 8, 16, false, 1, 6>;
  using V1 = Ir<1, 1, 8, 8, false, 1, 6>;
  using V2 = Ir<1, 1, 4, 16, false, 1, 6>;
};
template <int CT>
struct Variants<CT, 2, true> {  // stride 2
  using V0 = Ir<CT, 2, 8, 8, true, 1, 1>;
  using V1 = Ir<CT, 2, 4, 8, true, 1, 4>;
  using V2 = Ir<CT, 2, 4, 4, true, 1, 4>;
};
template <int CT>
struct Variants<CT, 1, true> {  // stride 1
  using V0 = Ir<CT, 1, 8, 8, true, 2, 4>;
  using V1 = Ir<CT, 1, 4, 8, true, 1, 6>;
  using V2 = Ir<CT, 1, 4, 4, true, 1, 6>;
};

// Wider blocks (input 96 or 160 channels: two or three slices of the
// window per pixel; expanded width up to 1024; output up to 320 channels).
template <int CT, int S, int XS>
struct VariantsX {
  using V0 = Ir<CT, 1, 8, 8, true, 2, 2, XS, 1024>;
  using V1 = Ir<CT, 1, 4, 8, true, 1, 2, XS, 1024>;
  using V2 = Ir<CT, 1, 4, 4, true, 1, 4, XS, 1024>;
};
template <int CT, int XS>
struct VariantsX<CT, 2, XS> {  // stride 2: the window is (2 TH + 1) x (2 TW + 1)
  using V0 = Ir<CT, 2, 4, 8, true, 1, 2, XS, 1024>;
  using V1 = Ir<CT, 2, 4, 4, true, 1, 4, XS, 1024>;
  using V2 = Ir<CT, 2, 2, 8, true, 1, 4, XS, 1024>;
};

template <class K, class R, class Fn>
R pick(int v, Fn&& fn) {
  return v == 0 ? fn(typename K::V0{}) : v == 1 ? fn(typename K::V1{}) : fn(typename K::V2{});
}

template <class R, class Fn>
R with_kind(int cin, int f, int cout, int s, int v, R none, Fn&& fn) {
  if (v < 0 || v > 2 || cin % 8 != 0 || f % 8 != 0 || cout % 8 != 0) return none;
  const int ct = (cout + 15) / 16;
  if (cin > 64) {  // MobileNetV2's later blocks
    if (f > 1024 || f == cin) return none;
    if (cin <= 128 && s == 1 && ct == 6) return pick<VariantsX<6, 1, 2>, R>(v, fn);
    if (cin <= 128 && s == 2 && ct == 10) return pick<VariantsX<10, 2, 2>, R>(v, fn);
    if (cin > 128 && cin <= 192 && s == 1 && ct == 10) return pick<VariantsX<10, 1, 3>, R>(v, fn);
    if (cin > 128 && cin <= 192 && s == 1 && ct == 20) return pick<VariantsX<20, 1, 3>, R>(v, fn);
    return none;
  }
  // the window is one slice of x, the expand reduction at most 64 channels
  if (f > 512) return none;
  if (f == cin) return ct == 1 && s == 1 ? pick<Variants<1, 1, false>, R>(v, fn) : none;
  if (s == 2) {
    if (ct == 2) return pick<Variants<2, 2, true>, R>(v, fn);
    if (ct == 4) return pick<Variants<4, 2, true>, R>(v, fn);
    return none;
  }
  if (s != 1) return none;
  if (ct == 2) return pick<Variants<2, 1, true>, R>(v, fn);
  if (ct == 4) return pick<Variants<4, 1, true>, R>(v, fn);
  if (ct == 6) return pick<Variants<6, 1, true>, R>(v, fn);
  return none;
}

template <class B>
const char* kind_name() {
  static char buf[64];
  static const int once = std::snprintf(buf, sizeof(buf), "ir_block_c%d_s%d_%dx%d_v%d_w%d%s%s", B::CT * 16, B::S,
                                        B::TH, B::TW, B::V, B::MINW, B::EXP ? "" : "_noexp",
                                        B::XS == 1 ? "" : B::XS == 2 ? "_x2" : "_x3");
  (void)once;
  return buf;
}

}  // namespace

int ir_block_variants(int cin, int f, int cout, int s) {
  return with_kind(cin, f, cout, s, 0, 0, [](auto) { return 3; });
}

const char* ir_block_name(int cin, int f, int cout, int s, int v) {
  return with_kind(cin, f, cout, s, v, (const char*)"ir_block_unsupported",
                   [](auto k) { return kind_name<decltype(k)>(); });
}

int ir_block_tiles(int cin, int f, int cout, int s, int v, int N, int P, int Q) {
  return with_kind(cin, f, cout, s, v, 0, [&](auto k) {
    using B = decltype(k);
    return N * ((P + B::TH - 1) / B::TH) * ((Q + B::TW - 1) / B::TW);
  });
}

hipError_t launch_ir_block(const IrParams& p, int v, hipStream_t s) {
  if (p.res && (p.CIN != p.COUT || p.S != 1)) return hipErrorInvalidValue;
  return with_kind(p.CIN, p.F, p.COUT, p.S, v, hipErrorInvalidValue,
                   [&](auto k) { return launch_one<decltype(k)>(p, s); });
}

}  // namespace byoc
