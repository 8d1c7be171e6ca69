// Implicit-GEMM convolution on CDNA4 bf16 MFMA with a direct HBM->LDS
// pipeline (buffer_load_dwordx4 ... lds).
//
// The conv composite y[n,p,q,k] = act(sum_{r,s,c} x[n, p*sh-pt+r, q*sw-pl+s, c]
// * w[k,r,s,c] + b[k] + res[n,p,q,k]) is a GEMM with M = N*P*Q output
// pixels, N = K output channels and a reduction of length R*S*C.  With NHWC
// activations and weights packed K-major with kk = (r*S+s)*Cp + c, a row of
// either operand is contiguous along the reduction: every lane moves 16 bytes
// (8 bf16, one MFMA operand register) per load.  Dense layers run through the
// same kernel as 1x1 convs on 1x1 images.
//
// Workgroup: 256 threads = 4 waves, tile BM pixels x BN channels, 64
// reduction elements per stage.  The operand tiles of NS stages live in NS
// LDS buffers; the loads of stage t+NS-1 are issued (straight into LDS, no
// registers) before the MFMAs of stage t, so NS-1 stages of loads are in
// flight while the matrix cores work.  Each buffer is its own __shared__
// array: the compiler then knows which pending LDS fills a read depends on
// and waits only for those; the wait before the one barrier per stage is
// explicit.  An out-of-range buffer offset fills zeros, which supplies the
// conv padding and the ragged pixel/reduction tails without branches.
//
// LDS rows are 128 bytes (8 chunks of 16 B).  A load instruction fills 8
// consecutive rows (lane l -> row l/8, slot l%8), so the swizzle that keeps
// MFMA operand reads conflict-free (logical chunk ch of row rw at slot
// ch ^ (rw & 7)) is applied on the fetch side: lane l fetches logical chunk
// (l%8) ^ (l/8).
//
// The weights are the MFMA A operand and the pixels the B operand, so each
// lane's 4 accumulators hold 4 consecutive output channels of one pixel.  The
// epilogue stages fp32 results through LDS in 32-channel passes so that each
// thread finishes 8 consecutive channels of one pixel (bias, residual,
// activation, bf16 rounding fused) with one 16-byte store.  With split-K each
// split writes fp32 partials and a second kernel reduces them in a fixed
// order.
#include <type_traits>

#include "lds_dma.h"

namespace byoc {
namespace {

using namespace dma;

constexpr int kBK = 64;        // reduction elements per stage
constexpr int kCH = kBK / 8;   // 16-byte chunks per tile row
constexpr int kMaxStages = 4;  // deepest operand ring (deeper rings measured no faster)

template <int BM, int BN, int WM, int WN, int KG, int NS, bool ALIGNED, bool SPLIT>
__global__ __launch_bounds__(64 * WM * WN * KG) void conv_dma_kernel(ConvParams p) {
  static_assert(WM * WN == 4 || WM * WN == 8, "4 or 8 waves per reduction group");
  static_assert(KG == 1 || ((KG == 2 || KG == 4) && !SPLIT), "reduction groups");
  constexpr int kNT = 64 * WM * WN;          // threads of one reduction group
  constexpr int kNTall = kNT * KG;           // threads per workgroup
  constexpr int kRowsPerPass = kNT / kCH;    // rows one load instruction of every wave covers
  static_assert(NS >= 1 && NS <= kMaxStages, "stages");
  constexpr int WTM = BM / WM, WTN = BN / WN;  // wave tile
  constexpr int TM = WTM / 16, TN = WTN / 16;  // 16x16 MFMA tiles per wave
  constexpr int AR = BM / kRowsPerPass, BR = BN / kRowsPerPass;
  static_assert(TM >= 1 && TN >= 1 && AR >= 1 && BR >= 1, "tile too small");
  constexpr int LPS = AR + BR;  // load instructions per thread per stage
  constexpr int STAGE = (BM + BN) * kCH;  // uint4 per stage buffer

  // KG reduction groups of WM x WN waves each run their own ring of NS
  // stage buffers over every KG-th stage of the reduction (group g: stages
  // g, g + KG, ...), which multiplies the loads in flight and the MFMA issue
  // of a workgroup; the groups' sums are added in group order at the end.
  __shared__ uint4 ring[KG * NS * STAGE];
  __shared__ float4 sbias[64];  // bias of the tile's channels (a whole wave's 16-byte fill)
  materialize_args(p);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int kg = __builtin_amdgcn_readfirstlane(tid / kNT);        // reduction group
  const int tg = tid - kg * kNT;                                      // thread within the group
  const int wave = __builtin_amdgcn_readfirstlane((tid >> 6) % (WM * WN));  // wave within the group
  uint4* const gring = ring + kg * NS * STAGE;
  auto buf = [&](auto tag) -> uint4* {
    constexpr int S = decltype(tag)::value;
    return gring + S * STAGE;
  };
  const int wm = wave / WN, wn = wave % WN;
  const int r0 = tg / kCH;                        // first row this thread fills
  const int cv = (lane & 7) ^ ((lane >> 3) & 7);  // logical chunk it fetches

  int tm, tn;
  if (!place_tile<BM, BN>(p, &tm, &tn)) return;
  const int m0 = tm * BM;
  const int n0 = tn * BN;

  const int nk_total = (p.Kg + kBK - 1) / kBK;
  int kt_begin = 0, kt_end = nk_total;
  if (SPLIT) {
    kt_begin = blockIdx.y * p.k_tiles_per_split;
    kt_end = min(nk_total, kt_begin + p.k_tiles_per_split);
  }

  // Activation rows of this thread.  Aligned path (Cp % 64 == 0, a stage is
  // 64 channels of one tap): pix = element offset of the row's window origin
  // plus this thread's chunk, tapmask bit r*S+s set when that tap lies inside
  // the image.  Non-aligned path: the window origin.
  int pix[AR], a_ih[AR], a_iw[AR];
  uint32_t tapmask[AR];
  const int PQ = p.P * p.Q;
#pragma unroll
  for (int i = 0; i < AR; ++i) {
    const int m = m0 + r0 + i * kRowsPerPass;
    int ih0 = -(1 << 28), iw0 = 0, n = 0;  // rows past M: never inside the image
    if (m < p.M) {
      n = mdiv(m, p.mg_pq);
      const int pq = m - n * PQ;
      const int pp = mdiv(pq, p.mg_q);
      const int qq = pq - pp * p.Q;
      ih0 = pp * p.sh - p.pt;
      iw0 = qq * p.sw - p.pl;
    }
    a_ih[i] = ih0;
    a_iw[i] = iw0;
    pix[i] = m < p.M ? ((n * p.H + ih0) * p.W + iw0) * p.Cp : 0;
    if (ALIGNED) {
      pix[i] += cv * 8;
      // taps inside the image: kernel rows [r_lo, r_hi) x columns [s_lo, s_hi)
      const int r_lo = max(0, -ih0), nr = max(0, min(p.R, p.H - ih0) - r_lo);
      const int s_lo = max(0, -iw0), s_hi = min(p.S, p.W - iw0);
      const uint32_t cols =
          s_hi > s_lo ? (uint32_t)(((1ull << s_hi) - 1ull) & ~((1ull << s_lo) - 1ull)) : 0u;
      uint32_t mask = 0;
      for (int r = 0; r < p.R; ++r)
        if ((unsigned)(r - r_lo) < (unsigned)nr) mask |= cols << (r * p.S);
      tapmask[i] = mask;
    }
  }
  const i32x4 xr = buffer_rsrc(p.x, p.x_bytes);
  const i32x4 wr = buffer_rsrc(p.w, p.w_bytes);
  uint32_t wvoff[BR];  // byte offset of this thread's weight rows and chunk
#pragma unroll
  for (int i = 0; i < BR; ++i) wvoff[i] = (uint32_t)(((n0 + r0 + i * kRowsPerPass) * p.Kgp + cv * 8) * 2);

  // Reduction position of the next stage to load: tap (r, s), channel c,
  // flattened index kk (non-aligned path: this thread's own chunk) and the
  // packed-weight column.
  int r, s, c, kk, wcol;
  {
    const int kk0 = (kt_begin + kg) * kBK + (ALIGNED ? 0 : cv * 8);
    const int rs = mdiv(kk0, p.mg_cp);
    c = kk0 - rs * p.Cp;
    r = mdiv(rs, p.mg_s);
    s = rs - r * p.S;
    kk = kk0;
    wcol = (kt_begin + kg) * kBK;
  }

  // Issues the loads of the next stage into buffer SET and advances the
  // position.  Every step issues the same number of loads, also past the end
  // of this split's reduction (those read zeros from an out-of-range offset
  // and are never computed), which keeps the count of loads in flight fixed.
  int kleft = (kt_end - kt_begin - kg + KG - 1) / KG;  // stages of this group
  auto issue = [&](auto set_tag) {
    uint4* dst = buf(set_tag);
    const bool live = kleft-- > 0;
    const int tap = (r * p.W + s) * p.Cp + c;
    const int bit = (r * p.S + s) & 31;
    const bool kval = live && (ALIGNED || kk < p.Kg);
#pragma unroll
    for (int i = 0; i < AR; ++i) {
      bool ok;
      if (ALIGNED) {
        ok = live && ((tapmask[i] >> bit) & 1u);
      } else {
        const int ih = a_ih[i] + r;
        const int iw = a_iw[i] + s;
        ok = kval && (unsigned)ih < (unsigned)p.H && (unsigned)iw < (unsigned)p.W;
      }
      const uint32_t off = ok ? (uint32_t)(pix[i] + tap) * 2u : kOOB;
      lds_fill16(xr, __builtin_amdgcn_readfirstlane(lds_addr(dst + (i * kRowsPerPass + wave * 8) * kCH)), off);
    }
    const uint32_t wc = (uint32_t)wcol * 2u;
#pragma unroll
    for (int i = 0; i < BR; ++i)
      lds_fill16(wr, __builtin_amdgcn_readfirstlane(lds_addr(dst + (BM + i * kRowsPerPass + wave * 8) * kCH)),
                 live ? wvoff[i] + wc : kOOB);
#pragma unroll
    for (int a = 0; a < KG; ++a) {  // to this group's next stage
      wcol += kBK;
      c += kBK;
      if (ALIGNED) {
        if (c == p.Cp) {
          c = 0;
          if (++s == p.S) {
            s = 0;
            ++r;
          }
        }
      } else {
        kk += kBK;
        while (c >= p.Cp) {
          c -= p.Cp;
          if (++s == p.S) {
            s = 0;
            ++r;
          }
        }
      }
    }
  };

  f32x4 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // One stage from LDS: 2 k-steps of the 16x16x32 MFMA.  Lane l reads 16
  // bytes (8 consecutive reduction elements) of row l % 16 at chunk
  // (k-step, l / 16).
  auto compute = [&](auto set_tag) {
    const uint4* sA = buf(set_tag);
    const uint4* sB = sA + BM * kCH;
#pragma unroll
    for (int ks = 0; ks < kBK / 32; ++ks) {
      const int chunk = ks * 4 + (lane >> 4);
      bf16x8 af[TN], bfr[TM];
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int row = wn * WTN + i * 16 + (lane & 15);
        af[i] = as_bf16x8(sB[row * kCH + (chunk ^ (row & 7))]);
      }
#pragma unroll
      for (int j = 0; j < TM; ++j) {
        const int row = wm * WTM + j * 16 + (lane & 15);
        bfr[j] = as_bf16x8(sA[row * kCH + (chunk ^ (row & 7))]);
      }
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
  };

  // Epilogue operands (bias and residual of the 8 channels this thread
  // finishes per pass) are fetched before the main loop so that their
  // latency overlaps the reduction.
  constexpr int kEC = 32;  // channels per epilogue pass
  constexpr int NPASS = BN / kEC;
  constexpr int TPP = kEC / 8;  // threads per pixel
  constexpr int EPV = (BM * TPP + kNTall - 1) / kNTall;  // pixels per thread per pass
  const int ec8 = (tid % TPP) * 8;
  uint4 resv[SPLIT ? 1 : NPASS][EPV];
  if (!SPLIT) {
    const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16_t*>(p.res), (short)0, p.res ? p.res_bytes : 0, kBufferFlags);
#pragma unroll
    for (int pass = 0; pass < NPASS; ++pass) {
      const int k = n0 + pass * kEC + ec8;
#pragma unroll
      for (int q = 0; q < EPV; ++q) {
        const int px = (tid + q * kNTall) / TPP;
        const int m = m0 + px;
        const uint32_t off =
            (px < BM && m < p.M && k < p.Kp) ? (uint32_t)(m * p.ldr + k) * 2u : kOOB;
        resv[pass][q] = p.res ? __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rr, off, 0, 0))
                              : make_uint4(0u, 0u, 0u, 0u);
      }
    }
  }

  const int nkt = (kt_end - kt_begin + KG - 1) / KG;  // steps (stages per group, rounded up)

  // Stage t lives in buffer t % NS.  Before computing it: wait for this
  // thread's fills of stage t (the NS-2 younger stages may stay in flight)
  // and for its own LDS reads, then barrier so every wave's fills are
  // visible and every wave is done with stage t-1, whose buffer the fills
  // of stage t+NS-1 then reuse.
  static_assert((NS - 2) * LPS <= 63, "vmcnt immediate");
  auto step = [&](auto cur, auto nxt) {
    if constexpr (NS == 1) {  // single buffer: load, compute, then refill it
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
      compute(cur);
      asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
      issue(nxt);
    } else {
      asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"((NS - 2) * LPS) : "memory");
      issue(nxt);
      compute(cur);
    }
  };
  // step i of a round of NS computes buffer i and refills buffer (i + NS - 1) % NS
  auto round_step = [&](auto i) {
    constexpr int I = decltype(i)::value;
    step(i, std::integral_constant<int, (I + NS - 1) % NS>{});
  };

  // the tile's bias, straight into LDS (zeros without a bias); issued first,
  // so every later wait of this wave covers it
  if (!SPLIT && tid < 64) {
    const i32x4 br = buffer_rsrc(p.bias, p.bias ? ((p.Kp + 255) / 256) * 256 * 4 : 0);
    const uint32_t off = lane < BN / 4 ? (uint32_t)(n0 + 4 * lane) * 4u : kOOB;
    lds_fill16(br, __builtin_amdgcn_readfirstlane(lds_addr(sbias)), off);
  }
  // NS - 1 stages ahead (one with a single buffer)
  static_for<0, (NS > 1 ? NS - 1 : 1)>([&](auto i) { issue(i); });
  // full rounds of NS stages (stage t in buffer t % NS), then the tail
  int t = 0;
  for (; t + NS <= nkt; t += NS) static_for<0, NS>(round_step);
  const int rem = nkt - t;
  if constexpr (NS > 1) {
    static_for<0, NS - 1>([&](auto i) {
      if (rem > decltype(i)::value) round_step(i);
    });
  }
  // all fills (including the zero fills past the end) landed, all waves
  // done reading the operand buffers
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");

  if (SPLIT) {
    // fp32 partials of this split: accumulator elements are 4 consecutive
    // channels (4 (lane/16) + e) of pixel lane % 16
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
      for (int j = 0; j < TM; ++j) {
        const int m = m0 + wm * WTM + j * 16 + (lane & 15);
        const int k = n0 + wn * WTN + i * 16 + 4 * (lane >> 4);
        if (m >= p.M || k >= p.Kp) continue;
        const f32x4 a = acc[i][j];
        *(float4*)(p.partial + ((size_t)blockIdx.y * p.M + m) * p.Kp + k) = make_float4(a[0], a[1], a[2], a[3]);
      }
    return;
  }

  // Epilogue through LDS: each group parks its fp32 sums of a 32-channel
  // slice in a [BM][kEC + 4] tile in its ring (the pad puts the 16 pixels of
  // one accumulator write on distinct banks); every thread then takes 8
  // consecutive channels of one pixel, adds the groups' sums in group order,
  // bias and residual, applies the activation and stores 16 bytes.
  constexpr int kLd = kEC + 4;
  static_assert(BM * kLd * 4 <= STAGE * 16, "staging tile");
  float* stage = reinterpret_cast<float*>(gring);
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
      for (int q = 0; q < EPV; ++q) {
        const int px = (tid + q * kNTall) / TPP;
        const int m = m0 + px;
        if (px >= BM || m >= p.M || k >= p.Kp) continue;
        const float* st0 = reinterpret_cast<const float*>(ring) + px * kLd + ec8;
        float4 lo = *(const float4*)st0;
        float4 hi = *(const float4*)(st0 + 4);
#pragma unroll
        for (int g = 1; g < KG; ++g) {
          const float* stg = reinterpret_cast<const float*>(ring + g * NS * STAGE) + px * kLd + ec8;
          const float4 l2 = *(const float4*)stg, h2 = *(const float4*)(stg + 4);
          lo.x += l2.x; lo.y += l2.y; lo.z += l2.z; lo.w += l2.w;
          hi.x += h2.x; hi.y += h2.y; hi.z += h2.z; hi.w += h2.w;
        }
        float f[8], rv[8];
        const float4 b0 = sbias[(pass * kEC + ec8) / 4], b1 = sbias[(pass * kEC + ec8) / 4 + 1];
        unpack8(resv[pass][q], rv);
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

template <int BM, int BN, int WM, int WN, int KG, int NS>
hipError_t launch_tile(const ConvParams& p_in, hipStream_t s) {
  ConvParams p = p_in;
  const bool aligned = (p.Cp % kBK) == 0 && p.R * p.S <= 32;
  const bool split = p.splits > 1;
  if (KG > 1 && split) return hipErrorInvalidValue;
  const int blocks = placed_blocks(p, BM, BN);
  dim3 grid(blocks, split ? p.splits : 1);
  constexpr int kThreads = 64 * WM * WN * KG;
  if constexpr (KG == 1) {
    if (aligned && !split) conv_dma_kernel<BM, BN, WM, WN, 1, NS, true, false><<<grid, kThreads, 0, s>>>(p);
    else if (aligned) conv_dma_kernel<BM, BN, WM, WN, 1, NS, true, true><<<grid, kThreads, 0, s>>>(p);
    else if (!split) conv_dma_kernel<BM, BN, WM, WN, 1, NS, false, false><<<grid, kThreads, 0, s>>>(p);
    else conv_dma_kernel<BM, BN, WM, WN, 1, NS, false, true><<<grid, kThreads, 0, s>>>(p);
  } else {
    if (aligned) conv_dma_kernel<BM, BN, WM, WN, KG, NS, true, false><<<grid, kThreads, 0, s>>>(p);
    else conv_dma_kernel<BM, BN, WM, WN, KG, NS, false, false><<<grid, kThreads, 0, s>>>(p);
  }
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN, int KG>
hipError_t launch_stages(const ConvParams& p, int ns, hipStream_t s) {
  constexpr int kStage = (BM + BN) * 128 * KG;  // bytes of one ring slot, all groups
  constexpr int kFixed = 64 * 16;                // the bias table (one wave's fill)
  hipError_t r = hipErrorInvalidValue;
  static_for<1, kMaxStages + 1>([&](auto i) {
    constexpr int NS = decltype(i)::value;
    if constexpr (NS * kStage + kFixed <= kLdsLimit)
      if (ns == NS) r = launch_tile<BM, BN, WM, WN, KG, NS>(p, s);
  });
  return r;
}

}  // namespace

bool conv_dma_tile_supported(int bm, int bn, int stages, int threads, int kgroups) {
  if (stages < 1 || stages > kMaxStages || (kgroups != 1 && kgroups != 2 && kgroups != 4)) return false;
  if ((bm + bn) * 128 * stages * kgroups + 64 * 16 > kLdsLimit) return false;  // LDS: stage rings + bias
  const int waves = threads / (64 * kgroups);  // per reduction group
  if (threads != 64 * waves * kgroups) return false;
  if (waves == 4 && kgroups == 4) return (bm == 64 && bn == 64) || (bm == 32 && bn == 64);
  if (waves == 4)
    return (bm == 128 && bn == 128) || (bm == 128 && bn == 64) || (bm == 64 && bn == 128) ||
           (bm == 64 && bn == 64) || (bm == 32 && bn == 64) ||
           (kgroups == 1 && ((bm == 64 && bn == 256) || (bm == 256 && bn == 64)));
  if (waves == 8 && kgroups == 1)
    return (bm == 128 && bn == 128) || (bm == 128 && bn == 64) || (bm == 64 && bn == 128) ||
           (bm == 128 && bn == 256) || (bm == 256 && bn == 128);
  return false;
}

hipError_t launch_conv_dma(const ConvParams& p, int bm, int bn, int stages, int threads, int kgroups,
                           hipStream_t s) {
  if (!conv_dma_tile_supported(bm, bn, stages, threads, kgroups)) return hipErrorInvalidValue;
  if (kgroups == 4) {
    if (bm == 64 && bn == 64) return launch_stages<64, 64, 2, 2, 4>(p, stages, s);
    if (bm == 32 && bn == 64) return launch_stages<32, 64, 1, 4, 4>(p, stages, s);
    return hipErrorInvalidValue;
  }
  if (kgroups == 2) {
    if (bm == 128 && bn == 128) return launch_stages<128, 128, 2, 2, 2>(p, stages, s);
    if (bm == 128 && bn == 64) return launch_stages<128, 64, 2, 2, 2>(p, stages, s);
    if (bm == 64 && bn == 128) return launch_stages<64, 128, 2, 2, 2>(p, stages, s);
    if (bm == 64 && bn == 64) return launch_stages<64, 64, 2, 2, 2>(p, stages, s);
    if (bm == 32 && bn == 64) return launch_stages<32, 64, 1, 4, 2>(p, stages, s);
    return hipErrorInvalidValue;
  }
  if (threads == 512) {
    if (bm == 128 && bn == 256) return launch_stages<128, 256, 2, 4, 1>(p, stages, s);
    if (bm == 256 && bn == 128) return launch_stages<256, 128, 4, 2, 1>(p, stages, s);
    if (bm == 128 && bn == 128) return launch_stages<128, 128, 2, 4, 1>(p, stages, s);
    if (bm == 128 && bn == 64) return launch_stages<128, 64, 4, 2, 1>(p, stages, s);
    if (bm == 64 && bn == 128) return launch_stages<64, 128, 2, 4, 1>(p, stages, s);
    return hipErrorInvalidValue;
  }
  if (bm == 64 && bn == 256) return launch_stages<64, 256, 1, 4, 1>(p, stages, s);
  if (bm == 256 && bn == 64) return launch_stages<256, 64, 4, 1, 1>(p, stages, s);
  if (bm == 128 && bn == 128) return launch_stages<128, 128, 2, 2, 1>(p, stages, s);
  if (bm == 128 && bn == 64) return launch_stages<128, 64, 2, 2, 1>(p, stages, s);
  if (bm == 64 && bn == 128) return launch_stages<64, 128, 2, 2, 1>(p, stages, s);
  if (bm == 64 && bn == 64) return launch_stages<64, 64, 2, 2, 1>(p, stages, s);
  if (bm == 32 && bn == 64) return launch_stages<32, 64, 1, 4, 1>(p, stages, s);
  return hipErrorInvalidValue;
}

}  // namespace byoc
