// Implicit-GEMM convolution on CDNA4 int8 MFMA (v_mfma_i32_16x16x64_i8)
// for partially quantized subgraphs (Sec. 3.2, Fig. 4a).
//
// The GEMM is the one of the bf16 kernels: M = N*P*Q output pixels, N = K
// output channels, a reduction over kk = (r*S + s)*Cp + c with NHWC int8
// activations and K-major packed int8 weights, so a row of either operand is
// contiguous along the reduction and every lane moves 16 bytes (16 codes,
// one MFMA operand register quadruple) per load.  The operand tiles stream
// from HBM straight into a ring of NS LDS buffers (buffer_load ... lds), 128
// reduction elements per stage; a 128-byte LDS row holds one operand row of
// a stage with the chunk swizzle ch ^ (row & 7) applied on the fetch side.
// Accumulation is exact in int32.
//
// Zero points.  The MFMA sums x_q * w_q over the taps inside the image (a
// tap outside reads zeros).  The affine input needs sum (x_q - Z_x) w_q: the
// host folds -Z_x * (sum of all weights of channel k) into the bias, and for
// a pixel whose window crosses the border the epilogue adds back Z_x times
// the weight sums of its taps outside the image (wtap[r*S + s][k]).
//
// Reduction groups (KG > 1): KG groups of WM x WN waves each run their own
// ring over every KG-th stage of the reduction (group g: stages g, g + KG,
// ...), which multiplies the loads in flight of a workgroup on layers with
// few tiles and long reductions; the groups' int32 sums are added in the
// epilogue (exact in any order, so every tile and group count gives the
// same codes).
//
// Epilogue: each thread finishes 8 consecutive channels of one pixel from
// int32 sums staged in LDS: bias, border correction, float32 rescaling
// (one rounding per term, the per-channel bias and factor read from LDS),
// the residual's own rescaling, the activation clamp in code space (which
// also clips to int8), one 8-byte store.
#include "lds_dma.h"
#include "quant_epilogue.h"

namespace byoc {
namespace {

using namespace dma;

constexpr int kBK = 128;       // reduction elements (bytes) per stage
constexpr int kCH = 8;         // 16-byte chunks per tile row
constexpr int kCE = 16;        // reduction elements per chunk
constexpr int kMaxStages = 4;

__device__ __forceinline__ i32x4 as_i32x4(uint4 u) { return __builtin_bit_cast(i32x4, u); }

template <int BM, int BN, int WM, int WN, int KG, int NS, bool ALIGNED>
__global__ __launch_bounds__(64 * WM * WN * KG) void conv_i8_kernel(QConvParams q) {
  static_assert(WM * WN == 4 || WM * WN == 8, "4 or 8 waves per reduction group");
  static_assert(KG == 1 || KG == 2 || KG == 4, "reduction groups");
  const ConvParams& p = q.g;
  constexpr int kNT = 64 * WM * WN;  // threads of one reduction group
  constexpr int kNTall = kNT * KG;   // threads of the workgroup
  constexpr int kRowsPerPass = kNT / kCH;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 16, TN = WTN / 16;
  constexpr int AR = BM / kRowsPerPass, BR = BN / kRowsPerPass;
  static_assert(TM >= 1 && TN >= 1 && AR >= 1 && BR >= 1, "tile too small");
  constexpr int LPS = AR + BR;
  constexpr int STAGE = (BM + BN) * kCH;  // uint4 per stage buffer
  static_assert(NS >= 2 && NS <= kMaxStages, "stages");

  __shared__ uint4 ring[KG * NS * STAGE];
  __shared__ int2 sq[128];  // the tile's {bias, factor} (one wave's 16-byte fill: 128 channels)
  materialize_args(p);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int kg = __builtin_amdgcn_readfirstlane(tid / kNT);                  // reduction group
  const int tg = tid - kg * kNT;                                               // thread within the group
  const int wave = __builtin_amdgcn_readfirstlane((tid >> 6) % (WM * WN));  // wave within the group
  uint4* const gring = ring + kg * NS * STAGE;
  auto buf = [&](auto tag) -> uint4* { return gring + decltype(tag)::value * STAGE; };
  const int wm = wave / WN, wn = wave % WN;
  const int r0 = tg / kCH;
  const int cv = (lane & 7) ^ ((lane >> 3) & 7);

  int tm, tn;
  if (!place_tile<BM, BN>(p, &tm, &tn)) return;
  const int m0 = tm * BM;
  const int n0 = tn * BN;
  const int nkt = (p.Kg + kBK - 1) / kBK;

  // Activation rows of this thread (see the bf16 kernel): element (= byte)
  // offset of the window origin plus this thread's chunk, and on the
  // aligned path (a stage is 128 channels of one tap) the taps inside.
  int pix[AR], a_ih[AR], a_iw[AR];
  uint32_t tapmask[AR];
  const int PQ = p.P * p.Q;
#pragma unroll
  for (int i = 0; i < AR; ++i) {
    const int m = m0 + r0 + i * kRowsPerPass;
    int ih0 = -(1 << 28), iw0 = 0, n = 0;
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
      pix[i] += cv * kCE;
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
  uint32_t wvoff[BR];
#pragma unroll
  for (int i = 0; i < BR; ++i) wvoff[i] = (uint32_t)((n0 + r0 + i * kRowsPerPass) * p.Kgp + cv * kCE);

  // reduction position of this group's first stage
  int r, s, c, kk, wcol = kg * kBK;
  {
    kk = kg * kBK + (ALIGNED ? 0 : cv * kCE);
    const int rs = mdiv(kk, p.mg_cp);
    c = kk - rs * p.Cp;
    r = mdiv(rs, p.mg_s);
    s = rs - r * p.S;
  }

  // Loads of the next stage into buffer SET; past the end of the reduction
  // the offsets are out of range (zero fills), which keeps the count of
  // loads in flight fixed.
  int kleft = (nkt - kg + KG - 1) / KG;  // stages of this group
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
      const uint32_t off = ok ? (uint32_t)(pix[i] + tap) : kOOB;
      lds_fill16(xr, __builtin_amdgcn_readfirstlane(lds_addr(dst + (i * kRowsPerPass + wave * 8) * kCH)), off);
    }
#pragma unroll
    for (int i = 0; i < BR; ++i)
      lds_fill16(wr, __builtin_amdgcn_readfirstlane(lds_addr(dst + (BM + i * kRowsPerPass + wave * 8) * kCH)),
                 live ? wvoff[i] + (uint32_t)wcol : kOOB);
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

  i32x4 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = i32x4{0, 0, 0, 0};

  // One stage: 2 k-steps of the 16x16x64 MFMA; lane l reads 16 codes of
  // row l % 16 at chunk (k-step, l / 16) of both operands.
  auto compute = [&](auto set_tag) {
    const uint4* sA = buf(set_tag);
    const uint4* sB = sA + BM * kCH;
#pragma unroll
    for (int ks = 0; ks < kBK / 64; ++ks) {
      const int chunk = ks * 4 + (lane >> 4);
      i32x4 af[TN], bfr[TM];
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int row = wn * WTN + i * 16 + (lane & 15);
        af[i] = as_i32x4(sB[row * kCH + (chunk ^ (row & 7))]);
      }
#pragma unroll
      for (int j = 0; j < TM; ++j) {
        const int row = wm * WTM + j * 16 + (lane & 15);
        bfr[j] = as_i32x4(sA[row * kCH + (chunk ^ (row & 7))]);
      }
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
  };

  // residual codes of the 8 channels this thread finishes per pass, fetched
  // before the reduction so that their latency overlaps it
  constexpr int kEC = 32;
  constexpr int NPASS = BN / kEC;
  constexpr int TPP = kEC / 8;
  constexpr int EPV = (BM * TPP + kNTall - 1) / kNTall;
  const int ec8 = (tid % TPP) * 8;
  uint2 resv[NPASS][EPV];
  {
    const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16_t*>(p.res), (short)0, p.res ? p.res_bytes : 0, kBufferFlags);
#pragma unroll
    for (int pass = 0; pass < NPASS; ++pass) {
      const int k = n0 + pass * kEC + ec8;
#pragma unroll
      for (int e = 0; e < EPV; ++e) {
        const int px = (tid + e * kNTall) / TPP;
        const int m = m0 + px;
        const uint32_t off = (px < BM && m < p.M && k < p.Kp) ? (uint32_t)(m * p.ldr + k) : kOOB;
        resv[pass][e] = p.res ? __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rr, off, 0, 0))
                              : make_uint2(0u, 0u);
      }
    }
  }

  // per-channel bias and factor of the tile, straight into LDS; issued
  // before the operand ring, so every later wait of this wave covers it
  static_assert(BN <= 128, "channel table");
  if (tid < 64) {
    const i32x4 qr = buffer_rsrc(q.qch, ((p.Kp + 255) / 256) * 256 * 8);
    lds_fill16(qr, __builtin_amdgcn_readfirstlane(lds_addr(sq)), 2 * lane < BN ? (uint32_t)(n0 + 2 * lane) * 8u : kOOB);
  }
  static_assert((NS - 2) * LPS <= 63, "vmcnt immediate");
  auto round_step = [&](auto i) {
    constexpr int I = decltype(i)::value;
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"((NS - 2) * LPS) : "memory");
    issue(std::integral_constant<int, (I + NS - 1) % NS>{});
    compute(i);
  };
  static_for<0, NS - 1>([&](auto i) { issue(i); });
  const int nsteps = (nkt + KG - 1) / KG;  // stages per group (the last ones may read zeros)
  int t = 0;
  for (; t + NS <= nsteps; t += NS) static_for<0, NS>(round_step);
  const int rem = nsteps - t;
  static_for<0, NS - 1>([&](auto i) {
    if (rem > decltype(i)::value) round_step(i);
  });
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");

  // each group parks its sums in its own ring; the finishing threads add
  // the groups' sums
  constexpr int kLd = kEC + 4;
  static_assert(BM * kLd * 4 <= STAGE * 16, "staging tile");
  int* stage = reinterpret_cast<int*>(gring);
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
      const int px = (tid + e * kNTall) / TPP;
      const int m = m0 + px;
      if (px >= BM || m >= p.M || k >= p.Kp) continue;
      const int* st = reinterpret_cast<const int*>(ring) + px * kLd + ec8;
      const int4 lo4 = *(const int4*)st, hi4 = *(const int4*)(st + 4);
      int a[8] = {lo4.x, lo4.y, lo4.z, lo4.w, hi4.x, hi4.y, hi4.z, hi4.w};
#pragma unroll
      for (int g = 1; g < KG; ++g) {
        const int* sg = reinterpret_cast<const int*>(ring + g * NS * STAGE) + px * kLd + ec8;
        const int4 l2 = *(const int4*)sg, h2 = *(const int4*)(sg + 4);
        a[0] += l2.x; a[1] += l2.y; a[2] += l2.z; a[3] += l2.w;
        a[4] += h2.x; a[5] += h2.y; a[6] += h2.z; a[7] += h2.w;
      }
      *(uint2*)(reinterpret_cast<int8_t*>(p.y) + (size_t)m * p.ldy + k) =
          finish8_i8(a, sq + pass * kEC + ec8, resv[pass][e], q, m, k);
    }
  }
}

template <int BM, int BN, int WM, int WN, int KG = 1>
hipError_t launch_tile(const QConvParams& q_in, int ns, hipStream_t s) {
  constexpr int kThreads = 64 * WM * WN * KG;
  QConvParams q = q_in;
  ConvParams& p = q.g;
  const bool aligned = (p.Cp % kBK) == 0 && p.R * p.S <= 32;
  const int blocks = placed_blocks(p, BM, BN);
  hipError_t r = hipErrorInvalidValue;
  static_for<2, kMaxStages + 1>([&](auto i) {
    constexpr int NS = decltype(i)::value;
    if constexpr (KG * NS * (BM + BN) * 128 + 1024 <= kLdsLimit) {
      if (ns != NS) return;
      if (aligned) conv_i8_kernel<BM, BN, WM, WN, KG, NS, true><<<blocks, kThreads, 0, s>>>(q);
      else conv_i8_kernel<BM, BN, WM, WN, KG, NS, false><<<blocks, kThreads, 0, s>>>(q);
      r = hipGetLastError();
    }
  });
  return r;
}

}  // namespace

bool conv_i8_tile_supported(int bm, int bn, int stages, int threads, int kgroups) {
  if (stages < 2 || stages > kMaxStages) return false;
  if (kgroups == 2 || kgroups == 4) {  // 4-wave groups
    if (threads != 256 * kgroups || kgroups * stages * (bm + bn) * 128 + 1024 > kLdsLimit) return false;
    return (bm == 64 && bn == 64) || (bm == 32 && bn == 64) || (kgroups == 2 && bm == 128 && bn == 64);
  }
  if (kgroups != 1) return false;
  if (threads == 512) return (bm == 128 && bn == 128) || (bm == 128 && bn == 64) || (bm == 64 && bn == 128);
  if (threads != 256) return false;
  return (bm == 128 && bn == 128) || (bm == 128 && bn == 64) || (bm == 64 && bn == 64) || (bm == 32 && bn == 64);
}

hipError_t launch_conv_i8(const QConvParams& p, int bm, int bn, int stages, int threads, int kgroups,
                          hipStream_t s) {
  if (!conv_i8_tile_supported(bm, bn, stages, threads, kgroups)) return hipErrorInvalidValue;
  if (p.g.Cp % kCE != 0 || p.g.Kp % 8 != 0 || p.g.Kgp % kBK != 0) return hipErrorInvalidValue;
  if (kgroups == 4) {
    if (bm == 64) return launch_tile<64, 64, 2, 2, 4>(p, stages, s);
    return launch_tile<32, 64, 1, 4, 4>(p, stages, s);
  }
  if (kgroups == 2) {
    if (bm == 128) return launch_tile<128, 64, 2, 2, 2>(p, stages, s);
    if (bm == 64) return launch_tile<64, 64, 2, 2, 2>(p, stages, s);
    return launch_tile<32, 64, 1, 4, 2>(p, stages, s);
  }
  if (threads == 512) {
    if (bm == 128 && bn == 128) return launch_tile<128, 128, 2, 4>(p, stages, s);
    if (bm == 128 && bn == 64) return launch_tile<128, 64, 4, 2>(p, stages, s);
    return launch_tile<64, 128, 2, 4>(p, stages, s);
  }
  if (bm == 128 && bn == 128) return launch_tile<128, 128, 2, 2>(p, stages, s);
  if (bm == 128 && bn == 64) return launch_tile<128, 64, 2, 2>(p, stages, s);
  if (bm == 64 && bn == 64) return launch_tile<64, 64, 2, 2>(p, stages, s);
  return launch_tile<32, 64, 1, 4>(p, stages, s);
}

}  // namespace byoc
