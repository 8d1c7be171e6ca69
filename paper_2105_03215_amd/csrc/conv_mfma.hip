// Implicit-GEMM convolution on CDNA4 bf16 MFMA (v_mfma_f32_16x16x32_bf16).
//
// The conv composite y[n,p,q,k] = act(sum_{r,s,c} x[n, p*sh-pt+r, q*sw-pl+s, c]
// * w[k,r,s,c] + b[k] + res[n,p,q,k]) is a GEMM with M = N*P*Q output
// pixels, N = K output channels and a reduction of length R*S*C.  With NHWC
// activations and weights packed K-major with kk = (r*S+s)*Cp + c, a row of
// either operand is contiguous along the reduction, so every lane moves 16
// bytes (8 bf16) per global load and per LDS read, which is exactly one MFMA
// operand register.  Dense layers run through the same kernel as 1x1 convs
// on 1x1 images.
//
// Workgroup: 256 threads = 4 waves; tile BM pixels x BN channels; the
// reduction advances 64 elements per LDS stage (two MFMA k-steps).  Global
// loads run two stages ahead through two register sets; LDS is double
// buffered with one barrier per stage.  LDS rows are 128
// bytes (8 chunks of 16 B) with the chunk index XOR-swizzled by the row so
// that the 16 rows one MFMA operand read touches fall on distinct banks.
//
// The weights are the MFMA A operand and the pixels the B operand, so each
// lane's 4 accumulators hold 4 consecutive output channels of one pixel:
// the epilogue reads 4 biases, 4 residual values and writes 8 contiguous
// bytes per lane, with bias, residual add, activation and bf16 rounding
// fused.  With split-K each split writes fp32 partials and a second kernel
// reduces them in a fixed order (bitwise reproducible) with the same
// epilogue.
#include <type_traits>

#include "device_common.h"

namespace byoc {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr int kBK = 64;          // reduction elements per stage
constexpr int kCH = kBK / 8;     // 16-byte chunks per tile row
constexpr int kNT = 256;         // threads per workgroup
constexpr int kRowsPerPass = kNT / kCH;
// Buffer resource word 3 for raw (untyped, stride 0) buffer access on gfx9.
constexpr int kBufferFlags = 0x00020000;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

// Per-thread state of one workgroup's main loop.  The two prefetch register
// sets are members indexed by a template parameter so that they stay in
// VGPRs (never addressable memory).
template <int BM, int BN, int WM, int WN, int MF, bool ALIGNED>
struct ConvTileLoop {
  static constexpr int WTM = BM / WM;
  static constexpr int WTN = BN / WN;
  static constexpr int TM = WTM / MF;  // MFMA tiles per wave along pixels
  static constexpr int TN = WTN / MF;  // and along channels
  static constexpr int AR = BM / kRowsPerPass;
  static constexpr int BR = BN / kRowsPerPass;

  using Acc = typename std::conditional<MF == 32, f32x16, f32x4>::type;
  uint4 ra[2][AR];
  uint4 rb[2][BR];
  Acc acc[TN][TM];
  // Activation rows.  Aligned path: pix = element offset of the row's
  // window origin plus this thread's 8 channels, tapmask bit r*S+s set when
  // that tap lies inside the image.  Non-aligned path: the window origin.
  int pix[AR], a_ih[AR], a_iw[AR];
  uint32_t tapmask[AR];
  __amdgpu_buffer_rsrc_t xr, wr;
  uint32_t wvoff[BR];  // byte offset of this thread's weight rows and chunk
  // reduction position of the next load: tap (r, s), channel c, flattened
  // index kk (non-aligned path) and packed-weight column
  int r, s, c, kk, wcol;
  int cv, r0, lane, wm, wn;

  __device__ __forceinline__ void advance(const ConvParams& p) {
    wcol += kBK;
    if (ALIGNED) {
      // c is the wave-uniform channel base of the stage (Cp % 64 == 0)
      c += kBK;
      if (c == p.Cp) {
        c = 0;
        if (++s == p.S) {
          s = 0;
          ++r;
        }
      }
    } else {
      kk += kBK;
      c += kBK;
      while (c >= p.Cp) {
        c -= p.Cp;
        if (++s == p.S) {
          s = 0;
          ++r;
        }
      }
    }
  }

  // Raw buffer loads: an out-of-range offset returns zeros, which supplies
  // the conv padding and the ragged pixel/reduction tails without branches.
  // The position advances before every load but the first; a load asked
  // for past the last stage (more == false) re-reads the last stage, whose
  // data is then never used.
  template <int SET>
  __device__ __forceinline__ void load(const ConvParams& p, bool first, bool more) {
    if (!first && more) advance(p);
    if (ALIGNED) {
      const int tap = (r * p.W + s) * p.Cp + c;
      const int bit = r * p.S + s;
#pragma unroll
      for (int i = 0; i < AR; ++i) {
        const bool ok = (tapmask[i] >> bit) & 1u;
        const uint32_t off = ok ? (uint32_t)(pix[i] + tap) * 2u : 0x80000000u;
        ra[SET][i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
      }
    } else {
      const bool kval = kk < p.Kg;
      const int tap = (r * p.W + s) * p.Cp + c;
#pragma unroll
      for (int i = 0; i < AR; ++i) {
        const int ih = a_ih[i] + r;
        const int iw = a_iw[i] + s;
        const bool ok = kval && (unsigned)ih < (unsigned)p.H && (unsigned)iw < (unsigned)p.W;
        const uint32_t off = ok ? (uint32_t)(pix[i] + tap) * 2u : 0x80000000u;
        ra[SET][i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
      }
    }
    const uint32_t wc = (uint32_t)wcol * 2u;
#pragma unroll
    for (int i = 0; i < BR; ++i)
      rb[SET][i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(wr, wvoff[i] + wc, 0, 0));
  }

  template <int SET>
  __device__ __forceinline__ void store(uint4* sA, uint4* sB) {
#pragma unroll
    for (int i = 0; i < AR; ++i) {
      const int row = r0 + i * kRowsPerPass;
      sA[row * kCH + (cv ^ (row & 7))] = ra[SET][i];
    }
#pragma unroll
    for (int i = 0; i < BR; ++i) {
      const int row = r0 + i * kRowsPerPass;
      sB[row * kCH + (cv ^ (row & 7))] = rb[SET][i];
    }
  }

  // One LDS stage (64 reduction elements): 2 k-steps of the 16x16x32 MFMA
  // or 4 of the 32x32x16 one.  Lane l reads 16 bytes (8 consecutive
  // reduction elements) of row l % MF at chunk (k-step, l / MF).
  __device__ __forceinline__ void compute(const uint4* sA, const uint4* sB) {
    constexpr int KS = MF == 32 ? 16 : 32;
    constexpr int GROUPS = 64 / MF;  // lane groups sharing a row
#pragma unroll
    for (int ks = 0; ks < kBK / KS; ++ks) {
      const int chunk = ks * (KS / 8) + (lane / MF);
      bf16x8 af[TN], bfr[TM];
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int row = wn * WTN + i * MF + (lane % MF);
        af[i] = as_bf16x8(sB[row * kCH + (chunk ^ (row & 7))]);
      }
#pragma unroll
      for (int j = 0; j < TM; ++j) {
        const int row = wm * WTM + j * MF + (lane % MF);
        bfr[j] = as_bf16x8(sA[row * kCH + (chunk ^ (row & 7))]);
      }
      (void)GROUPS;
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j) {
          if constexpr (MF == 32)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
          else
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
    }
  }

  // Channel (row of the MFMA output) held by accumulator element e of this
  // lane, relative to the MFMA tile: 16x16 -> 4 (lane/16) + e; 32x32 ->
  // 8 (e/4) + 4 (lane/32) + e%4.  The pixel (column) is lane % MF.
  __device__ __forceinline__ int acc_row(int e) const {
    if (MF == 32) return 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
    return 4 * (lane >> 4) + e;
  }
};

template <int BM, int BN, int WM, int WN, int MF, bool ALIGNED, bool SPLIT>
__global__ __launch_bounds__(kNT, 2) void conv_mfma_kernel(ConvParams p) {
  using L = ConvTileLoop<BM, BN, WM, WN, MF, ALIGNED>;
  static_assert(WM * WN == 4, "4 waves");
  static_assert(L::TM >= 1 && L::TN >= 1 && L::AR >= 1 && L::BR >= 1, "tile too small");
  constexpr int WTM = L::WTM, WTN = L::WTN, TM = L::TM, TN = L::TN, AR = L::AR;

  // Main-loop operand tiles (double buffered); the epilogue reuses the same
  // memory as an fp32 staging tile.
  __shared__ uint4 smem[2 * (BM + BN) * kCH];
  uint4 (*sA)[BM * kCH] = reinterpret_cast<uint4 (*)[BM * kCH]>(smem);
  uint4 (*sB)[BN * kCH] = reinterpret_cast<uint4 (*)[BN * kCH]>(smem + 2 * BM * kCH);

  materialize_args(p);
  L st;
  const int tid = threadIdx.x;
  st.lane = tid & 63;
  const int wave = tid >> 6;
  st.wm = wave / WN;
  st.wn = wave % WN;
  const int lane = st.lane, wm = st.wm, wn = st.wn;

  // Tile order: workgroups are dealt round-robin to the 8 XCDs; remap so
  // that each XCD gets a contiguous run of tiles (shared activation rows
  // stay in one L2).
  const int ntn = (p.Kp + BN - 1) / BN;
  int bid = blockIdx.x;
  const int nb = ((p.M + BM - 1) / BM) * ntn;  // the launch grid (no kernel-argument fetch)
  if ((nb & 7) == 0) bid = (bid & 7) * (nb >> 3) + (bid >> 3);
  const int tm = mdiv(bid, p.mg_tile);
  const int tn = bid - tm * ntn;
  const int m0 = tm * BM;
  const int n0 = tn * BN;

  const int nk_total = (p.Kg + kBK - 1) / kBK;
  int kt_begin = 0, kt_end = nk_total;
  if (SPLIT) {
    kt_begin = blockIdx.y * p.k_tiles_per_split;
    kt_end = min(nk_total, kt_begin + p.k_tiles_per_split);
  }

  st.cv = tid & (kCH - 1);
  st.r0 = tid / kCH;
  const int PQ = p.P * p.Q;
#pragma unroll
  for (int i = 0; i < AR; ++i) {
    const int m = m0 + st.r0 + i * kRowsPerPass;
    int ih0 = -(1 << 28), iw0 = 0, n = 0;  // rows past M: never inside the image
    if (m < p.M) {
      n = mdiv(m, p.mg_pq);
      const int pq = m - n * PQ;
      const int pp = mdiv(pq, p.mg_q);
      const int qq = pq - pp * p.Q;
      ih0 = pp * p.sh - p.pt;
      iw0 = qq * p.sw - p.pl;
    }
    st.a_ih[i] = ih0;
    st.a_iw[i] = iw0;
    st.pix[i] = m < p.M ? ((n * p.H + ih0) * p.W + iw0) * p.Cp : 0;
    if (ALIGNED) {
      st.pix[i] += st.cv * 8;
      uint32_t mask = 0;
      for (int r = 0; r < p.R; ++r)
        for (int s = 0; s < p.S; ++s)
          if ((unsigned)(ih0 + r) < (unsigned)p.H && (unsigned)(iw0 + s) < (unsigned)p.W)
            mask |= 1u << (r * p.S + s);
      st.tapmask[i] = mask;
    }
  }
  st.xr = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(p.x), (short)0, p.x_bytes, kBufferFlags);
  st.wr = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(p.w), (short)0, p.w_bytes, kBufferFlags);
#pragma unroll
  for (int i = 0; i < L::BR; ++i)
    st.wvoff[i] = (uint32_t)(((n0 + st.r0 + i * kRowsPerPass) * p.Kgp + st.cv * 8) * 2);
  // starting reduction position (aligned: wave-uniform stage origin; the
  // thread's 8 channels are added at use)
  {
    const int kk0 = kt_begin * kBK + (ALIGNED ? 0 : st.cv * 8);
    const int rs = mdiv(kk0, p.mg_cp);
    st.c = kk0 - rs * p.Cp;
    st.r = mdiv(rs, p.mg_s);
    st.s = rs - st.r * p.S;
    st.kk = kk0;
    st.wcol = kt_begin * kBK;
  }
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) st.acc[i][j] = typename L::Acc{};

  // Two register sets: the loads of tile t+2 are issued before the MFMAs
  // of tile t and written to LDS after those of tile t+1.
  // Epilogue operands (bias and residual of the 8 channels this thread will
  // finish for each of its pixels) are fetched before the main loop, so their
  // latency overlaps the reduction instead of following it.
  constexpr int kEC = 64;              // channels per epilogue pass
  constexpr int NPASS = BN / kEC;
  constexpr int EPV = BM * (kEC / 8) / kNT;  // pixels per thread per pass
  static_assert(EPV >= 1, "epilogue vectors");
  const int ec8 = (tid % (kEC / 8)) * 8;
  uint4 resv[NPASS][EPV];
  float4 biasv[NPASS][2];
  if (!SPLIT) {
    const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16_t*>(p.res), (short)0, p.res ? p.res_bytes : 0, kBufferFlags);
#pragma unroll
    for (int pass = 0; pass < NPASS; ++pass) {
      const int k = n0 + pass * kEC + ec8;
      if (p.bias) {
        biasv[pass][0] = *(const float4*)(p.bias + k);
        biasv[pass][1] = *(const float4*)(p.bias + k + 4);
      } else {
        biasv[pass][0] = biasv[pass][1] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int q = 0; q < EPV; ++q) {
        const int m = m0 + (tid + q * kNT) / (kEC / 8);
        const uint32_t off = (m < p.M && k < p.Kp) ? (uint32_t)(m * p.ldr + k) * 2u : 0x80000000u;
        resv[pass][q] = p.res ? __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rr, off, 0, 0))
                              : make_uint4(0u, 0u, 0u, 0u);
      }
    }
  }

  const int nkt = kt_end - kt_begin;
  if (nkt > 0) {
    st.template load<0>(p, true, true);
    st.template load<1>(p, false, nkt > 1);
    st.template store<0>(sA[0], sB[0]);
    __syncthreads();
    for (int t = 0; t < nkt; t += 2) {
      // LDS 0 holds tile t, register set 1 holds tile t+1
      st.template load<0>(p, false, t + 2 < nkt);
      st.compute(sA[0], sB[0]);
      st.template store<1>(sA[1], sB[1]);
      __syncthreads();
      // LDS 1 holds tile t+1 (a repeat of the last tile past the end),
      // register set 0 holds tile t+2
      st.template load<1>(p, false, t + 3 < nkt);
      if (t + 1 < nkt) st.compute(sA[1], sB[1]);
      st.template store<0>(sA[0], sB[0]);
      __syncthreads();
    }
  }

  constexpr int NE = MF == 32 ? 16 : 4;  // accumulator elements per lane per tile
  if (SPLIT) {
    // fp32 partials of this split: each group of 4 accumulator elements is
    // 4 consecutive channels of one pixel
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
      for (int j = 0; j < TM; ++j) {
        const int m = m0 + wm * WTM + j * MF + (lane % MF);
#pragma unroll
        for (int e = 0; e < NE; e += 4) {
          const int k = n0 + wn * WTN + i * MF + st.acc_row(e);
          if (m >= p.M || k >= p.Kp) continue;
          *(float4*)(p.partial + ((size_t)blockIdx.y * p.M + m) * p.Kp + k) =
              make_float4(st.acc[i][j][e], st.acc[i][j][e + 1], st.acc[i][j][e + 2], st.acc[i][j][e + 3]);
        }
      }
    return;
  }

  // Epilogue through LDS, 64 channels per pass: the waves park their fp32
  // accumulators in a [BM][64 + 4] tile, then every thread takes 8
  // consecutive channels of one pixel, adds bias and residual, applies the
  // activation, rounds to bf16 and writes 16 bytes; 8 neighbouring lanes
  // cover one pixel's 128-byte run, so stores and residual loads are whole
  // cache lines.
  constexpr int kLd = kEC + 4;  // padded row (floats): 16 rows hit distinct banks
  static_assert(BN % kEC == 0 && BM * kLd * 4 <= (int)sizeof(smem), "staging tile");
  float* stage = reinterpret_cast<float*>(smem);
  const ActClamp ac = act_clamp_of(p.act, p.alpha);
  auto epilogue = [&](auto mode_tag) {
    constexpr int G = decltype(mode_tag)::value;
#pragma unroll
    for (int pass = 0; pass < NPASS; ++pass) {
      lds_barrier();
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j) {
          const int px = wm * WTM + j * MF + (lane % MF);
#pragma unroll
          for (int e = 0; e < NE; e += 4) {
            const int ch = wn * WTN + i * MF + st.acc_row(e) - pass * kEC;
            if (ch < 0 || ch >= kEC) continue;
            *(float4*)(stage + px * kLd + ch) =
                make_float4(st.acc[i][j][e], st.acc[i][j][e + 1], st.acc[i][j][e + 2], st.acc[i][j][e + 3]);
          }
        }
      lds_barrier();
      const int k = n0 + pass * kEC + ec8;
#pragma unroll
      for (int q = 0; q < EPV; ++q) {
        const int px = (tid + q * kNT) / (kEC / 8);
        const int m = m0 + px;
        if (m >= p.M || k >= p.Kp) continue;
        float f[8], r[8];
        const float4 lo = *(const float4*)(stage + px * kLd + ec8);
        const float4 hi = *(const float4*)(stage + px * kLd + ec8 + 4);
        const float4 b0 = biasv[pass][0], b1 = biasv[pass][1];
        unpack8(resv[pass][q], r);
        f[0] = lo.x + b0.x; f[1] = lo.y + b0.y; f[2] = lo.z + b0.z; f[3] = lo.w + b0.w;
        f[4] = hi.x + b1.x; f[5] = hi.y + b1.y; f[6] = hi.z + b1.z; f[7] = hi.w + b1.w;
#pragma unroll
        for (int e = 0; e < 8; ++e) f[e] = epilogue_value<G>(f[e], r[e], ac);
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

// Split-K reduction: one thread per 4 channels of one pixel; partials summed
// in split order, then bias, residual, activation, bf16 rounding.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(ConvParams p) {
  const int k4 = p.Kp / 4;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;  // < M * Kp / 4 < 2^29
  if (idx >= p.M * k4) return;
  const int m = mdiv(idx, p.mg_tile);  // mg_tile divides by Kp / 4 here
  const int k = (idx - m * k4) * 4;
  // bias and residual first, then the partials of up to 8 splits at a time,
  // all loads in flight before the first add; the sum runs in split order
  const float4 bv = p.bias ? *(const float4*)(p.bias + k) : make_float4(0.f, 0.f, 0.f, 0.f);
  const uint2 rr = p.res ? *(const uint2*)(p.res + (size_t)m * p.ldr + k) : make_uint2(0u, 0u);
  const size_t stride = (size_t)p.M * p.Kp;
  const float* part = p.partial + (size_t)m * p.Kp + k;
  float4 acc = *(const float4*)part;
  for (int sp0 = 1; sp0 < p.splits; sp0 += 8) {
    float4 t[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      t[j] = sp0 + j < p.splits ? *(const float4*)(part + (size_t)(sp0 + j) * stride) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (sp0 + j < p.splits) {
        acc.x += t[j].x;
        acc.y += t[j].y;
        acc.z += t[j].z;
        acc.w += t[j].w;
      }
  }
  if (p.bias) {
    acc.x += bv.x;
    acc.y += bv.y;
    acc.z += bv.z;
    acc.w += bv.w;
  }
  float r[4] = {0.f, 0.f, 0.f, 0.f};
  if (p.res) {
    r[0] = __uint_as_float(rr.x << 16);
    r[1] = __uint_as_float(rr.x & 0xFFFF0000u);
    r[2] = __uint_as_float(rr.y << 16);
    r[3] = __uint_as_float(rr.y & 0xFFFF0000u);
  }
  float v[4] = {acc.x, acc.y, acc.z, acc.w};
  if (p.res_post) {
    const ActClamp ac = act_clamp_of(p.act, p.alpha);
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = epilogue_value<3>(v[e], r[e], ac);
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = apply_act(v[e] + r[e], p.act, p.alpha);
  }
  *(uint2*)(p.y + (size_t)m * p.ldy + k) = make_uint2(pack2_bf16(v[0], v[1]), pack2_bf16(v[2], v[3]));
}

template <int BM, int BN, int WM, int WN, int MF>
hipError_t launch_tile(const ConvParams& p_in, hipStream_t s) {
  ConvParams p = p_in;
  const int ntm = (p.M + BM - 1) / BM;
  const int ntn = (p.Kp + BN - 1) / BN;
  const bool aligned = (p.Cp % kBK) == 0 && p.R * p.S <= 32;
  const bool split = p.splits > 1;
  p.mg_tile = magic40(ntn);
  dim3 grid(ntm * ntn, split ? p.splits : 1);
  if (aligned && !split) conv_mfma_kernel<BM, BN, WM, WN, MF, true, false><<<grid, kNT, 0, s>>>(p);
  else if (aligned) conv_mfma_kernel<BM, BN, WM, WN, MF, true, true><<<grid, kNT, 0, s>>>(p);
  else if (!split) conv_mfma_kernel<BM, BN, WM, WN, MF, false, false><<<grid, kNT, 0, s>>>(p);
  else conv_mfma_kernel<BM, BN, WM, WN, MF, false, true><<<grid, kNT, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace

bool conv_mfma_tile_supported(int bm, int bn, int mf) {
  if (mf == 16)
    return (bm == 128 && bn == 128) || (bm == 128 && bn == 64) || (bm == 64 && bn == 128) ||
           (bm == 64 && bn == 64) || (bm == 32 && bn == 64);
  if (mf == 32)
    return (bm == 128 && bn == 128) || (bm == 128 && bn == 64) || (bm == 64 && bn == 128) ||
           (bm == 64 && bn == 64);
  return false;
}

hipError_t launch_conv_mfma(const ConvParams& p, ConvTile t, hipStream_t s) {
  if (t.mf == 32) {
    if (t.bm == 128 && t.bn == 128) return launch_tile<128, 128, 2, 2, 32>(p, s);
    if (t.bm == 128 && t.bn == 64) return launch_tile<128, 64, 2, 2, 32>(p, s);
    if (t.bm == 64 && t.bn == 128) return launch_tile<64, 128, 2, 2, 32>(p, s);
    if (t.bm == 64 && t.bn == 64) return launch_tile<64, 64, 2, 2, 32>(p, s);
    return hipErrorInvalidValue;
  }
  if (t.bm == 128 && t.bn == 128) return launch_tile<128, 128, 2, 2, 16>(p, s);
  if (t.bm == 128 && t.bn == 64) return launch_tile<128, 64, 4, 1, 16>(p, s);
  if (t.bm == 64 && t.bn == 128) return launch_tile<64, 128, 1, 4, 16>(p, s);
  if (t.bm == 64 && t.bn == 64) return launch_tile<64, 64, 2, 2, 16>(p, s);
  if (t.bm == 32 && t.bn == 64) return launch_tile<32, 64, 1, 4, 16>(p, s);
  return hipErrorInvalidValue;
}

hipError_t launch_splitk_reduce(const ConvParams& p_in, hipStream_t s) {
  ConvParams p = p_in;
  p.mg_tile = magic40(p.Kp / 4);
  const int64_t n = (int64_t)p.M * (p.Kp / 4);
  splitk_reduce_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace byoc
