// Device helpers shared by the kernel files: bf16 conversion and activations.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "kernels.h"

namespace byoc {

// Raw buffer accesses: descriptor word 3 for untyped access on gfx9, and an
// offset past any buffer (reads return zeros, nothing is fetched).
constexpr int kBufferFlags = 0x00020000;
constexpr uint32_t kOOB = 0x80000000u;

__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}

// Round to nearest, ties to even (the hardware v_cvt_pk_bf16_f32 rounding).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  __bf16 v = (__bf16)f;
  return __builtin_bit_cast(bf16_t, v);
}

// Two values in one v_cvt_pk_bf16_f32 (same rounding as f32_to_bf16).
__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

// GELU(x) = x * Phi(x), Phi(x) = erfc(-x / sqrt 2) / 2 (the exact, erf-based
// form).  With a = |x| / sqrt 2: Phi(x) = erfc(a) / 2 for x < 0 (no
// cancellation for x << 0) and 1 - erfc(a) / 2 otherwise.  erfc(a) = k P(k)
// exp(-a^2), k = 1 / (1 + a / 2), P a degree-8 polynomial fitted to the
// scaled function exp(a^2) erfc(a) / k (csrc/gelu_erfc_fit.py prints the
// coefficients and the error); exp(-a^2) takes the rounded square s and its
// exact residual r = fma(a, a, -s) as exp(-s) (1 - r).  Relative error of
// erfc below 1e-6 in float32 over the whole normal range - far below the
// bf16 rounding of the output - in about 25 instructions, inlined.
__device__ __forceinline__ float gelu(float v) {
  constexpr float kErfcP[9] = {2.820777595e-01f, 2.825488448e-01f, 2.416709065e-01f, 2.090727836e-01f,
                               -4.348613694e-02f, 3.051838875e-01f, -5.132555962e-01f, 2.983081341e-01f,
                               -6.212075427e-02f};
  // (a capped at 10: erfc(10) is below the float32 range, and an infinite
  // input then gives GELU(+inf) = +inf)
  const float a = fminf(fabsf(v) * 0.70710678118654752440f, 10.0f);
  const float k = __builtin_amdgcn_rcpf(__builtin_fmaf(0.5f, a, 1.0f));
  float p = kErfcP[8];
#pragma unroll
  for (int i = 7; i >= 0; --i) p = __builtin_fmaf(p, k, kErfcP[i]);
  const float s = a * a;
  const float r = __builtin_fmaf(a, a, -s);
  const float e = expf(-s);
  const float ec = k * p * __builtin_fmaf(-e, r, e);  // erfc(a)
  const float phi = v < 0.0f ? 0.5f * ec : __builtin_fmaf(-0.5f, ec, 1.0f);
  return v * phi;
}

// Epilogue activation.  Kernels pick the GELU or the clamp instantiation
// once (the choice is uniform), so the per-element code has no branch:
// none / ReLU / ReLU6 / leaky ReLU are med3(max(v, slope * v), lo, hi) —
// slope 1 makes the max the value itself, slope alpha < 1 the leaky ReLU,
// [lo, hi] the clamps (none: [-inf, +inf]) — and GELU the out-of-line call
// above.
struct ActClamp {
  float lo;     // 0 for ReLU / ReLU6, -inf otherwise
  float hi;     // 6 for ReLU6, +inf otherwise
  float slope;  // alpha for the leaky ReLU, 1 otherwise
};
__device__ __forceinline__ ActClamp act_clamp_of(int act, float alpha) {
  const bool clamp0 = act == kActRelu || act == kActRelu6;
  return ActClamp{clamp0 ? 0.0f : -INFINITY, act == kActRelu6 ? 6.0f : INFINITY, act == kActLeaky ? alpha : 1.0f};
}
// MODE 0: any activation but GELU; 1: GELU; 2: none / ReLU / ReLU6 only
// (the clamp alone, for the hot epilogues that dispatch on the activation).
template <int MODE>
__device__ __forceinline__ float act_apply(float v, ActClamp a) {
  if constexpr (MODE == 1)
    return gelu(v);
  else if constexpr (MODE == 2)
    return __builtin_amdgcn_fmed3f(v, a.lo, a.hi);
  else
    return __builtin_amdgcn_fmed3f(fmaxf(v, v * a.slope), a.lo, a.hi);
}
// One output of a conv epilogue with residual r.  MODE 0-2 as above, the
// residual added before the activation; MODE 3 (any activation but GELU):
// the activation first, its output rounded to bf16, then the residual added
// (the arithmetic of a separate add node reading the conv's output).
template <int MODE>
__device__ __forceinline__ float epilogue_value(float v, float r, ActClamp a) {
  if constexpr (MODE == 3)
    return bf16_to_f32(f32_to_bf16(act_apply<0>(v, a))) + r;
  else
    return act_apply<MODE>(v + r, a);
}
// The epilogue mode of an activation code.
__host__ __device__ constexpr int act_mode(int act) { return act == kActGelu ? 1 : (act == kActLeaky ? 0 : 2); }
__device__ __forceinline__ float apply_act(float v, int act, float alpha) {
  return act == kActGelu ? gelu(v) : act_apply<false>(v, act_clamp_of(act, alpha));
}

// Unpacks 8 bf16 held in a uint4 into floats.
__device__ __forceinline__ void unpack8(const uint4& u, float* f) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}

__device__ __forceinline__ uint4 pack8(const float* f) {
  uint4 u;
  u.x = pack2_bf16(f[0], f[1]);
  u.y = pack2_bf16(f[2], f[3]);
  u.z = pack2_bf16(f[4], f[5]);
  u.w = pack2_bf16(f[6], f[7]);
  return u;
}

// Pulls every field of the conv parameters into scalar registers at once.
// Left alone, the compiler fetches kernel arguments lazily where they are
// first used, which costs several dependent memory round trips spread over
// the prologue of every workgroup.
__device__ __forceinline__ void materialize_args(const ConvParams& p) {
  asm volatile("" ::"s"(p.x), "s"(p.w), "s"(p.bias), "s"(p.res), "s"(p.y), "s"(p.partial));
  asm volatile("" ::"s"(p.N), "s"(p.H), "s"(p.W), "s"(p.Cp), "s"(p.P), "s"(p.Q), "s"(p.R), "s"(p.S),
               "s"(p.sh), "s"(p.sw), "s"(p.pt), "s"(p.pl));
  asm volatile("" ::"s"(p.M), "s"(p.Kp), "s"(p.Kg), "s"(p.Kgp), "s"(p.ldy), "s"(p.ldr), "s"(p.act), "s"(p.alpha),
               "s"(p.splits), "s"(p.k_tiles_per_split), "s"(p.x_bytes), "s"(p.w_bytes), "s"(p.res_bytes),
               "s"(p.res_post), "s"(p.xcd_py));
  asm volatile("" ::"s"(p.mg_pq), "s"(p.mg_q), "s"(p.mg_cp), "s"(p.mg_s), "s"(p.mg_tile), "s"(p.mg_wp),
               "s"(p.mg_hp));
}

// floor(n / d) for 0 <= n with n * d < 2^40, given mg = ceil(2^40 / d).
__device__ __forceinline__ int mdiv(int n, uint64_t mg) { return (int)(((uint64_t)(uint32_t)n * mg) >> 40); }

// Workgroup barrier that orders LDS accesses only: each wave waits for its
// own LDS operations, not for its outstanding global stores (the release
// fence of __syncthreads() would wait for those to be acknowledged).
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// rint(fl32(fl32(a) * m)), ties to even, saturated to +-2^20 (the float32
// rescaling of int8 graphs; a product followed by a rounding is never
// contracted).
__device__ __forceinline__ int rescale(int a, float m) {
  return (int)__builtin_amdgcn_fmed3f(__builtin_rintf((float)a * m), -1048576.0f, 1048576.0f);
}

// Leaky ReLU on an output code: the offset t = v - zy is kept when t >= 0,
// otherwise it becomes rint(fl32(t * slope)) (ties to even; |t| < 2^24, so
// the conversion to float32 is exact).
__device__ __forceinline__ int leaky_code(int v, int zy, float slope) {
  const int t = v - zy;
  return t < 0 ? zy + (int)rintf((float)t * slope) : v;
}

__device__ __forceinline__ int clip_i8(int v) { return min(max(v, -128), 127); }

inline int ceil_div(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

}  // namespace byoc
