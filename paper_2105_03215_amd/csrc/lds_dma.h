// Helpers of the MFMA conv kernels that stream operands from HBM straight
// into LDS: operand vector types, raw buffer descriptors, the 16-byte
// buffer-to-LDS load, compile-time loops and the XCD-aware tile placement.
#pragma once

#include <type_traits>

#include "device_common.h"

namespace byoc {
namespace dma {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) int i32x4;

constexpr int kLdsLimit = 160 * 1024;  // LDS bytes per workgroup on gfx950

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

// Raw buffer resource (base, stride 0, num_records = bytes): offsets at or
// past `bytes` read zeros.
__device__ __forceinline__ i32x4 buffer_rsrc(const void* base, int bytes) {
  const uint64_t a = (uint64_t)base;
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r[1] = __builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32) & 0xFFFF);
  r[2] = __builtin_amdgcn_readfirstlane(bytes);
  r[3] = kBufferFlags;
  return r;
}

// 16 bytes per lane from a buffer straight into LDS: lane l writes bytes
// [16 l, 16 l + 16) after the wave-uniform LDS address.  Written as inline
// assembly so that the compiler neither tracks these fills (the kernels
// wait for them themselves, per stage, before their barrier) nor inserts
// conservative waits for them in front of unrelated LDS reads.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_fill16(i32x4 rsrc, uint32_t lds_addr, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds_addr), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}
#pragma clang diagnostic pop

__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)p; }

// f(integral_constant<int, i>) for i = I .. N-1, unrolled at compile time.
template <int I, int N, class F>
__host__ __device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

// Tile placement: the hardware deals workgroups round-robin to the 8 XCDs
// (block b runs on XCD b % 8).  With xcd_py > 0 every XCD owns one block of
// a (8 / xcd_py) x xcd_py partition of the tile grid and walks it channel
// tile fastest; the grid is padded to 8 equal shares and surplus workgroups
// get false (they exit at once).  Otherwise each XCD gets a contiguous run
// of the row-major tile order.  mg_tile divides by the channel tiles of one
// block (xcd_py > 0) or of the whole grid.
template <int BM, int BN>
__device__ __forceinline__ bool place_tile(const ConvParams& p, int* tm, int* tn) {
  const int ntn = (p.Kp + BN - 1) / BN;
  const int ntm = (p.M + BM - 1) / BM;
  if (p.xcd_py > 0) {
    // XCD x = (gx, gy) owns m tiles [gx*mh, gx*mh + mh) and n tiles
    // [gy*nh, gy*nh + nh) of the grid (clipped at its edge)
    const int x = blockIdx.x & 7, j = blockIdx.x >> 3;
    const int lpy = 31 - __builtin_clz(p.xcd_py);  // xcd_py is 1, 2, 4 or 8
    const int mh = (ntm + (8 >> lpy) - 1) >> (3 - lpy), nh = (ntn + p.xcd_py - 1) >> lpy;
    const int gx = x >> lpy, gy = x & (p.xcd_py - 1);
    const int jm = mdiv(j, p.mg_tile);
    *tm = gx * mh + jm;
    *tn = gy * nh + (j - jm * nh);
    return jm < mh && *tm < ntm && *tn < ntn;
  }
  int bid = blockIdx.x;
  const int nb = ntm * ntn;  // the launch grid (no kernel-argument fetch)
  if ((nb & 7) == 0) bid = (bid & 7) * (nb >> 3) + (bid >> 3);
  *tm = mdiv(bid, p.mg_tile);
  *tn = bid - *tm * ntn;
  return true;
}

// Workgroups of a launch with the placement above, and the tile divisor.
inline int placed_blocks(ConvParams& p, int bm, int bn) {
  const int ntm = (p.M + bm - 1) / bm;
  const int ntn = (p.Kp + bn - 1) / bn;
  if (p.xcd_py > 0) {
    const int py = p.xcd_py, px = 8 / py;
    const int mh = (ntm + px - 1) / px, nh = (ntn + py - 1) / py;
    p.mg_tile = magic40(nh);
    return 8 * mh * nh;
  }
  p.mg_tile = magic40(ntn);
  return ntm * ntn;
}

}  // namespace dma
}  // namespace byoc
