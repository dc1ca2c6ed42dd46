// Wave-level helpers shared by the gfx950 kernels: DPP reductions and scans over a
// 64-lane wavefront, fast transcendentals and an LDS-only barrier.
#pragma once
#include <hip/hip_runtime.h>

namespace wnk {

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xf, 0xf, false));
}
// Sums over aligned groups of 2, 4, 8, 16 lanes; every lane of a group gets the sum.
__device__ __forceinline__ float gsum2(float v) { return v + dpp<0xB1>(v); }                // quad_perm 1,0,3,2
__device__ __forceinline__ float gsum4(float v) { v = gsum2(v); return v + dpp<0x4E>(v); }  // quad_perm 2,3,0,1
__device__ __forceinline__ float gsum8(float v) { v = gsum4(v); return v + dpp<0x141>(v); } // row_half_mirror
__device__ __forceinline__ float gsum16(float v) { v = gsum8(v); return v + dpp<0x140>(v); } // row_mirror
template <int N>
__device__ __forceinline__ float gsum(float v) {
  if constexpr (N == 1) return v;
  else if constexpr (N == 2) return gsum2(v);
  else if constexpr (N == 4) return gsum4(v);
  else if constexpr (N == 8) return gsum8(v);
  else return gsum16(v);
}
// Transposed reductions over aligned 8-lane groups.  Each lane holds partial sums of several rows;
// a step pairs lane i with lane 7 - i (row_half_mirror) and each lane keeps half of the rows, adding
// its partner's partial of the rows it keeps, so the rows spread over the lanes instead of every
// lane summing every row.  `upper` is bit 2 of the lane index.
// Rows (a0, a1) and (b0, b1): the lower four lanes end with the sums of a0, a1 over their mirror
// pair, the upper four with b0, b1.
__device__ __forceinline__ void xsplit8_2(float a0, float a1, float b0, float b1, bool upper, float& k0, float& k1) {
  k0 = (upper ? b0 : a0) + dpp<0x141>(upper ? a0 : b0);
  k1 = (upper ? b1 : a1) + dpp<0x141>(upper ? a1 : b1);
}
// Rows a, b: the lower four lanes end with a, the upper four with b (over the mirror pair).
__device__ __forceinline__ float xsplit8_1(float a, float b, bool upper) {
  return (upper ? b : a) + dpp<0x141>(upper ? a : b);
}
// Full sums over the 8 lanes of N rows v[0..N-1] (N = 2 or 4): lane i ends with row
// (i >> 2 & 1) * N / 2 + (N == 4 ? (i >> 1 & 1) : 0); lanes differing only in the lowest bit
// (and, for N = 2, bit 1) hold the same row.
template <int N>
__device__ __forceinline__ float xreduce8(const float (&v)[N], int li) {
  const bool up = (li & 4) != 0;
  if constexpr (N == 2) {
    return gsum4(xsplit8_1(v[0], v[1], up));
  } else {
    static_assert(N == 4, "two or four rows");
    float k0, k1;
    xsplit8_2(v[0], v[1], v[2], v[3], up, k0, k1);
    const bool up2 = (li & 2) != 0;
    const float k = (up2 ? k1 : k0) + dpp<0x4E>(up2 ? k0 : k1);  // quad_perm 2,3,0,1
    return gsum2(k);
  }
}

// Inclusive prefix sum over the 64 lanes of a wave: row scans by row_shr, then row broadcasts.
__device__ __forceinline__ float wave_incl_scan(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x111, 0xf, 0xf, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x112, 0xf, 0xf, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x114, 0xf, 0xf, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x118, 0xf, 0xf, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x142, 0xa, 0xf, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x143, 0xc, 0xf, false));
  return v;
}
// The value of the previous lane (lane 0 gets 0).
__device__ __forceinline__ float wave_shr1(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x138, 0xf, 0xf, true));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp<0xB1>(v));
  v = fmaxf(v, dpp<0x4E>(v));
  v = fmaxf(v, dpp<0x141>(v));
  v = fmaxf(v, dpp<0x140>(v));
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}
__device__ __forceinline__ int wave_sum_int(int v) {
  float f = (float)v;  // counts are at most 255: exact in fp32
  f = gsum16(f);
  const int r0 = __builtin_amdgcn_readlane(__builtin_bit_cast(int, f), 0);
  const int r1 = __builtin_amdgcn_readlane(__builtin_bit_cast(int, f), 16);
  const int r2 = __builtin_amdgcn_readlane(__builtin_bit_cast(int, f), 32);
  const int r3 = __builtin_amdgcn_readlane(__builtin_bit_cast(int, f), 48);
  return (int)(__builtin_bit_cast(float, r0) + __builtin_bit_cast(float, r1) + __builtin_bit_cast(float, r2) +
               __builtin_bit_cast(float, r3));
}

__device__ __forceinline__ float expf_fast(float v) { return __builtin_amdgcn_exp2f(v * 1.4426950408889634f); }
__device__ __forceinline__ float tanh_f(float v) { return 1.0f - 2.0f * __builtin_amdgcn_rcpf(1.0f + expf_fast(2.0f * v)); }
__device__ __forceinline__ float sigmoid_f(float v) { return __builtin_amdgcn_rcpf(1.0f + expf_fast(-v)); }

// LDS-only barrier: waits for this wave's LDS traffic, not for its global stores.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

}  // namespace wnk
