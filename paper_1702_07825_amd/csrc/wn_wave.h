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
