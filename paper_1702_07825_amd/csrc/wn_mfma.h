// bf16 helpers for the MFMA kernels (gfx950): an fp32 activation that enters a product is kept as
// a pair of bf16 values, hi = bf16(v) and lo = bf16(v - hi), and both parts are multiplied, so the
// product sees about 16 bits of the activation.  A "split row" of K values is K hi parts followed by
// K lo parts.
#pragma once
#include <hip/hip_runtime.h>

namespace wnk {

typedef unsigned short u16;
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// bf16 of a and b (nearest even; v_cvt_pk_bf16_f32), a in the low half
__device__ __forceinline__ unsigned pack_bf16(float a, float b) {
  const bf16x2 h = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(unsigned, h);
}
__device__ __forceinline__ float low_bf16(unsigned p) { return __uint_as_float(p << 16); }
__device__ __forceinline__ float high_bf16(unsigned p) { return __uint_as_float(p & 0xffff0000u); }
__device__ __forceinline__ float bf16_val(u16 b) { return __uint_as_float((unsigned)b << 16); }
// hi / lo parts of four consecutive values
__device__ __forceinline__ void split4(float4 v, uint2& hi, uint2& lo) {
  const unsigned h01 = pack_bf16(v.x, v.y), h23 = pack_bf16(v.z, v.w);
  hi = make_uint2(h01, h23);
  lo = make_uint2(pack_bf16(v.x - low_bf16(h01), v.y - high_bf16(h01)),
                  pack_bf16(v.z - low_bf16(h23), v.w - high_bf16(h23)));
}
// hi / lo parts of one value, as 16-bit patterns
__device__ __forceinline__ void split1(float v, u16& hi, u16& lo) {
  const unsigned p = pack_bf16(v, 0.f);
  hi = (u16)p;
  lo = (u16)pack_bf16(v - low_bf16(p), 0.f);
}
// hi / lo parts of four rows m0..m0+3 into a split row of K values
template <int K>
__device__ __forceinline__ void store_split4(u16* row, int m0, float4 v) {
  uint2 hi, lo;
  split4(v, hi, lo);
  *reinterpret_cast<uint2*>(row + m0) = hi;
  *reinterpret_cast<uint2*>(row + K + m0) = lo;
}
// Product of a weight tile with the B operand taken from a split row: inputs k0 .. k0 + 7 of
// this lane's stream, hi and lo parts.
template <int K>
__device__ __forceinline__ f32x4 mfma_row(u32x4 w, const u16* row, int k0, f32x4 acc) {
  const bf16x8 a = __builtin_bit_cast(bf16x8, w);
  const bf16x8 hi = *reinterpret_cast<const bf16x8*>(row + k0);
  const bf16x8 lo = *reinterpret_cast<const bf16x8*>(row + K + k0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, hi, acc, 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, lo, acc, 0, 0, 0);
}

}  // namespace wnk
