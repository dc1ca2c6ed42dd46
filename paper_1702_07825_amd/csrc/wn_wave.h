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

__device__ __forceinline__ float expf_fast(float v) { return __builtin_amdgcn_exp2f(v * 1.4426950408889634f); }
__device__ __forceinline__ float tanh_f(float v) { return 1.0f - 2.0f * __builtin_amdgcn_rcpf(1.0f + expf_fast(2.0f * v)); }
__device__ __forceinline__ float sigmoid_f(float v) { return __builtin_amdgcn_rcpf(1.0f + expf_fast(-v)); }

// The approximate nonlinearities of the paper's Appendix C.  e~(x) = 1 + |x| + 0.5658 x^2 +
// 0.143 x^4 stands in for e^|x| in tanh(x) ~ sign(x) (e~ - 1/e~) / (e~ + 1/e~) and sigmoid(x) ~
// e~ / (1 + e~) (x >= 0) or 1 / (1 + e~) (x < 0); |x| is clamped to 1e9 so that e~ stays finite
// (the results there are +-1, 1 or 0 to fp32 either way).
__device__ __forceinline__ float e_tilde(float x) {
  const float c = fminf(fmaxf(x, -1e9f), 1e9f), a = fabsf(c), x2 = c * c;
  return 1.0f + a + x2 * (0.5658f + 0.143f * x2);
}
__device__ __forceinline__ float tanh_paper(float x) {
  const float e = e_tilde(x), r = __builtin_amdgcn_rcpf(e);
  return copysignf((e - r) * __builtin_amdgcn_rcpf(e + r), x);
}
__device__ __forceinline__ float sigmoid_paper(float x) {
  const float e = e_tilde(x), r = __builtin_amdgcn_rcpf(1.0f + e);
  return x >= 0.0f ? e * r : r;
}
// e^x for x <= 0 (the softmax's arguments) through the fp32 bit pattern of 2^y, y = x / ln 2:
// with z = y - floor(y) the pattern is (floor(y) + 126) 2^23 + (z + g(z)) 2^23, g the rational
// fit of 2^z - z, truncated to an integer (the integer part of the first term is exact, so fp32
// rounds only z + g); 0 where y <= -126.
__device__ __forceinline__ float exp_paper(float x) {
  const float y = x * 1.4426950408889634f;
  if (!(y > -126.0f)) return 0.0f;
  const float fl = floorf(y), z = y - fl;
  const float g = -4.7259162f + 27.7280233f * __builtin_amdgcn_rcpf(4.84252568f - z) - 1.49012907f * z;
  const unsigned bits = ((unsigned)((int)fl + 126) << 23) + (unsigned)((z + g) * 8388608.0f);
  return __uint_as_float(bits);
}
// h = tanh(ah) * sigmoid(ag) for a pair of lanes (2k, 2k + 1) that hold the same ah and ag: the
// even lane evaluates the tanh and the odd one the sigmoid, one exp2 and one reciprocal each (so a
// wave issues two quarter-rate transcendental instructions rather than four), and the two meet
// through a DPP swap; both lanes return h.  The formulas are tanh_f's and sigmoid_f's and the
// product is the same, so the result is bit for bit that of tanh_f(ah) * sigmoid_f(ag).
__device__ __forceinline__ float gate_pair(float ah, float ag, int lane) {
  const bool even = (lane & 1) == 0;
  const float r = __builtin_amdgcn_rcpf(1.0f + expf_fast(even ? 2.0f * ah : -ag));
  const float v = even ? 1.0f - 2.0f * r : r;
  const float o = dpp<0xB1>(v);
  return even ? v * o : o * v;
}
// Exact (AX = false) or approximate (AX = true) nonlinearities.
template <bool AX> __device__ __forceinline__ float tanh_nl(float v) { return AX ? tanh_paper(v) : tanh_f(v); }
template <bool AX> __device__ __forceinline__ float sigmoid_nl(float v) { return AX ? sigmoid_paper(v) : sigmoid_f(v); }
template <bool AX> __device__ __forceinline__ float exp_nl(float v) { return AX ? exp_paper(v) : expf_fast(v); }
template <bool AX> __device__ __forceinline__ float gate_nl(float ah, float ag, int lane) {
  if constexpr (AX) return tanh_paper(ah) * sigmoid_paper(ag);
  else return gate_pair(ah, ag, lane);
}

// Sum over the 64 lanes of a wave (every lane gets it).
__device__ __forceinline__ float wave_sum(float v) {
  v = gsum16(v);
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return (r0 + r1) + (r2 + r3);
}

// Order-preserving map of a (non-NaN) float to an unsigned key.
__device__ __forceinline__ unsigned float_key(float f) {
  const unsigned b = __float_as_uint(f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Rules for turning a step's output distribution P into a sample (Deep Voice, Appendix A.4,
// "Sampling from Output Distribution"); the values are those of wn_sample_mode_t.
enum { WN_DRAW_DIRECT = 0, WN_DRAW_TEMPERATURE = 1, WN_DRAW_TOPK = 2, WN_DRAW_MODE = 3, WN_DRAW_MEAN = 4 };

// #{k <= 254 : excl + s_i <= uz} over a wave, k = 4 lane + i: the inverse CDF at u with unnormalised
// prefix sums (excl the lane's exclusive prefix, s_i its own running sums) and uz = u Z, Z the total;
// counted by ballots.
__device__ __forceinline__ int cdf_count(float excl, const float (&s)[4], float uz) {
  return __popcll(__ballot(excl + s[0] <= uz)) + __popcll(__ballot(excl + s[1] <= uz)) +
         __popcll(__ballot(excl + s[2] <= uz)) + __popcll(__ballot(excl + s[3] <= uz) & 0x7fffffffffffffffull);
}

// One step's sample from the a = 256 logits held by one wave, lane l holding logits 4l .. 4l+3;
// every lane returns it.  P = softmax(logits).  Rules (mode is wave-uniform):
//   direct       y = #{k <= 254 : C_k <= u}, C_k = (p_0 + .. + p_k), the inverse CDF at u
//   temperature  the same on softmax(logits * inv_t), i.e. P^(1/t) / Z
//   top k        the same on P kept where its logit is at least the k-th largest logit (ties
//                kept) and renormalised; a result past the last kept class (only possible by
//                rounding) becomes that class
//   mode         the smallest index of the largest logit
//   mean         floor(sum_k k p_k + 1/2)
// The CDF rules compare the unnormalised prefix sums with u Z.  AX: e^x of the softmax by the
// approximation of Appendix C.
template <bool AX = false>
__device__ __forceinline__ int wave_draw(float4 lv, float u, int mode, float inv_t, int top_k, int lane) {
  float l[4] = {lv.x, lv.y, lv.z, lv.w};
  if (mode == WN_DRAW_MODE) {
    const float m = wave_max(fmaxf(fmaxf(l[0], l[1]), fmaxf(l[2], l[3])));
    int best = 256;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const unsigned long long mk = __ballot(l[i] == m);
      if (mk) best = min(best, 4 * (__ffsll((long long)mk) - 1) + i);
    }
    return best;
  }
  if (mode == WN_DRAW_TEMPERATURE) {
#pragma unroll
    for (int i = 0; i < 4; ++i) l[i] *= inv_t;
  }
  const float m = wave_max(fmaxf(fmaxf(l[0], l[1]), fmaxf(l[2], l[3])));
  float e[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) e[i] = exp_nl<AX>(l[i] - m);
  int last = 255;
  if (mode == WN_DRAW_TOPK) {
    // the k-th largest key, built bit by bit: the largest t with #{key >= t} >= k
    unsigned key[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) key[i] = float_key(l[i]);
    unsigned thr = 0;
    for (int bit = 31; bit >= 0; --bit) {
      const unsigned cand = thr | (1u << bit);
      int cnt = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) cnt += __popcll(__ballot(key[i] >= cand));
      if (cnt >= top_k) thr = cand;
    }
    last = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool keep = key[i] >= thr;
      e[i] = keep ? e[i] : 0.f;
      const unsigned long long mk = __ballot(keep);
      if (mk) last = max(last, 4 * (63 - __clzll((long long)mk)) + i);
    }
  }
  const float s[4] = {e[0], e[0] + e[1], e[0] + e[1] + e[2], e[0] + e[1] + e[2] + e[3]};
  const float incl = wave_incl_scan(s[3]);
  const float excl = wave_shr1(incl);
  const float Z = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, incl), 63));
  if (mode == WN_DRAW_MEAN) {
    const float k0 = (float)(4 * lane);
    const float part = k0 * e[0] + (k0 + 1.f) * e[1] + (k0 + 2.f) * e[2] + (k0 + 3.f) * e[3];
    const int y = (int)floorf(wave_sum(part) * (1.0f / Z) + 0.5f);
    return y < 0 ? 0 : (y > 255 ? 255 : y);
  }
  const int y = cdf_count(excl, s, u * Z);
  return y > last ? last : y;
}

// The direct rule (sc = 1) or the temperature rule (sc = 1 / t) for N streams of one wave at once,
// the same arithmetic as wave_draw's; straight-line code, so that the streams' cross-lane steps
// interleave.
template <bool AX, int N>
__device__ __forceinline__ void wave_draw_cdf(const float4 (&lv)[N], const float (&u)[N], float sc, int (&y)[N]) {
  float l[N][4], m[N], s[N][4], incl[N];
#pragma unroll
  for (int n = 0; n < N; ++n) {
    l[n][0] = lv[n].x * sc;
    l[n][1] = lv[n].y * sc;
    l[n][2] = lv[n].z * sc;
    l[n][3] = lv[n].w * sc;
    m[n] = fmaxf(fmaxf(l[n][0], l[n][1]), fmaxf(l[n][2], l[n][3]));
  }
#pragma unroll
  for (int n = 0; n < N; ++n) m[n] = wave_max(m[n]);
#pragma unroll
  for (int n = 0; n < N; ++n) {
    float e[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) e[i] = exp_nl<AX>(l[n][i] - m[n]);
    s[n][0] = e[0];
    s[n][1] = e[0] + e[1];
    s[n][2] = e[0] + e[1] + e[2];
    s[n][3] = e[0] + e[1] + e[2] + e[3];
  }
#pragma unroll
  for (int n = 0; n < N; ++n) incl[n] = wave_incl_scan(s[n][3]);
#pragma unroll
  for (int n = 0; n < N; ++n) {
    const float excl = wave_shr1(incl[n]);
    const float Z = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, incl[n]), 63));
    y[n] = cdf_count(excl, s[n], u[n] * Z);
  }
}

// True when the host has requested an abort (wn_abort): the word lives in pinned host memory, so
// the load is at system scope (it crosses PCIe and takes ~1-2 us).
__device__ __forceinline__ bool abort_requested(const int* flag) {
  return flag && __hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) != 0;
}
// LDS-only barrier: waits for this wave's LDS traffic, not for its global stores.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

}  // namespace wnk
