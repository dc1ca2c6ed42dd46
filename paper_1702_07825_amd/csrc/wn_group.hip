// Batched generation kernel for bf16 weights on gfx950 MFMA (many independent streams).
//
// With many streams a step's layer becomes a real contraction: a = [W_prev | W_cur] [x_prev; x]
// is [2r x 2r] . [2r x B], and likewise W_res, W_skip and the two head layers (Deep Voice,
// arXiv 1702.07825, Appendix A.1).  One 512-thread workgroup owns a group of 16 streams (one
// MFMA N-tile) for the whole call and runs every layer of every step for them.  Per layer:
//
//   phase A  waves 0-3: gate.  Wave g computes the tanh rows 16g..16g+15 of a and the matching
//            sigmoid rows r+16g.., so h = tanh * sigmoid needs no exchange between waves.
//            wave 7: writes x_{j-1}[t] to the dilation history, moves the history and
//            conditioning rows of the next layer (loaded a layer earlier) into LDS and issues
//            the loads for the layer after that.  Only this wave touches HBM, so the in-order
//            completion counters of the weight-loading waves never wait on an HBM access.
//   phase B  waves 0-3: x += W_res h + B_res.   waves 4-6: q += W_skip h (q in MFMA accumulators).
//
// After the last layer: z_s = relu(q + B_skip), z_a = relu(W_relu z_s + B_relu), logits =
// W_out z_a + B_out (all 8 waves), then the softmax and draw (two streams per wave), which also
// lays out the next step's x0 = E[y] + B_embed.
//
// Weights are packed on the host into MFMA A-operand tiles (16 rows x 32 inputs of bf16, 1 KB,
// one 16-byte load per lane) and streamed from L2 every step; each wave issues the loads of the
// next layer's tiles before it waits for the current ones.  Activations stay fp32 in LDS; a B
// operand is split into bf16 hi + lo and both parts are multiplied, so a product keeps about 16
// bits of the activation (the weights are exactly bf16).  Accumulation is fp32.
#include "wn_internal.h"
#include "wn_wave.h"

#include <cstring>
#include <type_traits>

namespace {

using namespace wnk;

constexpr int NT = 512;
constexpr int G = 16;      // streams per workgroup (the MFMA N dimension)
constexpr int R = 64;      // residual channels
constexpr int A = WN_A;
constexpr int PX = R + 4;  // padded LDS rows
constexpr int PC = 2 * R + 4;
constexpr int PA = A + 4;
constexpr int PF = 12;     // 16-byte values each lane prefetches per layer

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ unsigned short bf16_bits(float v) {  // nearest even; activations are finite
  unsigned u = __float_as_uint(v);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (unsigned short)(u >> 16);
}
__device__ __forceinline__ float bf16_val(unsigned short b) { return __uint_as_float((unsigned)b << 16); }

// B operand of a 16x16x32 MFMA for one stream: 8 consecutive fp32 activations as hi = bf16(v)
// and lo = bf16(v - hi).
__device__ __forceinline__ void split8(const float* p, bf16x8& hi, bf16x8& lo) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const unsigned short h = bf16_bits(v[e]);
    hi[e] = __builtin_bit_cast(__bf16, h);
    lo[e] = __builtin_bit_cast(__bf16, bf16_bits(v[e] - bf16_val(h)));
  }
}
__device__ __forceinline__ f32x4 mfma2(uint4 w, const bf16x8& hi, const bf16x8& lo, f32x4 acc) {
  const bf16x8 a = __builtin_bit_cast(bf16x8, w);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, hi, acc, 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, lo, acc, 0, 0, 0);
}
__device__ __forceinline__ float4 as_f4(uint4 v) { return __builtin_bit_cast(float4, v); }

// Tile order of the packed weights, in 1 KB blocks (64 lanes x 16 bytes).
template <int S>
struct Pack {
  static constexpr int KTG = 2 * R / 32;  // gate inputs [x_prev | x]
  static constexpr int KTR = R / 32;
  static constexpr int KTH = S / 32;
  static constexpr int KTO = A / 32;
  static constexpr int GATE = 0;                              // [2R x 2R]: block mt * KTG + kt
  static constexpr int RES = GATE + (2 * R / 16) * KTG;       // [R x R]
  static constexpr int SKIP = RES + (R / 16) * KTR;           // [S x R]
  static constexpr int LAYER = SKIP + (S / 16) * KTR;         // blocks per layer
  static constexpr int NSKT = S / 16;                         // skip row tiles
  static constexpr int SKW = (NSKT + 2) / 3;                  // skip row tiles per skip wave
  static_assert(2 * KTG + KTR <= PF && SKW * KTR <= PF, "prefetch buffer too small");
};

template <int S>
constexpr size_t lds_floats(int L) {
  return (size_t)G * PX * 4 + (size_t)2 * G * PC + (size_t)G * (S + 4) + (size_t)2 * G * PA +
         (size_t)L * 3 * R + R + S + 2 * A + (size_t)A * R / 2;
}

template <int S, bool TF>
__global__ __launch_bounds__(NT) void wn_group_kernel(const WnGroupArgs g) {
  using P = Pack<S>;
  constexpr int PS = S + 4;
  const WnDims& D = g.d;
  const int L = D.L;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: tile addresses go to SGPRs
  const int b0 = blockIdx.x * G;
  const int T = g.io.T, B = g.io.B;
  const int n = lane & 15, quad = lane >> 4;  // MFMA column (stream) and row quad of this lane

  extern __shared__ __align__(16) float sm[];
  float* X = sm;                  // [G][PX]  x_{j-1}, updated in place
  float* H = X + G * PX;          // [G][PX]  h_j
  float* XP = H + G * PX;         // [2][G][PX] history rows x_{j-1}[t - d_j] (position parity)
  float* CD = XP + 2 * G * PX;    // [2][G][PC] conditioning rows
  float* ZS = CD + 2 * G * PC;    // [G][PS]  relu(q + B_skip)
  float* ZA = ZS + G * PS;        // [G][PA]
  float* LG = ZA + G * PA;        // [G][PA]  logits
  float* BG = LG + G * PA;        // [L][2R]
  float* BR = BG + L * 2 * R;     // [L][R]
  float* BE = BR + L * R;         // [R]
  float* BS = BE + R;             // [S]
  float* BRL = BS + S;            // [A]
  float* BO = BRL + A;            // [A]
  unsigned short* EMB = reinterpret_cast<unsigned short*>(BO + A);  // [A][R] bf16
  __shared__ int s_y[G];
  __shared__ float s_u[G];
  __shared__ int s_yin[G];

  const uint4* pk = static_cast<const uint4*>(g.packed);
  int64_t tg0 = 0;
  {
    // every stream of a call has taken the same number of steps
    const int64_t* st = g.ws.state;
    if (!g.io.reset) tg0 = st[2 * (size_t)b0];
    if (tid < G) {
      int y = g.io.init_sample;
      if (!g.io.reset && b0 + tid < B) y = (int)st[2 * (size_t)(b0 + tid) + 1];
      s_y[tid] = y < 0 ? 0 : (y > A - 1 ? A - 1 : y);
    }
  }
  for (int i = tid; i < L * 2 * R; i += NT) BG[i] = g.w.b_gate[i];
  for (int i = tid; i < L * R; i += NT) BR[i] = g.w.b_res[i];
  for (int i = tid; i < R; i += NT) BE[i] = g.w.b_embed[i];
  for (int i = tid; i < S; i += NT) BS[i] = g.w.b_skip[i];
  for (int i = tid; i < A; i += NT) BRL[i] = g.w.b_relu[i];
  for (int i = tid; i < A; i += NT) BO[i] = g.w.b_out[i];
  {
    const unsigned short* E = static_cast<const unsigned short*>(g.w.embed);
    for (int i = tid; i < A * R; i += NT) EMB[i] = E[i];
  }
  if (g.io.reset) {
    for (int nn = 0; nn < G && b0 + nn < B; ++nn) {
      float4* hist = reinterpret_cast<float4*>(g.ws.hist + (size_t)(b0 + nn) * D.hist_len);
      for (int i = tid; i < D.hist_len / 4; i += NT) hist[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    if (blockIdx.x == 0 && tid == 0) *g.ws.status = 0;
  }
  __syncthreads();  // also orders the history zeroing before the loader's reads
  for (int i = tid; i < G * R; i += NT) {
    const int nn = i / R, c = i % R;
    X[nn * PX + c] = bf16_val(EMB[s_y[nn] * R + c]) + BE[c];
  }

  const int64_t nq = (int64_t)T * L;  // positions (step, layer) of this call

  // Runs every position (step, layer) of the call; positions alternate between two prefetch
  // buffers, passed to the body as a compile-time parity.  The loop leaves right after the
  // position that used a buffer or goes on to the one that refills it.
  auto run = [&](auto&& body) __attribute__((always_inline)) {
    int64_t tl = 0;
    int j = 0;
    for (int64_t q = 0;;) {
      body(std::integral_constant<int, 0>{}, q, tl, j);
      if (++j == L) j = 0, ++tl;
      if (++q == nq) break;
      body(std::integral_constant<int, 1>{}, q, tl, j);
      if (++j == L) j = 0, ++tl;
      if (++q == nq) break;
    }
  };

  // After the last layer of step tl: the head (every wave: row tiles 2w and 2w + 1 of W_relu,
  // then of W_out), the draw (streams 2w and 2w + 1) and the next step's x0.  Three barriers.
  // Results stay in LDS (logits in LG, samples in s_y); the loader wave writes them out.
  auto head_and_draw = [&](int64_t tl) __attribute__((always_inline)) {
    {
      const uint4* hw = pk + (size_t)L * P::LAYER * 64 + lane;
      uint4 w[2 * P::KTH];
#pragma unroll
      for (int k = 0; k < 2; ++k)
#pragma unroll
        for (int kt = 0; kt < P::KTH; ++kt) w[k * P::KTH + kt] = hw[((2 * wave + k) * P::KTH + kt) * 64];
      f32x4 acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
      for (int kt = 0; kt < P::KTH; ++kt) {
        bf16x8 hi, lo;
        split8(ZS + n * PS + kt * 32 + quad * 8, hi, lo);
        acc[0] = mfma2(w[kt], hi, lo, acc[0]);
        acc[1] = mfma2(w[P::KTH + kt], hi, lo, acc[1]);
      }
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int m0 = (2 * wave + k) * 16 + quad * 4;
        const float4 b = *reinterpret_cast<const float4*>(BRL + m0);
        *reinterpret_cast<float4*>(ZA + n * PA + m0) =
            make_float4(fmaxf(acc[k][0] + b.x, 0.f), fmaxf(acc[k][1] + b.y, 0.f), fmaxf(acc[k][2] + b.z, 0.f),
                        fmaxf(acc[k][3] + b.w, 0.f));
      }
    }
    lds_barrier();
    {
      const uint4* ow = pk + ((size_t)L * P::LAYER + (A / 16) * P::KTH) * 64 + lane;
      uint4 w[2 * P::KTO];
#pragma unroll
      for (int k = 0; k < 2; ++k)
#pragma unroll
        for (int kt = 0; kt < P::KTO; ++kt) w[k * P::KTO + kt] = ow[((2 * wave + k) * P::KTO + kt) * 64];
      f32x4 acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
      for (int kt = 0; kt < P::KTO; ++kt) {
        bf16x8 hi, lo;
        split8(ZA + n * PA + kt * 32 + quad * 8, hi, lo);
        acc[0] = mfma2(w[kt], hi, lo, acc[0]);
        acc[1] = mfma2(w[P::KTO + kt], hi, lo, acc[1]);
      }
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int m0 = (2 * wave + k) * 16 + quad * 4;
        const float4 b = *reinterpret_cast<const float4*>(BO + m0);
        const float4 lv = make_float4(acc[k][0] + b.x, acc[k][1] + b.y, acc[k][2] + b.z, acc[k][3] + b.w);
        *reinterpret_cast<float4*>(LG + n * PA + m0) = lv;
      }
    }
    lds_barrier();
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int nn = 2 * wave + k;
      int y;
      if constexpr (TF) {
        y = s_yin[nn];
      } else {
        const float4 lv = *reinterpret_cast<const float4*>(LG + nn * PA + 4 * lane);
        const float m = wave_max(fmaxf(fmaxf(lv.x, lv.y), fmaxf(lv.z, lv.w)));
        const float e0 = expf_fast(lv.x - m), e1 = expf_fast(lv.y - m), e2 = expf_fast(lv.z - m),
                    e3 = expf_fast(lv.w - m);
        const float s0 = e0, s1 = s0 + e1, s2 = s1 + e2, s3 = s2 + e3;
        const float incl = wave_incl_scan(s3);
        const float excl = wave_shr1(incl);
        const float Z = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, incl), 63));
        const float iz = 1.0f / Z;
        const float u = s_u[nn];
        int cnt = ((excl + s0) * iz <= u) + ((excl + s1) * iz <= u) + ((excl + s2) * iz <= u);
        if (lane != 63) cnt += ((excl + s3) * iz <= u);
        y = wave_sum_int(cnt);
      }
      if (lane == 0) s_y[nn] = y;
      X[nn * PX + lane] = bf16_val(EMB[y * R + lane]) + BE[lane];
    }
    lds_barrier();
  };

  // Each role runs its own copy of the position loop, so the completion counters of its loads
  // are tracked exactly; all roles meet at the same barriers.
  if (wave < 4) {
    // ---------------- gate and residual: row tile gi of W_res, gi and gi + 4 of [W_prev | W_cur] ----------------
    constexpr int NB = 2 * P::KTG + P::KTR;
    const int gi = wave;
    auto issue = [&](uint4 (&buf)[NB], int j) __attribute__((always_inline)) {
      const uint4* lw = pk + (size_t)j * P::LAYER * 64 + lane;
#pragma unroll
      for (int kt = 0; kt < P::KTG; ++kt) {
        buf[kt] = lw[(P::GATE + gi * P::KTG + kt) * 64];
        buf[P::KTG + kt] = lw[(P::GATE + (gi + R / 16) * P::KTG + kt) * 64];
      }
      if (j != L - 1) {  // the last layer's x feeds nothing
#pragma unroll
        for (int kt = 0; kt < P::KTR; ++kt) buf[2 * P::KTG + kt] = lw[(P::RES + gi * P::KTR + kt) * 64];
      }
    };
    uint4 bufA[NB], bufB[NB];
    issue(bufA, 0);
    __syncthreads();
    run([&](auto parity, int64_t q, int64_t tl, int j) __attribute__((always_inline)) {
      uint4(&cur)[NB] = decltype(parity)::value == 0 ? bufA : bufB;
      uint4(&nxt)[NB] = decltype(parity)::value == 0 ? bufB : bufA;
      const int slot = (int)(q & 1);
      issue(nxt, j + 1 == L ? 0 : j + 1);
      f32x4 at = {0.f, 0.f, 0.f, 0.f}, as = {0.f, 0.f, 0.f, 0.f};
      const float* xp = XP + slot * G * PX + n * PX;
      const float* xc = X + n * PX;
#pragma unroll
      for (int kt = 0; kt < P::KTG; ++kt) {
        // inputs 0..R-1: the history row x_{j-1}[t - d_j]; R..2R-1: the current x_{j-1}[t]
        const float* src = (kt < R / 32) ? xp + kt * 32 + quad * 8 : xc + (kt - R / 32) * 32 + quad * 8;
        bf16x8 hi, lo;
        split8(src, hi, lo);
        at = mfma2(cur[kt], hi, lo, at);
        as = mfma2(cur[P::KTG + kt], hi, lo, as);
      }
      const float* cd = CD + slot * G * PC + n * PC;
      const int m0 = gi * 16 + quad * 4;
      const float4 ch = *reinterpret_cast<const float4*>(cd + m0);
      const float4 cg = *reinterpret_cast<const float4*>(cd + R + m0);
      const float4 bh = *reinterpret_cast<const float4*>(BG + j * 2 * R + m0);
      const float4 bg = *reinterpret_cast<const float4*>(BG + j * 2 * R + R + m0);
      float4 hv;
      hv.x = tanh_f(at[0] + bh.x + ch.x) * sigmoid_f(as[0] + bg.x + cg.x);
      hv.y = tanh_f(at[1] + bh.y + ch.y) * sigmoid_f(as[1] + bg.y + cg.y);
      hv.z = tanh_f(at[2] + bh.z + ch.z) * sigmoid_f(as[2] + bg.z + cg.z);
      hv.w = tanh_f(at[3] + bh.w + ch.w) * sigmoid_f(as[3] + bg.w + cg.w);
      *reinterpret_cast<float4*>(H + n * PX + m0) = hv;
      lds_barrier();
      if (j < L - 1) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kt = 0; kt < P::KTR; ++kt) {
          bf16x8 hi, lo;
          split8(H + n * PX + kt * 32 + quad * 8, hi, lo);
          acc = mfma2(cur[2 * P::KTG + kt], hi, lo, acc);
        }
        float4 xv = *reinterpret_cast<const float4*>(X + n * PX + m0);
        const float4 br = *reinterpret_cast<const float4*>(BR + j * R + m0);
        xv.x += acc[0] + br.x;
        xv.y += acc[1] + br.y;
        xv.z += acc[2] + br.z;
        xv.w += acc[3] + br.w;
        *reinterpret_cast<float4*>(X + n * PX + m0) = xv;
      }
      lds_barrier();
      if (j == L - 1) head_and_draw(tl);
    });
  } else if (wave < 7) {
    // ---------------- skip: row tiles sk0 .. sk0 + nsk - 1 of W_skip ----------------
    constexpr int NB = P::SKW * P::KTR;
    const int sk0 = (wave - 4) * P::SKW;
    const int nsk = min(P::SKW, P::NSKT - sk0);
    auto issue = [&](uint4 (&buf)[NB], int j) __attribute__((always_inline)) {
      const uint4* lw = pk + (size_t)j * P::LAYER * 64 + lane;
#pragma unroll
      for (int k = 0; k < P::SKW; ++k)
        if (k < nsk) {
#pragma unroll
          for (int kt = 0; kt < P::KTR; ++kt) buf[k * P::KTR + kt] = lw[(P::SKIP + (sk0 + k) * P::KTR + kt) * 64];
        }
    };
    uint4 bufA[NB], bufB[NB];
    f32x4 qacc[P::SKW];
    issue(bufA, 0);
    __syncthreads();
    run([&](auto parity, int64_t q, int64_t tl, int j) __attribute__((always_inline)) {
      uint4(&cur)[NB] = decltype(parity)::value == 0 ? bufA : bufB;
      uint4(&nxt)[NB] = decltype(parity)::value == 0 ? bufB : bufA;
      issue(nxt, j + 1 == L ? 0 : j + 1);
      lds_barrier();
      bf16x8 hi[P::KTR], lo[P::KTR];
#pragma unroll
      for (int kt = 0; kt < P::KTR; ++kt) split8(H + n * PX + kt * 32 + quad * 8, hi[kt], lo[kt]);
      // the first layer starts the sum, so q holds nothing between the head and the next step
      const bool first = j == 0;
#pragma unroll
      for (int k = 0; k < P::SKW; ++k) {
        if (k < nsk) {
          f32x4 acc = first ? f32x4{0.f, 0.f, 0.f, 0.f} : qacc[k];
#pragma unroll
          for (int kt = 0; kt < P::KTR; ++kt) acc = mfma2(cur[k * P::KTR + kt], hi[kt], lo[kt], acc);
          qacc[k] = acc;
        }
      }
      if (j == L - 1) {
#pragma unroll
        for (int k = 0; k < P::SKW; ++k) {
          if (k < nsk) {
            const int m0 = (sk0 + k) * 16 + quad * 4;
            const float4 bs = *reinterpret_cast<const float4*>(BS + m0);
            const float4 z = make_float4(fmaxf(qacc[k][0] + bs.x, 0.f), fmaxf(qacc[k][1] + bs.y, 0.f),
                                         fmaxf(qacc[k][2] + bs.z, 0.f), fmaxf(qacc[k][3] + bs.w, 0.f));
            *reinterpret_cast<float4*>(ZS + n * PS + m0) = z;
          }
        }
      }
      lds_barrier();
      if (j == L - 1) head_and_draw(tl);
    });
  } else {
    // ---------------- loader: lane = stream ldn, quarter ldq of a row ----------------
    constexpr int NB = 12;  // 4 x 16 B of the history row, 8 x 16 B of the conditioning row
    const int ldn = lane >> 2, ldq = lane & 3;
    const int ldb = min(b0 + ldn, B - 1);  // reads of a partial group are clamped
    const int lub = min(b0 + lane, B - 1);
    // history row x_{j-1}[ts - d_j] and conditioning row of position q for stream ldn
    auto issue = [&](uint4 (&buf)[NB], int64_t q) __attribute__((always_inline)) {
      if (q >= nq) return;
      const int64_t tl = q / L;
      const int j = (int)(q - tl * L);
      const int64_t ts = tg0 + tl;
      const int d = D.dil[j];
      const uint4* hist = reinterpret_cast<const uint4*>(g.ws.hist + (size_t)ldb * D.hist_len + D.hoff[j] +
                                                         (size_t)(ts % d) * R + ldq * 16);
#pragma unroll
      for (int k = 0; k < 4; ++k) buf[k] = hist[k];
      const uint4* c =
          reinterpret_cast<const uint4*>(g.io.cond + (((size_t)ldb * T + tl) * L + j) * 2 * R + ldq * 32);
#pragma unroll
      for (int k = 0; k < 8; ++k) buf[4 + k] = c[k];
    };
    auto store = [&](int slot, const uint4 (&buf)[NB]) __attribute__((always_inline)) {
      float* xp = XP + slot * G * PX + ldn * PX + ldq * 16;
#pragma unroll
      for (int k = 0; k < 4; ++k) reinterpret_cast<float4*>(xp)[k] = as_f4(buf[k]);
      float* cd = CD + slot * G * PC + ldn * PC + ldq * 32;
#pragma unroll
      for (int k = 0; k < 8; ++k) reinterpret_cast<float4*>(cd)[k] = as_f4(buf[4 + k]);
    };
    // Samples (generation) or logits (teacher forcing) of step tl, from s_y / LG, for the 16 streams.
    auto write_outputs = [&](int64_t tl) __attribute__((always_inline)) {
      if constexpr (TF) {
#pragma unroll
        for (int c = 0; c < G; c += 4) {
          f32x4 v[4];
#pragma unroll
          for (int k = 0; k < 4; ++k) v[k] = *reinterpret_cast<const f32x4*>(LG + (c + k) * PA + 4 * lane);
          asm volatile("" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]));
#pragma unroll
          for (int k = 0; k < 4; ++k)
            if (b0 + c + k < B) reinterpret_cast<f32x4*>(g.io.logits + ((size_t)(b0 + c + k) * T + tl) * A)[lane] = v[k];
        }
      } else {
        if (lane < G && b0 + lane < B) g.io.y_out[(size_t)(b0 + lane) * T + tl] = s_y[lane];
      }
    };
    uint4 bufA[NB], bufB[NB];
    float pre_u = 0.f;
    int pre_y = 0;
    issue(bufB, 0);
    store(0, bufB);
    issue(bufA, 1);
    __syncthreads();
    run([&](auto parity, int64_t q, int64_t tl, int j) __attribute__((always_inline)) {
      uint4(&cur)[NB] = decltype(parity)::value == 0 ? bufA : bufB;
      uint4(&nxt)[NB] = decltype(parity)::value == 0 ? bufB : bufA;
      const int64_t t = tg0 + tl;
      // On gfx950 a wait for a load while stores are outstanding also waits for the stores, so
      // this wave first consumes what it loaded a layer ago, then stores, then issues its loads:
      // the next layer's wait then covers only stores that were issued before the loads it needs.
      if (q + 1 < nq) store((int)((q + 1) & 1), cur);
      // this step's uniform (or teacher sample): read at the first layer, staged at the second
      if (j == 1 && lane < G) {
        if constexpr (TF) s_yin[lane] = pre_y < 0 ? 0 : (pre_y > A - 1 ? A - 1 : pre_y);
        else s_u[lane] = pre_u;
      }
      // x_{j-1}[t] into slot t mod d_j of layer j's history; it is read again at step t + d_j
      // (by a load issued below when d_j l = 2).  All four values are read before the first
      // store so that each store has registers of its own.
      {
        const size_t so = D.hoff[j] + (size_t)(t % D.dil[j]) * R;
        static_assert(G * R / 4 / 64 == 4, "four history values per loader lane");
        f32x4 v[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int i = lane + 64 * k;
          v[k] = *reinterpret_cast<const f32x4*>(X + (i / (R / 4)) * PX + (i % (R / 4)) * 4);
        }
        asm volatile("" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]));
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int i = lane + 64 * k;
          const int nn = i / (R / 4), c4 = i % (R / 4);
          if (b0 + nn < B) reinterpret_cast<f32x4*>(g.ws.hist + (size_t)(b0 + nn) * D.hist_len + so)[c4] = v[k];
        }
      }
      // outputs of the previous step, left in LDS by its head and draw
      if (j == 0 && tl > 0) write_outputs(tl - 1);
      if (j == 0 && lane < G) {
        if constexpr (TF) pre_y = g.io.y_in[(size_t)lub * T + tl];
        else pre_u = g.io.u[(size_t)lub * T + tl];
      }
      issue(nxt, q + 2);
      lds_barrier();
      lds_barrier();
      if (j == L - 1) head_and_draw(tl);
    });
    write_outputs(T - 1);  // the last step's, after its draw
  }
  __syncthreads();
  if (tid < G && b0 + tid < B) {
    int64_t* st = g.ws.state + 2 * (size_t)(b0 + tid);
    st[0] = tg0 + T;
    st[1] = s_y[tid];
  }
}

template <int S>
hipError_t launch_group_s(const WnGroupArgs& g, bool teacher, hipStream_t stream) {
  const size_t dyn = lds_floats<S>(g.d.L) * sizeof(float);
  const dim3 grid((g.io.B + G - 1) / G), block(NT);
  const void* k = teacher ? reinterpret_cast<const void*>(wn_group_kernel<S, true>)
                          : reinterpret_cast<const void*>(wn_group_kernel<S, false>);
  hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
  if (e != hipSuccess) return e;
  if (teacher) hipLaunchKernelGGL((wn_group_kernel<S, true>), grid, block, dyn, stream, g);
  else hipLaunchKernelGGL((wn_group_kernel<S, false>), grid, block, dyn, stream, g);
  return hipGetLastError();
}

// Append W [M][K] (element (m, k) from `at`) as MFMA A tiles: block (mt, kt) holds, for lane i,
// W[16 mt + i % 16][32 kt + 8 (i / 16) + e], e = 0..7.
template <class F>
void pack_tiles(std::vector<uint16_t>& out, int M, int K, F at) {
  for (int mt = 0; mt < M / 16; ++mt)
    for (int kt = 0; kt < K / 32; ++kt)
      for (int i = 0; i < 64; ++i)
        for (int e = 0; e < 8; ++e) out.push_back(wn_to_bf16(at(mt * 16 + i % 16, kt * 32 + 8 * (i / 16) + e)));
}

}  // namespace

bool wn_group_supported(int R_, int S_, int L) {
  return R_ == R && (S_ == 256 || S_ == 128) && L >= 2 && L <= WN_GROUP_MAX_LAYERS;
}

size_t wn_group_lds_bytes(int L, int S_) {
  return (S_ == 256 ? lds_floats<256>(L) : lds_floats<128>(L)) * sizeof(float);
}

std::vector<uint16_t> wn_group_pack(int L, int R_, int S_, const float* w_prev, const float* w_cur,
                                    const float* w_res, const float* w_skip, const float* w_relu,
                                    const float* w_out) {
  std::vector<uint16_t> out;
  if (R_ != R) return out;
  out.reserve((size_t)L * (2 * R * 2 * R + R * R + S_ * R) + (size_t)A * S_ + (size_t)A * A);
  for (int j = 0; j < L; ++j) {
    const float* wp = w_prev + (size_t)j * 2 * R * R;
    const float* wc = w_cur + (size_t)j * 2 * R * R;
    pack_tiles(out, 2 * R, 2 * R, [&](int m, int k) { return k < R ? wp[m * R + k] : wc[m * R + (k - R)]; });
    const float* wr = w_res + (size_t)j * R * R;
    pack_tiles(out, R, R, [&](int m, int k) { return wr[m * R + k]; });
    const float* wk = w_skip + (size_t)j * S_ * R;
    pack_tiles(out, S_, R, [&](int m, int k) { return wk[m * R + k]; });
  }
  pack_tiles(out, A, S_, [&](int m, int k) { return w_relu[m * S_ + k]; });
  pack_tiles(out, A, A, [&](int m, int k) { return w_out[m * A + k]; });
  return out;
}

hipError_t wn_group_launch(const WnGroupArgs& g, bool teacher, hipStream_t stream) {
  if (g.d.S == 256) return launch_group_s<256>(g, teacher, stream);
  if (g.d.S == 128) return launch_group_s<128>(g, teacher, stream);
  return hipErrorInvalidValue;
}
