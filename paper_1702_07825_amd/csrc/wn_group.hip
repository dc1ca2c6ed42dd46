// Batched generation kernel for bf16 weights on gfx950 MFMA (many independent streams).
//
// With many streams a step's layer becomes a real contraction: a = [W_prev | W_cur] [x_prev; x]
// is [2r x 2r] . [2r x B], and likewise W_res, W_skip and the two head layers (Deep Voice,
// arXiv 1702.07825, Appendix A.1).  One 512-thread workgroup owns a group of 8 streams (16 when
// a call has more than 2048) for the whole call and runs every layer of every step for them; the
// group fills the 16 columns of an MFMA N-tile (with 8 streams, each stream's hi and lo parts
// side by side, see mfma_split).  Per layer:
//
//   phase A  waves 0-3: gate.  Wave g computes the tanh rows 16g..16g+15 of a and the matching
//            sigmoid rows r+16g.., so h = tanh * sigmoid needs no exchange between waves.
//            wave 7: moves the history and conditioning rows of the next layer (loaded a layer
//            earlier) into LDS, writes x_{j-1}[t] to the dilation history and issues the loads
//            for the layer after that.  Only this wave touches HBM, and it alone stores to
//            global memory, so the weight-loading waves never wait on an HBM access or a store.
//   phase B  waves 0-3: x += W_res h + B_res (each lane keeps its four rows of x in registers).
//            waves 4-6: q += W_skip h (q in MFMA accumulators).
//
// After the last layer: z_s = relu(q + B_skip), z_a = relu(W_relu z_s + B_relu), logits =
// W_out z_a + B_out (all 8 waves; the head's tiles are loaded during the last layer), then the
// softmax and draw (two streams per wave), which also lays out the next step's x0 = E[y] +
// B_embed (+ E_prev[y_{t-1}] with the two-tap input convolution of Section 5.1: the loader reads
// that row during the step, since the sample it embeds is known a step ahead).
//
// Weights are packed on the host into MFMA A-operand tiles (16 rows x 32 inputs of bf16, 1 KB,
// one 16-byte load per lane) and streamed from L2 every step; each wave issues the loads of the
// next layer's tiles before it waits for the current ones.  An activation that feeds a product
// is kept as a pair of bf16 values, hi = bf16(v) and lo = bf16(v - hi), and both parts are
// multiplied, so a product sees about 16 bits of the activation (the weights are exactly bf16);
// accumulation, the gate, the residual sum and the softmax are fp32.  Activation rows in LDS
// and the dilation histories in the workspace hold the pairs: a row of K values is K hi parts
// followed by K lo parts.
#include "wn_internal.h"
#include "wn_mfma.h"
#include "wn_wave.h"

#include "wn.h"

#include <cstdlib>
#include <cstring>
#include <type_traits>

namespace {

using namespace wnk;

constexpr int NT = 512;
constexpr int G = 16;  // MFMA N dimension: columns of a workgroup's products (g.gs <= G of them are streams)
constexpr int R = 64;  // residual channels
constexpr int A = WN_A;
constexpr int PC = 2 * R + 4;  // fp32 row pitches in LDS
constexpr int PA = A + 4;
constexpr int SR = 2 * R + 8;  // split-row pitch of an r-vector, in 16-bit units
constexpr int SA = 2 * A + 8;
constexpr int WB = 3;  // weight-tile buffers per wave: tiles are issued two layers ahead

// With 8 streams per workgroup the 16 MFMA columns are paired: column n < 8 takes the hi part of
// stream n's split row and column n + 8 its lo part, so one MFMA does what two do with 16
// streams; fold8 then adds the two halves (lanes n and n + 8 of each 16-lane row, row_ror:8).
template <int K, bool PAIR>
__device__ __forceinline__ f32x4 mfma_split(u32x4 w, const u16* row, int k0, int part, f32x4 acc) {
  if constexpr (PAIR) {
    const bf16x8 a = __builtin_bit_cast(bf16x8, w);
    const bf16x8 v = *reinterpret_cast<const bf16x8*>(row + part * K + k0);
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, v, acc, 0, 0, 0);
  } else {
    return mfma_row<K>(w, row, k0, acc);
  }
}
// tanh(ah) sigmoid(ag) with paired columns: lane n < 8 (part 0) evaluates the tanh and lane
// n + 8 the sigmoid of the same values (after fold8 both hold the same sums), then they swap
// results (row_ror:8), so a wave issues half the transcendental instructions
__device__ __forceinline__ float gate_pair8(float ah, float ag, int part) {
  const bool th = part == 0;
  const float r = __builtin_amdgcn_rcpf(1.0f + wnk::expf_fast(th ? 2.0f * ah : -ag));
  const float v = th ? 1.0f - 2.0f * r : r;
  const float o = wnk::dpp<0x128>(v);
  return th ? v * o : o * v;
}
template <bool PAIR>
__device__ __forceinline__ f32x4 fold8(f32x4 a) {
  if constexpr (PAIR) {
#pragma unroll
    for (int e = 0; e < 4; ++e) a[e] += wnk::dpp<0x128>(a[e]);
  }
  return a;
}

// Tile order of the packed weights, in 1 KB blocks (64 lanes x 16 bytes).
template <int S>
struct Pack {
  static constexpr int KTG = 2 * R / 32;  // gate inputs [x_prev | x]
  static constexpr int KTR = R / 32;
  static constexpr int KTH = S / 32;
  static constexpr int KTO = A / 32;
  static constexpr int GATE = 0;                         // [2R x 2R]: block mt * KTG + kt
  static constexpr int RES = GATE + (2 * R / 16) * KTG;  // [R x R]
  static constexpr int SKIP = RES + (R / 16) * KTR;      // [S x R]
  static constexpr int LAYER = SKIP + (S / 16) * KTR;    // blocks per layer
  static constexpr int NSKT = S / 16;                    // skip row tiles
  static constexpr int SKW = (NSKT + 2) / 3;             // skip row tiles per skip wave
  static constexpr int SS = 2 * S + 8;                   // split-row pitch of an s-vector
};

template <int S>
constexpr size_t lds_bytes(int L) {
  return 4 * ((size_t)2 * G * PC + (size_t)G * PA + (size_t)L * 3 * R + R + S + 2 * A) +
         2 * ((size_t)5 * G * SR + (size_t)G * Pack<S>::SS + (size_t)G * SA + (size_t)A * R + (size_t)G * R);
}

template <int S, bool TF, bool AX, int GS>
__global__ __launch_bounds__(NT) void wn_group_kernel(const WnGroupArgs g) {
  using P = Pack<S>;
  constexpr int SS = P::SS;
  const WnDims& D = g.d;
  const int L = D.L;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: tile addresses go to SGPRs
  constexpr int gs = GS;  // streams of this workgroup: columns 0 .. GS - 1; the others are padding
  const int b0 = blockIdx.x * gs;
  const int T = g.io.T, B = g.io.B;
  const int n = lane & 15, quad = lane >> 4;  // MFMA column and row quad of this lane
  constexpr bool PAIR = GS == 8;              // paired hi / lo columns (see mfma_split)
  const int sn = PAIR ? (n & 7) : n;          // the stream of this lane's column
  const int part = n >> 3;                    // with PAIR: 0 hi, 1 lo
  const bool wl = !PAIR || n < 8;             // the lane that stores its stream's results

  extern __shared__ __align__(16) float sm[];
  float* CD = sm;                // [2][G][PC] conditioning rows (layer parity)
  float* LG = CD + 2 * G * PC;   // [G][PA]    logits
  float* BG = LG + G * PA;       // [L][2R]
  float* BR = BG + L * 2 * R;    // [L][R]
  float* BE = BR + L * R;        // [R]
  float* BS = BE + R;            // [S]
  float* BRL = BS + S;           // [A]
  float* BO = BRL + A;           // [A]
  u16* XS = reinterpret_cast<u16*>(BO + A);  // [2][G][SR] x_{j-1}, split, in buffer j mod 2
  u16* HS = XS + 2 * G * SR;                  // [G][SR]    h_j, split
  u16* XP = HS + G * SR;                      // [2][G][SR] history rows x_{j-1}[t - d_j] (layer parity)
  u16* ZS = XP + 2 * G * SR;                  // [G][SS]    relu(q + B_skip), split
  u16* ZA = ZS + G * SS;                      // [G][SA]    z_a, split
  u16* EMB = ZA + G * SA;                     // [A][R]     embedding of y_{t-1} (bf16)
  u16* EPB = EMB + A * R;                     // [G][R]     embedding row of y_{t-2} (two taps; else 0)
  __shared__ int s_y[G];   // y_{t-1}
  __shared__ int s_y2[G];  // y_{t-2}, -1 before the first input
  __shared__ float s_u[G];
  __shared__ int s_yin[G];
  __shared__ int s_slot[WN_GROUP_MAX_LAYERS];  // history slot (t mod d_j) of the next write of layer j
  // layer j's history offset and dilation: read from LDS in the loop (a dynamically indexed
  // kernel argument would be a scalar memory load each time)
  __shared__ int s_hoff[WN_GROUP_MAX_LAYERS], s_dil[WN_GROUP_MAX_LAYERS];
  // 1 once the loader has seen a host abort request (written before a barrier of a step's first
  // position, read by every wave after that position's last barrier)
  __shared__ int s_abort;

  const u32x4* pk = static_cast<const u32x4*>(g.packed);
  const unsigned loff = (unsigned)lane * 16u;  // this lane's bytes within a 1 KB tile
  // Opaque copies of the tile base and the lane offset keep the compiler from hoisting the
  // addresses of loop-invariant tiles (head, first layer) out of the loops, where they would
  // hold registers for the whole call; the load takes the base in SGPRs and the lane offset.
  // The opaque pointer is generic, so it is cast back to the global address space: a generic
  // (flat) load also counts against the LDS counter, and every wait for an LDS access or an LDS
  // barrier would then wait for the weight tiles in flight from L2 as well.
  typedef const u32x4 __attribute__((address_space(1)))* gtile_ptr;
  auto tile = [&](size_t blk) __attribute__((always_inline)) {
    const char* b = reinterpret_cast<const char*>(pk + blk * 64);
    unsigned o = loff;
    asm volatile("" : "+s"(b), "+v"(o));
    return *(gtile_ptr)(b + o);
  };
  int64_t tg0 = 0;
  {
    // every stream of a call has taken the same number of steps
    const int64_t* st = g.ws.state;
    if (!g.io.reset) tg0 = st[WN_STATE_WORDS * (size_t)b0];
    if (tid < G) {
      int y = g.io.init_sample, y2 = -1;
      if (!g.io.reset && tid < gs && b0 + tid < B) {
        y = (int)st[WN_STATE_WORDS * (size_t)(b0 + tid) + 1];
        y2 = (int)st[WN_STATE_WORDS * (size_t)(b0 + tid) + 2];
      }
      s_y[tid] = y < 0 ? 0 : (y > A - 1 ? A - 1 : y);
      s_y2[tid] = y2 < 0 ? -1 : (y2 > A - 1 ? A - 1 : y2);
    }
  }
  if (tid == 0) s_abort = 0;
  if (tid < L) {
    s_slot[tid] = (int)(tg0 % D.dil[tid]);
    s_hoff[tid] = D.hoff[tid];
    s_dil[tid] = D.dil[tid];
  }
  for (int i = tid; i < L * 2 * R; i += NT) BG[i] = g.w.b_gate[i];
  for (int i = tid; i < L * R; i += NT) BR[i] = g.w.b_res[i];
  for (int i = tid; i < R; i += NT) BE[i] = g.w.b_embed[i];
  for (int i = tid; i < S; i += NT) BS[i] = g.w.b_skip[i];
  for (int i = tid; i < A; i += NT) BRL[i] = g.w.b_relu[i];
  for (int i = tid; i < A; i += NT) BO[i] = g.w.b_out[i];
  {
    const u16* E = static_cast<const u16*>(g.w.embed);
    for (int i = tid; i < A * R; i += NT) EMB[i] = E[i];
  }
  if (g.io.reset) {
    for (int nn = 0; nn < gs && b0 + nn < B; ++nn) {
      float4* hist = reinterpret_cast<float4*>(g.ws.hist + (size_t)(b0 + nn) * D.hist_len);
      for (int i = tid; i < D.hist_len / 4; i += NT) hist[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
  // padding columns never receive rows: zero them once (their products then stay finite)
  for (int i = tid; i < 2 * G * SR; i += NT) XP[i] = 0;
  for (int i = tid; i < 2 * G * PC; i += NT) CD[i] = 0.f;
  __syncthreads();  // also orders the history zeroing before the loader's reads
  // x0 of the first step; EPB holds E_prev[y_{t-2}] of the step whose x0 is formed next (the
  // loader refreshes it a step ahead)
  const u16* Eprev = static_cast<const u16*>(g.w.embed_prev);  // null with one tap
  for (int i = tid; i < G * R; i += NT) {
    const int nn = i / R, c = i % R;
    const u16 ep = (Eprev && s_y2[nn] >= 0) ? Eprev[(size_t)s_y2[nn] * R + c] : (u16)0;
    EPB[i] = ep;
    split1(bf16_val(EMB[s_y[nn] * R + c]) + BE[c] + bf16_val(ep), XS[nn * SR + c], XS[nn * SR + R + c]);
  }

  const int64_t nq = (int64_t)T * L;  // positions (step, layer) of this call

  // Runs every position (step, layer) of the call.  Positions rotate through NBUF prefetch
  // buffers; the body gets the buffer index as a compile-time constant.  The loop leaves right
  // after the position that used a buffer or goes on to the one that refills it, or after the
  // first position of a step once the loader has seen an abort request (every wave reads s_abort
  // at the same position, after its barriers, so all leave together).
  auto run = [&](auto nbuf, auto&& body) __attribute__((always_inline)) {
    constexpr int NBUF = decltype(nbuf)::value;
    static_assert(NBUF == 2 || NBUF == 3, "two or three prefetch buffers");
    int64_t tl = 0;
    int j = 0;
    int64_t q = 0;
    auto step = [&](auto kc) __attribute__((always_inline)) {
      body(kc, q, tl, j);
      const bool stop = j == 0 && s_abort != 0;
      if (++j == L) j = 0, ++tl;
      return ++q == nq || stop;
    };
    for (;;) {
      if (step(std::integral_constant<int, 0>{})) break;
      if (step(std::integral_constant<int, 1>{})) break;
      if constexpr (NBUF == 3) {
        if (step(std::integral_constant<int, 2>{})) break;
      }
    }
  };

  // Head tiles of this wave: row tiles 2w and 2w + 1 of W_relu (issued during the last layer)
  // and of W_out (issued after the W_relu products).
  constexpr size_t HEAD1 = 0, HEAD2 = (size_t)(A / 16) * P::KTH;
  const size_t hbase = (size_t)L * P::LAYER;
  auto issue_head1 = [&](u32x4 (&w)[2 * P::KTH]) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < 2; ++k)
#pragma unroll
      for (int kt = 0; kt < P::KTH; ++kt) w[k * P::KTH + kt] = tile(hbase + HEAD1 + (2 * wave + k) * P::KTH + kt);
  };
  // After the last layer of step tl: the head, the draw (streams 2w and 2w + 1) and the next
  // step's x0.  Three barriers.  Results stay in LDS (logits in LG, samples in s_y); the loader
  // wave writes them out.
  auto head_and_draw = [&](int64_t tl, const u32x4 (&w1)[2 * P::KTH]) __attribute__((always_inline)) {
    u32x4 w2[2 * P::KTO];
    {
      f32x4 acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
      const u16* row = ZS + sn * SS;
#pragma unroll
      for (int kt = 0; kt < P::KTH; ++kt) {
        acc[0] = mfma_split<S, PAIR>(w1[kt], row, kt * 32 + quad * 8, part, acc[0]);
        acc[1] = mfma_split<S, PAIR>(w1[P::KTH + kt], row, kt * 32 + quad * 8, part, acc[1]);
      }
      acc[0] = fold8<PAIR>(acc[0]);
      acc[1] = fold8<PAIR>(acc[1]);
      // W_out tiles: issued once the W_relu tiles are consumed (the empty asm keeps the loads
      // behind the products), so the two sets never hold registers at the same time
      asm volatile("" : "+v"(acc[0]), "+v"(acc[1])::"memory");
#pragma unroll
      for (int k = 0; k < 2; ++k)
#pragma unroll
        for (int kt = 0; kt < P::KTO; ++kt) w2[k * P::KTO + kt] = tile(hbase + HEAD2 + (2 * wave + k) * P::KTO + kt);
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int m0 = (2 * wave + k) * 16 + quad * 4;
        const float4 b = *reinterpret_cast<const float4*>(BRL + m0);
        if (wl)
          store_split4<A>(ZA + sn * SA, m0,
                          make_float4(fmaxf(acc[k][0] + b.x, 0.f), fmaxf(acc[k][1] + b.y, 0.f),
                                      fmaxf(acc[k][2] + b.z, 0.f), fmaxf(acc[k][3] + b.w, 0.f)));
      }
    }
    lds_barrier();
    {
      f32x4 acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
      const u16* row = ZA + sn * SA;
#pragma unroll
      for (int kt = 0; kt < P::KTO; ++kt) {
        acc[0] = mfma_split<A, PAIR>(w2[kt], row, kt * 32 + quad * 8, part, acc[0]);
        acc[1] = mfma_split<A, PAIR>(w2[P::KTO + kt], row, kt * 32 + quad * 8, part, acc[1]);
      }
      acc[0] = fold8<PAIR>(acc[0]);
      acc[1] = fold8<PAIR>(acc[1]);
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int m0 = (2 * wave + k) * 16 + quad * 4;
        const float4 b = *reinterpret_cast<const float4*>(BO + m0);
        if (wl)
          *reinterpret_cast<float4*>(LG + sn * PA + m0) =
              make_float4(acc[k][0] + b.x, acc[k][1] + b.y, acc[k][2] + b.z, acc[k][3] + b.w);
      }
    }
    lds_barrier();
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int nn = 2 * wave + k;
      if (PAIR && nn >= GS) break;  // padding columns: no logits
      int y;
      if constexpr (TF) {
        y = s_yin[nn];
      } else {
        const float4 lv = *reinterpret_cast<const float4*>(LG + nn * PA + 4 * lane);
        y = wave_draw<AX>(lv, s_u[nn], g.io.smode, g.io.inv_t, g.io.top_k, lane);
      }
      if (lane == 0) {
        s_y2[nn] = s_y[nn];
        s_y[nn] = y;
      }
      split1(bf16_val(EMB[y * R + lane]) + BE[lane] + bf16_val(EPB[nn * R + lane]), XS[nn * SR + lane],
             XS[nn * SR + R + lane]);
    }
    lds_barrier();
  };

  // Each role runs its own copy of the position loop, so the completion counters of its loads
  // are tracked exactly; all roles meet at the same barriers.
  if (wave < 4) {
    // ---------------- gate and residual: row tile gi of W_res, gi and gi + 4 of [W_prev | W_cur] ----------------
    constexpr int NB = 2 * P::KTG + P::KTR;
    const int gi = wave;
    const int m0 = gi * 16 + quad * 4;  // this lane's rows of x, h and the tanh half of a
    auto issue = [&](u32x4 (&buf)[NB], int j) __attribute__((always_inline)) {
      const size_t lb = (size_t)j * P::LAYER;
#pragma unroll
      for (int kt = 0; kt < P::KTG; ++kt) {
        buf[kt] = tile(lb + P::GATE + gi * P::KTG + kt);
        buf[P::KTG + kt] = tile(lb + P::GATE + (gi + R / 16) * P::KTG + kt);
      }
      if (j != L - 1) {  // the last layer's x feeds nothing
#pragma unroll
        for (int kt = 0; kt < P::KTR; ++kt) buf[2 * P::KTG + kt] = tile(lb + P::RES + gi * P::KTR + kt);
      }
    };
    u32x4 buf[WB][NB];  // tiles of layers j, j + 1, j + 2
    float4 xr = make_float4(0.f, 0.f, 0.f, 0.f);  // x_{j-1}[t], rows m0 .. m0 + 3 of stream n, fp32
    for (int k = 0; k + 1 < WB; ++k) issue(buf[k], k % L);
    __syncthreads();
    run(std::integral_constant<int, WB>{}, [&](auto kc, int64_t q, int64_t tl, int j) __attribute__((always_inline)) {
      constexpr int k = decltype(kc)::value;
      u32x4(&cur)[NB] = buf[k];
      const int slot = (int)(q & 1);
      if (j == 0) {  // x0 = E[y_{t-1}] + B_embed (+ E_prev[y_{t-2}])
        const u16* e = EMB + s_y[sn] * R + m0;
        const u16* ep = EPB + sn * R + m0;
        xr = make_float4(bf16_val(e[0]) + BE[m0] + bf16_val(ep[0]), bf16_val(e[1]) + BE[m0 + 1] + bf16_val(ep[1]),
                         bf16_val(e[2]) + BE[m0 + 2] + bf16_val(ep[2]), bf16_val(e[3]) + BE[m0 + 3] + bf16_val(ep[3]));
      }
      f32x4 at = {0.f, 0.f, 0.f, 0.f}, as = {0.f, 0.f, 0.f, 0.f};
      const u16* xp = XP + (slot * G + sn) * SR;
      const u16* xc = XS + ((j & 1) * G + sn) * SR;
#pragma unroll
      for (int kt = 0; kt < P::KTG; ++kt) {
        // inputs 0..R-1: the history row x_{j-1}[t - d_j]; R..2R-1: the current x_{j-1}[t]
        const u16* row = kt < R / 32 ? xp : xc;
        const int k0 = (kt % (R / 32)) * 32 + quad * 8;
        at = mfma_split<R, PAIR>(cur[kt], row, k0, part, at);
        as = mfma_split<R, PAIR>(cur[P::KTG + kt], row, k0, part, as);
      }
      at = fold8<PAIR>(at);
      as = fold8<PAIR>(as);
      // the next tiles, issued once this layer's products are under way
      issue(buf[(k + WB - 1) % WB], (j + WB - 1) % L);
      const float* cd = CD + (slot * G + sn) * PC;
      const float4 ch = *reinterpret_cast<const float4*>(cd + m0);
      const float4 cg = *reinterpret_cast<const float4*>(cd + R + m0);
      const float4 bh = *reinterpret_cast<const float4*>(BG + j * 2 * R + m0);
      const float4 bg = *reinterpret_cast<const float4*>(BG + j * 2 * R + R + m0);
      float4 hv;
      if constexpr (PAIR && !AX) {
        hv.x = gate_pair8(at[0] + bh.x + ch.x, as[0] + bg.x + cg.x, part);
        hv.y = gate_pair8(at[1] + bh.y + ch.y, as[1] + bg.y + cg.y, part);
        hv.z = gate_pair8(at[2] + bh.z + ch.z, as[2] + bg.z + cg.z, part);
        hv.w = gate_pair8(at[3] + bh.w + ch.w, as[3] + bg.w + cg.w, part);
      } else {
        hv.x = tanh_nl<AX>(at[0] + bh.x + ch.x) * sigmoid_nl<AX>(as[0] + bg.x + cg.x);
        hv.y = tanh_nl<AX>(at[1] + bh.y + ch.y) * sigmoid_nl<AX>(as[1] + bg.y + cg.y);
        hv.z = tanh_nl<AX>(at[2] + bh.z + ch.z) * sigmoid_nl<AX>(as[2] + bg.z + cg.z);
        hv.w = tanh_nl<AX>(at[3] + bh.w + ch.w) * sigmoid_nl<AX>(as[3] + bg.w + cg.w);
      }
      if (wl) store_split4<R>(HS + sn * SR, m0, hv);
      lds_barrier();
      if (j < L - 1) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kt = 0; kt < P::KTR; ++kt)
          acc = mfma_split<R, PAIR>(cur[2 * P::KTG + kt], HS + sn * SR, kt * 32 + quad * 8, part, acc);
        acc = fold8<PAIR>(acc);
        const float4 br = *reinterpret_cast<const float4*>(BR + j * R + m0);
        xr.x += acc[0] + br.x;
        xr.y += acc[1] + br.y;
        xr.z += acc[2] + br.z;
        xr.w += acc[3] + br.w;
        if (wl) store_split4<R>(XS + (((j + 1) & 1) * G + sn) * SR, m0, xr);
        lds_barrier();
      } else {
        u32x4 w1[2 * P::KTH];
        issue_head1(w1);
        lds_barrier();
        head_and_draw(tl, w1);
      }
    });
  } else if (wave < 7) {
    // ---------------- skip: row tiles sk0 .. sk0 + nsk - 1 of W_skip ----------------
    constexpr int NB = P::SKW * P::KTR;
    const int sk0 = (wave - 4) * P::SKW;
    const int nsk = min(P::SKW, P::NSKT - sk0);
    auto issue = [&](u32x4 (&buf)[NB], int j) __attribute__((always_inline)) {
      const size_t lb = (size_t)j * P::LAYER;
#pragma unroll
      for (int k = 0; k < P::SKW; ++k)
        if (k < nsk) {
#pragma unroll
          for (int kt = 0; kt < P::KTR; ++kt) buf[k * P::KTR + kt] = tile(lb + P::SKIP + (sk0 + k) * P::KTR + kt);
        }
    };
    constexpr int SB = 2;  // tiles of layers j and j + 1 (three sets would not fit in registers)
    u32x4 buf[SB][NB];
    f32x4 qacc[P::SKW];
    for (int k = 0; k + 1 < SB; ++k) issue(buf[k], k % L);
    __syncthreads();
    run(std::integral_constant<int, SB>{}, [&](auto kc, int64_t q, int64_t tl, int j) __attribute__((always_inline)) {
      constexpr int k = decltype(kc)::value;
      u32x4(&cur)[NB] = buf[k];
      issue(buf[(k + SB - 1) % SB], (j + SB - 1) % L);
      lds_barrier();
      // q += W_skip h_j; the first layer starts the sum, so q holds nothing between the head and
      // the next step
      auto skip = [&](bool first) __attribute__((always_inline)) {
#pragma unroll
        for (int k = 0; k < P::SKW; ++k) {
          if (k < nsk) {
            f32x4 acc = first ? f32x4{0.f, 0.f, 0.f, 0.f} : qacc[k];
#pragma unroll
            for (int kt = 0; kt < P::KTR; ++kt)
              acc = mfma_split<R, PAIR>(cur[k * P::KTR + kt], HS + sn * SR, kt * 32 + quad * 8, part, acc);
            qacc[k] = acc;
          }
        }
      };
      if (j < L - 1) {
        skip(j == 0);
        lds_barrier();
      } else {
        skip(false);
#pragma unroll
        for (int k = 0; k < P::SKW; ++k) {
          if (k < nsk) {
            const int m0 = (sk0 + k) * 16 + quad * 4;
            const float4 bs = *reinterpret_cast<const float4*>(BS + m0);
            const f32x4 q = fold8<PAIR>(qacc[k]);
            if (wl)
              store_split4<S>(ZS + sn * SS, m0,
                              make_float4(fmaxf(q[0] + bs.x, 0.f), fmaxf(q[1] + bs.y, 0.f),
                                          fmaxf(q[2] + bs.z, 0.f), fmaxf(q[3] + bs.w, 0.f)));
          }
        }
        u32x4 w1[2 * P::KTH];  // after the skip products, whose tiles no longer hold registers
        issue_head1(w1);
        lds_barrier();
        head_and_draw(tl, w1);
      }
    });
  } else {
    // ---------------- loader ----------------
    // The rows of a position for the GS streams: LPS lanes per stream, lane q of a stream reading
    // 16-byte pieces q, q + LPS, .. of its history row x_{j-1}[t - d_j] (split, 16 pieces) and of
    // its conditioning row (32 pieces), so each load instruction reads contiguous bytes of every
    // stream, and a group of fewer streams issues fewer loads.
    constexpr int LPS = 64 / GS;
    constexpr int NH = (16 + LPS - 1) / LPS, NC = (32 + LPS - 1) / LPS;
    constexpr int NB = NH + NC;
    const int lsn = lane / LPS, lq = lane % LPS;  // stream and lane within it
    const int ldn = lane >> 2, ldq = lane & 3;    // quarter ldq of stream ldn's E_prev row (two taps)
    const int lub = min(b0 + lane, B - 1);        // reads of a partial group are clamped
    const size_t lsb = (size_t)min(b0 + lsn, B - 1);
    const float* hrd = g.ws.hist + lsb * D.hist_len + lq * 4;
    const float* crd = g.io.cond + lsb * T * L * 2 * R + lq * 4;
    auto issue = [&](u32x4 (&buf)[NB], int64_t tl, int j) __attribute__((always_inline)) {
      if (tl >= T) return;
      const int hoff = __builtin_amdgcn_readfirstlane(s_hoff[j] + s_slot[j] * R);
      const float* h = hrd + hoff;
      const float* c = crd + ((size_t)tl * L + j) * 2 * R;
#pragma unroll
      for (int k = 0; k < NH; ++k)
        if (lq + LPS * k < 16) buf[k] = *reinterpret_cast<const u32x4*>(h + 4 * LPS * k);
#pragma unroll
      for (int k = 0; k < NC; ++k)
        if (lq + LPS * k < 32) buf[NH + k] = *reinterpret_cast<const u32x4*>(c + 4 * LPS * k);
    };
    auto store = [&](int slot, const u32x4 (&buf)[NB]) __attribute__((always_inline)) {
      u32x4* xp = reinterpret_cast<u32x4*>(XP + (slot * G + lsn) * SR) + lq;
#pragma unroll
      for (int k = 0; k < NH; ++k)
        if (lq + LPS * k < 16) xp[LPS * k] = buf[k];
      u32x4* cd = reinterpret_cast<u32x4*>(CD + (slot * G + lsn) * PC) + lq;
#pragma unroll
      for (int k = 0; k < NC; ++k)
        if (lq + LPS * k < 32) cd[LPS * k] = buf[NH + k];
    };
    // Samples (generation) or logits (teacher forcing) of step tl, from s_y / LG, for the group.
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
            if (c + k < gs && b0 + c + k < B) reinterpret_cast<f32x4*>(g.io.logits + ((size_t)(b0 + c + k) * T + tl) * A)[lane] = v[k];
        }
      } else {
        if (lane < gs && b0 + lane < B) g.io.y_out[(size_t)(b0 + lane) * T + tl] = s_y[lane];
      }
    };
    u32x4 bufA[NB], bufB[NB];
    float pre_u = 0.f;
    int pre_y = 0;
    u32x4 pre_e[2];  // two taps: quarter ldq of E_prev[y_{t-1}] of stream ldn, for the next step
    // rows of positions 0 and 1 (both in the first step: the kernel takes l >= 2)
    issue(bufB, 0, 0);
    store(0, bufB);
    issue(bufA, 0, 1);
    int64_t tl2 = 2 / L;  // position q + 2 of the loop below
    int j2 = 2 % L;
    __syncthreads();
    run(std::integral_constant<int, 2>{}, [&](auto parity, int64_t q, int64_t tl, int j) __attribute__((always_inline)) {
      u32x4(&cur)[NB] = decltype(parity)::value == 0 ? bufA : bufB;
      u32x4(&nxt)[NB] = decltype(parity)::value == 0 ? bufB : bufA;
      // On gfx950 a wait for a load while stores are outstanding also waits for the stores, so
      // this wave first consumes what it loaded a layer ago, then stores, then issues its loads:
      // the next layer's wait then covers only stores that were issued before the loads it needs.
      // (Moving this work to phase B, when the weight waves issue nothing, measured slower.)
      if (q + 1 < nq) store((int)((q + 1) & 1), cur);
      // this step's uniform (or teacher sample): read at the first layer, staged at the second
      if (j == 1 && lane < G) {
        if constexpr (TF) s_yin[lane] = pre_y < 0 ? 0 : (pre_y > A - 1 ? A - 1 : pre_y);
        else s_u[lane] = pre_u;
      }
      // two taps: E_prev[y_{t-1}], read at the first layer, replaces E_prev[y_{t-2}] once the first
      // layer has used it; the draw at the end of this step forms the next x0 from it
      if (j == 1 && Eprev) {
        u32x4* d = reinterpret_cast<u32x4*>(EPB + ldn * R + ldq * 16);
        d[0] = pre_e[0];
        d[1] = pre_e[1];
      }
      // x_{j-1}[t] (split) into slot t mod d_j of layer j's history, read again at step t + d_j.
      // The slot counter of layer j then moves on to step t + 1, so a read issued from here on
      // for layer j (step t + 1) or for a layer after j (step t) finds its slot in s_slot.
      {
        const int slot = __builtin_amdgcn_readfirstlane(s_slot[j]);
        char* hw = reinterpret_cast<char*>(g.ws.hist) + ((size_t)s_hoff[j] + (size_t)slot * R) * 4;
        static_assert(G * 2 * R * 2 / 16 / 64 == 4, "four 16-byte pieces of x per loader lane");
        f32x4 v[4] = {};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int i = lane + 64 * k;  // stream i / 16, piece i % 16 of its 256-byte row
          if (4 * k < gs) v[k] = *reinterpret_cast<const f32x4*>(XS + ((j & 1) * G + (i >> 4)) * SR + (i & 15) * 8);
        }
        asm volatile("" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]));
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int i = lane + 64 * k, nn = i >> 4;
          if (4 * k < gs && nn < gs && b0 + nn < B)
            *reinterpret_cast<f32x4*>(hw + (size_t)(b0 + nn) * D.hist_len * 4 + (i & 15) * 16) = v[k];
        }
        if (lane == 0) s_slot[j] = slot + 1 == s_dil[j] ? 0 : slot + 1;
      }
      // outputs of the previous step, left in LDS by its head and draw
      if (j == 0 && tl > 0) write_outputs(tl - 1);
      if (j == 0 && lane < G) {
        if constexpr (TF) pre_y = g.io.y_in[(size_t)lub * T + tl];
        else pre_u = g.io.u[(size_t)lub * T + tl];
      }
      if (j == 0 && Eprev) {
        const u32x4* e = reinterpret_cast<const u32x4*>(Eprev + (size_t)s_y[ldn] * R + ldq * 16);
        pre_e[0] = e[0];
        pre_e[1] = e[1];
      }
      // a host abort request, read every WN_ABORT_CHECK steps
      if (j == 0 && lane == 0 && (tl & (WN_ABORT_CHECK - 1)) == 0 && abort_requested(g.io.abort_flag)) {
        atomicCAS(g.ws.status, 0, (int)WN_EABORTED);
        s_abort = 1;
      }
      issue(nxt, tl2, j2);
      if (++j2 == L) j2 = 0, ++tl2;
      lds_barrier();
      if (j < L - 1) {
        lds_barrier();
      } else {
        u32x4 w1[2 * P::KTH];
        issue_head1(w1);
        lds_barrier();
        head_and_draw(tl, w1);
      }
    });
    if (!s_abort) write_outputs(T - 1);  // the last step's, after its draw
  }
  __syncthreads();
  // after an abort the state stays as it was (the next call must start from zero)
  if (tid < gs && b0 + tid < B && !s_abort) {
    int64_t* st = g.ws.state + WN_STATE_WORDS * (size_t)(b0 + tid);
    st[0] = tg0 + T;
    st[1] = s_y[tid];
    st[2] = s_y2[tid];
  }
}

template <int S, bool TF, bool AX, int GS>
hipError_t launch_group_k(const WnGroupArgs& g, hipStream_t stream) {
  const size_t dyn = lds_bytes<S>(g.d.L);
  const dim3 grid((g.io.B + GS - 1) / GS), block(NT);
  const void* k = reinterpret_cast<const void*>(wn_group_kernel<S, TF, AX, GS>);
  const hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((wn_group_kernel<S, TF, AX, GS>), grid, block, dyn, stream, g);
  return hipGetLastError();
}

template <int S, bool TF, bool AX>
hipError_t launch_group_gs(const WnGroupArgs& g, hipStream_t stream) {
  if (g.gs == 8) return launch_group_k<S, TF, AX, 8>(g, stream);
  if (g.gs == 16) return launch_group_k<S, TF, AX, 16>(g, stream);
  return hipErrorInvalidValue;
}

template <int S>
hipError_t launch_group_s(const WnGroupArgs& g, bool teacher, hipStream_t stream) {
  const bool ax = g.w.approx_nl != 0;
  if (teacher) return ax ? launch_group_gs<S, true, true>(g, stream) : launch_group_gs<S, true, false>(g, stream);
  return ax ? launch_group_gs<S, false, true>(g, stream) : launch_group_gs<S, false, false>(g, stream);
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

// Eight streams per workgroup fill the MFMA columns with their hi and lo parts (one MFMA per
// product instead of two) while the loader wave moves half the rows, and up to 2048 streams still
// fit one workgroup per CU.  Measured at l = 20, r = 64, B = 256: 25.4 us per step against 29.0
// with 16 streams per workgroup (with one stream per column, 4, 2 and 1 streams per workgroup
// took 28.3, 27.9 and 31.2 us).
int wn_group_streams(int B) {
  if (const char* e = std::getenv("WN_GROUP_STREAMS")) {
    const int v = std::atoi(e);
    if (v == 8 || v == 16) return v;
  }
  return B <= 8 * WN_CHAIN_GRID ? 8 : 16;
}

size_t wn_group_lds_bytes(int L, int S_, bool) {
  return S_ == 256 ? lds_bytes<256>(L) : lds_bytes<128>(L);
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
