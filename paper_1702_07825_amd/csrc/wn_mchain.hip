// Multi-CU persistent generation kernel for bf16 and int8 models (r = 64) on gfx950 MFMA: the
// streams of a replica go through the layer chain together.
//
// The roles and the messages are those of the fp32 multi-CU kernel: the weights stay resident for
// the whole call, as in the paper's persistent GPU kernel (Deep Voice, arXiv 1702.07825, Appendix
// D), and the work that does not depend on the current step's chain is done off the chain, a step
// ahead, as its CPU design does with auxiliary threads (Section 5.1); the arithmetic is Appendix
// A.1's.  What differs is the batch: every product of a layer is a [rows x 64] . [64 x 16]
// contraction on v_mfma_f32_16x16x32_bf16, and every message is a block of tiles.
//
// An activation enters a product as a pair of bf16 values, hi = bf16(v) and lo = bf16(v - hi),
// and both are multiplied, so a product sees about 16 bits of the activation; the weights are
// exactly bf16 (int8 codes are exact in bf16, and each row's scale multiplies its fp32 result).
// Accumulation, the gate, the residual and skip sums and the softmax are fp32.  The 16 columns of a
// tile take the streams in one of two ways:
//   paired   8 streams per replica: column n < 8 holds the hi part of stream n and column n + 8 its
//            lo part, so one MFMA per 32 inputs does the work of two, and fold8 (row_ror:8) adds the
//            halves, leaving lanes n and n + 8 with the same sums.  The two lanes then share the
//            gates (each evaluates two of its four whole and they swap results; the Appendix C
//            forms split each gate into the tanh and the sigmoid instead) and the posts.  One
//            head CU.
//   16-wide  16 streams per replica, one per column, two MFMAs per 32 inputs (hi, lo); two head
//            CUs of 8 streams each.  Used when the paired replicas cannot carry the batch.
//
//   chain CU  (up to NLC layers) wave w keeps row tile w of the tanh half and of the sigmoid half
//             of W_cur and row tile w of W_res in registers, as MFMA A operands.  Per layer:
//               phase A  a = pre + W_cur x; h = tanh(a_tanh) sigmoid(a_sigmoid) (a wave holds both
//                        halves of its rows, so the gate needs no exchange); h goes to the layer's
//                        aux CU (skip projection), and the layer's input x_{j-1}[t] to its dilation
//                        history, as tagged tiles;
//               phase B  x += W_res h + B_res (each lane keeps its four rows of x in fp32).
//             The last chain CU also computes the last layer's skip projection (its W_skip in LDS)
//             and posts it to the head.
//   aux CU    (up to NLA layers) wave v keeps row tiles 2v, 2v + 1 of W_prev and four of W_skip.
//             For the next step it computes pre = W_prev x_{j-1}[t + 1 - d] + B + L[t + 1] of each
//             layer (the dilated half, the bias and the HBM read of the conditioning all happen a
//             step early), and for the current step the sum of W_skip h over its layers.
//   head CU   8 streams; wave v keeps four row tiles of W_relu and of W_out.  It sums the skip
//             partials, z_s = relu(.. + B_skip), z_a = relu(W_relu z_s + B_relu), logits = W_out
//             z_a + B_out (paired columns), draws two streams per wave and posts the next step's
//             x0 = E[y] + B_embed (+ E_prev[y_{t-1}], the two-tap input of Section 5.1) to chain
//             CU 0.
//
// A CU runs four waves, one per SIMD, so that each wave can hold 512 registers (the resident weights
// take up to 240 of them); the layer's critical path is the gate waves' either way.
//
// Messages are tagged 64-bit words (fp32 value, step + 1; see wn_msg.h) laid out in the MFMA
// accumulator order: in a block of NS-column tiles (NS streams), word 16 NS tile + 4 (NS quad + c) +
// e holds row 16 tile + 4 quad + e of column c, so the lanes that computed a tile post it as it lies
// in their registers.  A mailbox has one slot: a producer writes step t + 1 only after something
// that depends on its consumer's read of step t (the aux CU posts pre_j[t + 1] once h_j[t] is in,
// which the chain posts after reading pre_j[t]; every role's step t + 1 needs x0[t + 1], which the
// head posts after reading the skip partials of step t, the last of the step's messages), and the
// tags keep the steps apart.  The dilation histories are rings of such blocks: slot t mod d_j of
// layer j holds x_{j-1}[t].  Every wait is bounded: a block that times out stores WN_ETIMEOUT in the
// status word, and every other block sees it in its next wait and leaves, so the grid always drains.
#include "wn_internal.h"
#include "wn_mfma.h"
#include "wn_msg.h"
#include "wn_wave.h"

#include "wn.h"

#include <algorithm>
#include <cstdlib>
#include <type_traits>

namespace {

using namespace wnk;

constexpr int NT = 256;        // four waves: one per SIMD, so each can hold 512 registers
constexpr int R = 64;
constexpr int A = WN_A;
constexpr int NLC = 10;        // layers per chain CU
constexpr int NLA = 5;         // layers per aux CU
constexpr int SR = 2 * R + 8;  // split-row pitch (16-bit units) of an r-vector in LDS
constexpr int HG = 8;          // streams per head CU

// Column layout of a replica's tiles.
template <bool PAIR>
struct Cols {
  static constexpr int NS = PAIR ? 8 : 16;  // streams of a replica
  static constexpr int NH = PAIR ? 1 : 2;   // head CUs of a replica
  static constexpr int XW = R * NS;         // words of an r-vector block (x, h)
  static constexpr int PW = 2 * R * NS;     // words of a pre-activation block
  static constexpr int TW = 16 * NS;        // words of one 16-row tile of a block
};
// Place of (row m, column c) in a block of NS-column tiles; trow / tcol invert it.
template <int NS>
__device__ __forceinline__ int tpos(int m, int c) {
  return (m >> 4) * 16 * NS + (((m >> 2) & 3) * NS + c) * 4 + (m & 3);
}
template <int NS>
__device__ __forceinline__ int trow(int i) { return (i / (16 * NS)) * 16 + ((i / (4 * NS)) & 3) * 4 + (i & 3); }
template <int NS>
__device__ __forceinline__ int tcol(int i) { return (i >> 2) & (NS - 1); }

// MFMA A operand from a row-major [rows][K] matrix: row `row`, inputs col .. col + 7 as bf16 (int8
// codes are exact in bf16).
template <bool I8>
__device__ __forceinline__ u32x4 wfrag(const void* W, size_t row, int K, int col) {
  if constexpr (I8) {
    const uint2 q = *reinterpret_cast<const uint2*>(static_cast<const signed char*>(W) + row * K + col);
    auto cv = [](unsigned w, int b) { return (float)(signed char)(w >> (8 * b)); };
    u32x4 r;
    r[0] = pack_bf16(cv(q.x, 0), cv(q.x, 1));
    r[1] = pack_bf16(cv(q.x, 2), cv(q.x, 3));
    r[2] = pack_bf16(cv(q.y, 0), cv(q.y, 1));
    r[3] = pack_bf16(cv(q.y, 2), cv(q.y, 3));
    // the fragment moves to AGPRs once, here: a value a VALU instruction produced otherwise stays in
    // VGPRs and is copied to AGPRs before every product that reads it
    asm volatile("" : "+a"(r));
    return r;
  } else {
    return *reinterpret_cast<const u32x4*>(static_cast<const u16*>(W) + row * K + col);
  }
}

__device__ __forceinline__ f32x4 f4(float4 v) { return f32x4{v.x, v.y, v.z, v.w}; }
__device__ __forceinline__ float4 v4(f32x4 v) { return make_float4(v[0], v[1], v[2], v[3]); }
__device__ __forceinline__ u32x4 ld16(const u16* p) { return *reinterpret_cast<const u32x4*>(p); }

// Products whose A operand (resident weights) stays in AGPRs.  The gfx950 MFMA reads its A operand
// from AGPRs directly; the compiler's builtin takes it from VGPRs and would copy four AGPRs before
// every product.  A block issues its MFMAs back to back (accumulating into the same registers needs
// no wait), starts with 2 wait states (an operand a VALU instruction has just written) and ends with
// 16 (a VALU read of an 8-pass MFMA result needs 11-12), so no instruction around it can see a result
// in flight.  Two tiles that share their B operands are interleaved.
#define WN_MFMA "v_mfma_f32_16x16x32_bf16 "
// a += Wa [hi; lo], b += Wb [hi; lo] over 64 inputs: w*0 / w*1 hold inputs 0-31 / 32-63 of the rows;
// h0, l0 / h1, l1 the hi and lo parts of this lane's B operand for each half
__device__ __forceinline__ void mfma_k64_2(f32x4& a, f32x4& b, const u32x4& wa0, const u32x4& wa1, const u32x4& wb0,
                                           const u32x4& wb1, u32x4 h0, u32x4 l0, u32x4 h1, u32x4 l1) {
  asm volatile("s_nop 1\n\t"
               WN_MFMA "%0, %2, %6, %0\n\t" WN_MFMA "%1, %4, %6, %1\n\t"
               WN_MFMA "%0, %2, %7, %0\n\t" WN_MFMA "%1, %4, %7, %1\n\t"
               WN_MFMA "%0, %3, %8, %0\n\t" WN_MFMA "%1, %5, %8, %1\n\t"
               WN_MFMA "%0, %3, %9, %0\n\t" WN_MFMA "%1, %5, %9, %1\n\t"
               "s_nop 7\n\ts_nop 7"
               : "+v"(a), "+v"(b)
               : "a"(wa0), "a"(wa1), "a"(wb0), "a"(wb1), "v"(h0), "v"(l0), "v"(h1), "v"(l1));
}
__device__ __forceinline__ f32x4 mfma_k64(f32x4 a, const u32x4& w0, const u32x4& w1, u32x4 h0, u32x4 l0, u32x4 h1,
                                          u32x4 l1) {
  asm volatile("s_nop 1\n\t"
               WN_MFMA "%0, %1, %3, %0\n\t" WN_MFMA "%0, %1, %4, %0\n\t"
               WN_MFMA "%0, %2, %5, %0\n\t" WN_MFMA "%0, %2, %6, %0\n\t"
               "s_nop 7\n\ts_nop 7"
               : "+v"(a)
               : "a"(w0), "a"(w1), "v"(h0), "v"(l0), "v"(h1), "v"(l1));
  return a;
}
// The same products with paired columns: one B operand per 32 inputs (this lane's part of its stream).
__device__ __forceinline__ void mfma_k64_2p(f32x4& a, f32x4& b, const u32x4& wa0, const u32x4& wa1, const u32x4& wb0,
                                            const u32x4& wb1, u32x4 x0, u32x4 x1) {
  asm volatile("s_nop 1\n\t"
               WN_MFMA "%0, %2, %6, %0\n\t" WN_MFMA "%1, %4, %6, %1\n\t"
               WN_MFMA "%0, %3, %7, %0\n\t" WN_MFMA "%1, %5, %7, %1\n\t"
               "s_nop 7\n\ts_nop 7"
               : "+v"(a), "+v"(b)
               : "a"(wa0), "a"(wa1), "a"(wb0), "a"(wb1), "v"(x0), "v"(x1));
}
__device__ __forceinline__ f32x4 mfma_k64p(f32x4 a, const u32x4& w0, const u32x4& w1, u32x4 x0, u32x4 x1) {
  asm volatile("s_nop 1\n\t"
               WN_MFMA "%0, %1, %3, %0\n\t" WN_MFMA "%0, %2, %4, %0\n\t"
               "s_nop 7\n\ts_nop 7"
               : "+v"(a)
               : "a"(w0), "a"(w1), "v"(x0), "v"(x1));
  return a;
}
// a += Wa x, b += Wb x over 128 inputs in paired columns (four 32-input chunks k: wa[k], x[k])
__device__ __forceinline__ void mfma_k128_2p(f32x4& a, f32x4& b, const u32x4 (&wa)[4], const u32x4 (&wb)[4],
                                             const u32x4 (&x)[4]) {
  asm volatile("s_nop 1\n\t"
               WN_MFMA "%0, %2, %10, %0\n\t" WN_MFMA "%1, %6, %10, %1\n\t"
               WN_MFMA "%0, %3, %11, %0\n\t" WN_MFMA "%1, %7, %11, %1\n\t"
               WN_MFMA "%0, %4, %12, %0\n\t" WN_MFMA "%1, %8, %12, %1\n\t"
               WN_MFMA "%0, %5, %13, %0\n\t" WN_MFMA "%1, %9, %13, %1\n\t"
               "s_nop 7\n\ts_nop 7"
               : "+v"(a), "+v"(b)
               : "a"(wa[0]), "a"(wa[1]), "a"(wa[2]), "a"(wa[3]), "a"(wb[0]), "a"(wb[1]), "a"(wb[2]), "a"(wb[3]),
                 "v"(x[0]), "v"(x[1]), "v"(x[2]), "v"(x[3]));
}
// Products over 64 inputs taken from a split row (the lane's stream): a += Wa x, b += Wb x.  With
// paired columns the lane reads its part (hi or lo) only and the caller folds.
template <bool PAIR>
__device__ __forceinline__ void prod2(f32x4& a, f32x4& b, const u32x4& wa0, const u32x4& wa1, const u32x4& wb0,
                                      const u32x4& wb1, const u16* row, int quad, int part) {
  if constexpr (PAIR) {
    const u16* r = row + part * R + 8 * quad;
    mfma_k64_2p(a, b, wa0, wa1, wb0, wb1, ld16(r), ld16(r + 32));
  } else {
    mfma_k64_2(a, b, wa0, wa1, wb0, wb1, ld16(row + 8 * quad), ld16(row + R + 8 * quad), ld16(row + 32 + 8 * quad),
               ld16(row + R + 32 + 8 * quad));
  }
}
template <bool PAIR>
__device__ __forceinline__ f32x4 prod1(f32x4 a, const u32x4& w0, const u32x4& w1, const u16* row, int quad, int part) {
  if constexpr (PAIR) {
    const u16* r = row + part * R + 8 * quad;
    return mfma_k64p(a, w0, w1, ld16(r), ld16(r + 32));
  } else {
    return mfma_k64(a, w0, w1, ld16(row + 8 * quad), ld16(row + R + 8 * quad), ld16(row + 32 + 8 * quad),
                    ld16(row + R + 32 + 8 * quad));
  }
}
// Paired columns: lanes n and n + 8 of each 16-lane row add their sums (row_ror:8).
__device__ __forceinline__ f32x4 fold8(f32x4 a) {
#pragma unroll
  for (int e = 0; e < 4; ++e) a[e] += dpp<0x128>(a[e]);
  return a;
}

// Four tagged words (one lane's element run of a tile) with one scope decision.
__device__ __forceinline__ void stw4(u64* p, float4 v, unsigned tag, bool local) {
  const u64 a = pack(v.x, tag), b = pack(v.y, tag), c = pack(v.z, tag), d = pack(v.w, tag);
  if (local) {
    __hip_atomic_store(p + 0, a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    __hip_atomic_store(p + 1, b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    __hip_atomic_store(p + 2, c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    __hip_atomic_store(p + 3, d, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  } else {
    __hip_atomic_store(p + 0, a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(p + 1, b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(p + 2, c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(p + 3, d, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Two tagged words.
__device__ __forceinline__ void stw2(u64* p, float a, float b, unsigned tag, bool local) {
  const u64 x = pack(a, tag), y = pack(b, tag);
  if (local) {
    __hip_atomic_store(p + 0, x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    __hip_atomic_store(p + 1, y, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  } else {
    __hip_atomic_store(p + 0, x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(p + 1, y, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}
// A lane's four rows of a tile, posted at p (its run of four words): with paired columns the two
// lanes of a stream post two words each (part 0 elements 0 and 1, part 1 elements 2 and 3).
template <bool PAIR>
__device__ __forceinline__ void post4(u64* p, float4 v, unsigned tag, bool local, int part) {
  if constexpr (PAIR) {
    if (part) stw2(p + 2, v.z, v.w, tag, local);
    else stw2(p, v.x, v.y, tag, local);
  } else {
    stw4(p, v, tag, local);
  }
}

// Pair polls (wn_msg.h) over the replicas' histories and mailboxes.  Pair p holds words 2p and 2p + 1
// of a block; word(p) is the word offset of word 2p in the region.
__device__ __forceinline__ wrsrc tagged_region(const WnChainArgs& g) {
  return region_rsrc(g.ring, (size_t)(g.mb + (size_t)g.nrep * g.mb_words - g.ring));
}
template <int K, int NP = NT, class Word>
__device__ __forceinline__ void pairs_start(u32x4 (&w)[K], wrsrc rs, int ti, int np, Word word) {
#pragma unroll
  for (int k = 0; k < K; ++k)
    if (ti + k * NP < np) w[k] = ld_pair(rs, word(ti + k * NP));
}
// Waits until both words of each of this thread's pairs carry their tags, then sink(i, q, value) for
// words i = 2p, 2p + 1 in order (q = 2k or 2k + 1: the word's place in the batch).
// ZZ: s_sleep units (64 clocks each) between two reloads of words that are not there yet: long for
// waits off the critical path (they would otherwise keep the L2 busy for microseconds), none for the
// rest (a one-unit sleep there measured 0.7 us/step slower at l = 20, B = 256), with a compiler barrier
// in its place so that the loads stay in the loop.
template <int K, int NP = NT, int ZZ = 0, class Word, class Tag, class Sink>
__device__ __forceinline__ void pairs_finish(const WnChainArgs& g, u32x4 (&w)[K], wrsrc rs, int ti, int np, Word word,
                                             Tag tag, Sink sink, Sync s) {
  static_assert(K <= 32, "pending bits");
  unsigned pend = 0;
#pragma unroll
  for (int k = 0; k < K; ++k)
    if (ti + k * NP < np) pend |= 1u << k;
  int spins = 0;
  for (;;) {
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int p = ti + k * NP;
      if (((pend >> k) & 1u) && w[k][1] == tag(2 * p) && w[k][3] == tag(2 * p + 1)) pend &= ~(1u << k);
    }
    if (!pend) break;
    if (++spins > g.spin_limit || ((spins & 63) == 0 && ld_status(g.status) != 0)) {
      if (ld_status(g.status) == 0) atomicCAS(g.status, 0, (int)WN_ETIMEOUT);
      *s.flag = 1;
      return;
    }
    if constexpr (ZZ > 0) __builtin_amdgcn_s_sleep(ZZ);
    else asm volatile("" ::: "memory");  // keeps the reloads in the loop
#pragma unroll
    for (int k = 0; k < K; ++k)
      if ((pend >> k) & 1u) w[k] = ld_pair(rs, word(ti + k * NP));
  }
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const int p = ti + k * NP;
    if (p < np) {
      sink(2 * p, 2 * k, __uint_as_float(w[k][0]));
      sink(2 * p + 1, 2 * k + 1, __uint_as_float(w[k][2]));
    }
  }
}
// Both halves at once, in batches of K pairs per thread.
template <int K, int NP = NT, int ZZ = 0, class Word, class Tag, class Sink>
__device__ __forceinline__ void poll_pairs(const WnChainArgs& g, wrsrc rs, int ti, int np, Word word, Tag tag, Sink sink,
                                           Sync s) {
  for (int base = 0; base < np; base += K * NP) {
    u32x4 w[K];
    const int rem = np - base;
    auto wd = [&](int p) { return word(base + p); };
    auto tg = [&](int i) { return tag(2 * base + i); };
    auto sk = [&](int i, int q, float v) { sink(2 * base + i, q, v); };
    pairs_start<K, NP>(w, rs, ti, rem, wd);
    pairs_finish<K, NP, ZZ>(g, w, rs, ti, rem, wd, tg, sk, s);
    if (s.failed()) return;
  }
}

// tanh(a) sigmoid(g) with two exponentials and one reciprocal: (e^{2a} - 1) / ((e^{2a} + 1)(1 + e^{-g})).
// a is clamped to +-15, where tanh is +-1 to fp32 already; a large -g makes e^{-g} infinite and the
// product 0, as sigmoid's limit.
__device__ __forceinline__ float gate_tanh_sigmoid(float a, float g) {
  const float e2a = expf_fast(2.0f * fminf(fmaxf(a, -15.0f), 15.0f));
  const float eg = expf_fast(-g);
  return (e2a - 1.0f) * __builtin_amdgcn_rcpf((e2a + 1.0f) * (1.0f + eg));
}
template <bool AX>
__device__ __forceinline__ float gate_h(float a, float g) {
  if constexpr (AX) return tanh_paper(a) * sigmoid_paper(g);
  else return gate_tanh_sigmoid(a, g);
}

// Appendix C's tanh(ah) sigmoid(ag) with paired columns: after fold8 lanes n and n + 8 hold the
// same ah and ag; lane n (part 0) evaluates the tanh and lane n + 8 the sigmoid, with the same
// operations as tanh_paper and sigmoid_paper, and they swap results (row_ror:8).
__device__ __forceinline__ float gate_pair8_paper(float ah, float ag, int part) {
  const bool th = part == 0;
  const float x = th ? ah : ag;
  const float e = e_tilde(x);
  const float r = __builtin_amdgcn_rcpf(th ? e : 1.0f + e);
  const float v = th ? copysignf((e - r) * __builtin_amdgcn_rcpf(e + r), x) : (x >= 0.0f ? e * r : r);
  const float o = dpp<0x128>(v);
  return th ? v * o : o * v;
}
// Four gates of paired columns.  Exact forms (AX false): lane part 0 evaluates elements 0 and 1 and part 1
// elements 2 and 3 in the unpaired form (three transcendental instructions each), and the two lanes
// swap results, fewer instructions than splitting every element into tanh and sigmoid halves.
template <bool AX, bool PAIR>
__device__ __forceinline__ float4 gate4(f32x4 at, f32x4 ag, int part) {
  if constexpr (PAIR && !AX) {
    const float h0 = gate_tanh_sigmoid(part ? at[2] : at[0], part ? ag[2] : ag[0]);
    const float h1 = gate_tanh_sigmoid(part ? at[3] : at[1], part ? ag[3] : ag[1]);
    const float o0 = dpp<0x128>(h0), o1 = dpp<0x128>(h1);
    return part ? make_float4(o0, o1, h0, h1) : make_float4(h0, h1, o0, o1);
  } else if constexpr (PAIR)
    return make_float4(gate_pair8_paper(at[0], ag[0], part), gate_pair8_paper(at[1], ag[1], part),
                       gate_pair8_paper(at[2], ag[2], part), gate_pair8_paper(at[3], ag[3], part));
  else
    return make_float4(gate_h<AX>(at[0], ag[0]), gate_h<AX>(at[1], ag[1]), gate_h<AX>(at[2], ag[2]),
                       gate_h<AX>(at[3], ag[3]));
}
// Rows m0 .. m0 + 3 of an r-vector into a split row: with paired columns lane part 0 writes the hi
// parts and part 1 the lo parts.
template <bool PAIR>
__device__ __forceinline__ void put_split4(u16* row, int m0, float4 v, int part) {
  if constexpr (PAIR) {
    uint2 hi, lo;
    split4(v, hi, lo);
    *reinterpret_cast<uint2*>(row + part * R + m0) = part ? lo : hi;
  } else {
    store_split4<R>(row, m0, v);
  }
}

// A polled word of an r-vector block into a split row set [NS][SR] (hi and lo parts).
template <int NS>
__device__ __forceinline__ void split_into(u16* rows, int i, float v) {
  const int m = trow<NS>(i), c = tcol<NS>(i);
  split1(v, rows[c * SR + m], rows[c * SR + R + m]);
}

// Dynamic LDS of each role, in bytes (the launch takes the largest); mirrors the carving below.
template <bool PAIR>
constexpr size_t chain_lds(int S) {
  using C = Cols<PAIR>;
  return 4 * ((size_t)NLC * C::PW + (size_t)C::XW + (size_t)NLC * R + (size_t)NLC * 3 * R + S) +
         2 * (size_t)3 * C::NS * SR + (size_t)(S / 16) * 2 * 64 * 16;
}
template <bool PAIR>
constexpr size_t aux_lds(int S) {
  using C = Cols<PAIR>;
  return 4 * ((size_t)NLA * C::PW + (size_t)NLA * 4 * R + (size_t)NLA * S) + 2 * (size_t)2 * NLA * C::NS * SR;
}
constexpr size_t head_lds(int S) {
  return 2 * ((size_t)HG * (2 * S + 8) + (size_t)HG * (2 * A + 8)) + 4 * ((size_t)HG * (A + 4) + S + 6 * A + R) +
         2 * (size_t)2 * A * R;
}

// ------------------------------------------------------------------------------------------
// chain CU: layers j0 .. j0 + nl - 1
// ------------------------------------------------------------------------------------------
// NLK > 0: this CU holds NLK layers, a compile-time count, so that no layer of the unrolled loop
// tests a run-time count; NLK = 0: the count is read at run time.
template <int S, bool AX, bool I8, bool PAIR, int NLK, class LM>
__device__ __forceinline__ void mc_chain(const WnChainArgs& g, const int c, const int rep, float* dyn, Sync sy,
                                         const int64_t tg0, const LM lm) {
  using C = Cols<PAIR>;
  constexpr int NS = C::NS, XW = C::XW, PW = C::PW, TW = C::TW;
  constexpr int KS = S / 64;  // row tiles per wave of the last layer's W_skip (tail)
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 15, quad = lane >> 4;
  const int sn = PAIR ? (n & 7) : n, part = PAIR ? (n >> 3) : 0;  // this lane's stream and part
  const int L = g.d.L, T = g.io.T;
  const int j0 = g.layer_begin[c], nl = NLK > 0 ? NLK : g.layer_begin[c + 1] - j0;
  const bool lastc = c + 1 == g.nch;
  const bool tail = lastc && g.tail_on_chain;
  u64* const mb = g.mb + (size_t)rep * g.mb_words;
  u64* const ring = g.ring + (size_t)rep * g.d.hist_len * NS;
  const wrsrc rs = tagged_region(g);
  const unsigned mbw = (unsigned)(mb - g.ring);  // word offset of my replica's mailboxes in the region
  float* PRE = dyn;                  // [NLC][PW] this step's pre-activations of my layers
  float* XF = PRE + NLC * PW;        // [XW]      the step's input x, fp32
  float* BRS = XF + XW;              // [NLC][R]  B_res
  float* SCL = BRS + NLC * R;        // [NLC][3R] int8: row scales of W_cur (2R rows) and W_res (R)
  float* SSK = SCL + NLC * 3 * R;    // [S]       int8: row scales of the last layer's W_skip
  u16* XS = reinterpret_cast<u16*>(SSK + S);             // [2][NS][SR] x, split, by layer parity
  u16* HS = XS + 2 * NS * SR;                            // [NS][SR]    h, split
  u32x4* WSK = reinterpret_cast<u32x4*>(HS + NS * SR);   // [S/16][2][64] the last layer's W_skip tiles

  // wave w: row tile w of the tanh half and of the sigmoid half of W_cur, row tile w of W_res
  const int m0 = 16 * wave + 4 * quad;  // this lane's rows of x, h and the tanh half of a
  u32x4 wt[NLC][2], wg[NLC][2], wr[NLC][2];
#pragma unroll
  for (int l = 0; l < NLC; ++l) {
    const size_t j = (size_t)j0 + (l < nl ? l : 0);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const int col = 32 * kt + 8 * quad;
      wt[l][kt] = wfrag<I8>(g.w.w_cur, j * 2 * R + 16 * wave + n, R, col);
      wg[l][kt] = wfrag<I8>(g.w.w_cur, j * 2 * R + R + 16 * wave + n, R, col);
      wr[l][kt] = wfrag<I8>(g.w.w_res, j * R + 16 * wave + n, R, col);
    }
  }
  for (int i = tid; i < nl * R; i += NT) BRS[i] = g.w.b_res[(size_t)j0 * R + i];
  if constexpr (I8) {
    for (int i = tid; i < nl * 3 * R; i += NT) {
      const int l = i / (3 * R), m = i % (3 * R);
      SCL[i] = m < 2 * R ? g.w.s_cur[(size_t)(j0 + l) * 2 * R + m] : g.w.s_res[(size_t)(j0 + l) * R + (m - 2 * R)];
    }
  }
  if (tail) {
    for (int i = tid; i < (S / 16) * 2 * 64; i += NT) {
      const int ln = i & 63, kt = (i >> 6) & 1, rt = i >> 7;
      WSK[i] = wfrag<I8>(g.w.w_skip, (size_t)(L - 1) * S + 16 * rt + (ln & 15), R, 32 * kt + 8 * (ln >> 4));
    }
    if constexpr (I8)
      for (int i = tid; i < S; i += NT) SSK[i] = g.w.s_skip[(size_t)(L - 1) * S + i];
  }
  // history slot (t mod d_j), dilation and offset of each of my layers
  int slot[NLC], dil[NLC], hoff[NLC];
#pragma unroll
  for (int l = 0; l < NLC; ++l) {
    const int j = j0 + (l < nl ? l : 0);
    dil[l] = g.d.dil[j];
    hoff[l] = g.d.hoff[j];
    slot[l] = (int)(tg0 % dil[l]);
  }
  __syncthreads();

  const int ot = wave * TW + (quad * NS + sn) * 4;  // this lane's words of tile `wave` of a block
  const bool p0 = part == 0;                        // the lane that adds the fp32 terms before a fold
  float4 xr = make_float4(0.f, 0.f, 0.f, 0.f);      // x_{j-1}[t], rows m0 .. m0 + 3 of stream sn, fp32
  for (int64_t t = tg0; t < tg0 + T; ++t) {
    const unsigned tag = (unsigned)(t + 1);
    // the pre-activations of my layers (posted by their aux CUs during the previous step), then the
    // input x: from the previous chain CU, or for chain CU 0 the head's x0
    const unsigned pre_w = mbw + (unsigned)j0 * PW;
    poll_pairs<16, NT, 16>(
        g, rs, tid, nl * PW / 2, [&](int p) { return pre_w + 2 * p; },
        [&](int) { return tag; }, [&](int i, int, float v) { PRE[i] = v; }, sy);
    const unsigned x_w = mbw + g.off_x + (unsigned)c * XW;
    poll_pairs<XW / 2 / NT>(
        g, rs, tid, XW / 2, [&](int p) { return x_w + 2 * p; }, [&](int) { return tag; },
        [&](int i, int, float v) {
          XF[i] = v;
          split_into<NS>(XS, i, v);
        },
        sy);
    lds_barrier();
    if (sy.failed()) return;
    xr = *reinterpret_cast<const float4*>(XF + ot);
#pragma unroll
    for (int l = 0; l < NLC; ++l) {
      if (l < nl) {
        const int j = j0 + l;
        {
          // a = pre + W_cur x_{j-1}; h = tanh(a[rows]) sigmoid(a[R + rows])
          const float4 pt = *reinterpret_cast<const float4*>(PRE + l * PW + ot);
          const float4 pg = *reinterpret_cast<const float4*>(PRE + l * PW + 4 * TW + ot);
          f32x4 at = {0.f, 0.f, 0.f, 0.f}, ag = {0.f, 0.f, 0.f, 0.f};
          if (!I8 && p0) {
            at = f4(pt);
            ag = f4(pg);
          }
          prod2<PAIR>(at, ag, wt[l][0], wt[l][1], wg[l][0], wg[l][1], XS + (l & 1) * NS * SR + sn * SR, quad, part);
          if constexpr (PAIR) {
            at = fold8(at);
            ag = fold8(ag);
          }
          // x_{j-1}[t] goes into slot t mod d_j of layer j's history, which its aux CU reads at t + d_j
          u64* const hist = ring + ((size_t)hoff[l] + (size_t)slot[l] * R) * NS + ot;
          slot[l] = slot[l] + 1 == dil[l] ? 0 : slot[l] + 1;
          if constexpr (!PAIR) stw4(hist, xr, tag, lm(l));
          if constexpr (I8) {
            const float4 st = *reinterpret_cast<const float4*>(SCL + l * 3 * R + m0);
            const float4 sg = *reinterpret_cast<const float4*>(SCL + l * 3 * R + R + m0);
            at = f32x4{pt.x + st.x * at[0], pt.y + st.y * at[1], pt.z + st.z * at[2], pt.w + st.w * at[3]};
            ag = f32x4{pg.x + sg.x * ag[0], pg.y + sg.y * ag[1], pg.z + sg.z * ag[2], pg.w + sg.w * ag[3]};
          }
          const float4 h = gate4<AX, PAIR>(at, ag, part);
          put_split4<PAIR>(HS + sn * SR, m0, h, part);
          // h_j[t] -> the layer's aux CU (with paired columns lane n posts h, lane n + 8 the history row)
          u64* const hpost = mb + g.off_h + (size_t)j * XW + ot;
          if constexpr (PAIR) stw4(p0 ? hpost : hist, p0 ? h : xr, tag, lm(l));
          else stw4(hpost, h, tag, lm(l));
        }
        lds_barrier();
        if (!(lastc && l == nl - 1)) {  // j < L - 1: x_l feeds nothing
          // x_j = x_{j-1} + W_res h + B_res
          const float4 br = *reinterpret_cast<const float4*>(BRS + l * R + m0);
          f32x4 acc = {0.f, 0.f, 0.f, 0.f};
          if (!I8 && p0) acc = f32x4{xr.x + br.x, xr.y + br.y, xr.z + br.z, xr.w + br.w};
          acc = prod1<PAIR>(acc, wr[l][0], wr[l][1], HS + sn * SR, quad, part);
          if constexpr (PAIR) acc = fold8(acc);
          if constexpr (I8) {
            const float4 sr = *reinterpret_cast<const float4*>(SCL + l * 3 * R + 2 * R + m0);
            xr = make_float4(xr.x + br.x + sr.x * acc[0], xr.y + br.y + sr.y * acc[1], xr.z + br.z + sr.z * acc[2],
                             xr.w + br.w + sr.w * acc[3]);
          } else {
            xr = v4(acc);
          }
          put_split4<PAIR>(XS + ((l + 1) & 1) * NS * SR + sn * SR, m0, xr, part);
          if (l == nl - 1 && !lastc) {
            // x of my last layer -> the next chain CU
            post4<PAIR>(mb + g.off_x + (size_t)(c + 1) * XW + ot, xr, tag, lm(16), part);
          }
          lds_barrier();
        }
      }
    }
    if (tail) {
      // the last layer's skip projection W_skip h_{l-1} (h is in HS): row tiles KS wave .. + KS - 1
#pragma unroll
      for (int k = 0; k < KS; ++k) {
        const int rt = KS * wave + k;
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        const u16* hs = HS + sn * SR;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          const u32x4 w = WSK[(rt * 2 + kt) * 64 + lane];
          if constexpr (PAIR) {
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, w),
                                                         *reinterpret_cast<const bf16x8*>(hs + part * R + 32 * kt + 8 * quad),
                                                         acc, 0, 0, 0);
          } else {
            acc = mfma_row<R>(w, hs, 32 * kt + 8 * quad, acc);
          }
        }
        if constexpr (PAIR) acc = fold8(acc);
        if constexpr (I8) {
          const float4 s4 = *reinterpret_cast<const float4*>(SSK + rt * 16 + 4 * quad);
          acc = f32x4{s4.x * acc[0], s4.y * acc[1], s4.z * acc[2], s4.w * acc[3]};
        }
        post4<PAIR>(mb + g.off_qtail + rt * TW + (quad * NS + sn) * 4, v4(acc), tag,
                    lm(17), part);
      }
      lds_barrier();  // HS is rewritten in the next step's first layer
    }
  }
}

// ------------------------------------------------------------------------------------------
// aux CU: layers ja .. ja + nl - 1
// ------------------------------------------------------------------------------------------
// NLK > 0: this CU holds NLK layers, a compile-time count; NLK = 0: read at run time.
template <int S, bool AX, bool I8, bool PAIR, int NLK, class LM>
__device__ __forceinline__ void mc_aux(const WnChainArgs& g, const int ai, const int rep, float* dyn, Sync sy,
                                       const int64_t tg0, const LM lm) {
  using C = Cols<PAIR>;
  constexpr int NS = C::NS, XW = C::XW, PW = C::PW, TW = C::TW;
  constexpr int KS = S / 64;  // row tiles of W_skip per wave
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 15, quad = lane >> 4;
  const int sn = PAIR ? (n & 7) : n, part = PAIR ? (n >> 3) : 0;
  const int L = g.d.L, T = g.io.T;
  const int ja = g.aux_begin[ai], nl = NLK > 0 ? NLK : g.aux_begin[ai + 1] - ja;  // nl <= NLA
  // layers whose skip projection this CU computes (the last layer's runs on the last chain CU)
  const int nsk = (g.tail_on_chain && ja + nl == L) ? nl - 1 : nl;
  const int b0 = rep * g.G, ns = min(g.G, g.io.B - b0);
  u64* const mb = g.mb + (size_t)rep * g.mb_words;
  const u64* const ring = g.ring + (size_t)rep * g.d.hist_len * NS;
  const wrsrc rs = tagged_region(g);
  const unsigned mbw = (unsigned)(mb - g.ring), rgw = (unsigned)(ring - g.ring);
  float* CD = dyn;                 // [NLA][PW]  conditioning rows L[b, t + 1, j], tile order
  float* BG = CD + NLA * PW;       // [NLA][2R]  B (gate bias)
  float* SP = BG + NLA * 2 * R;    // [NLA][2R]  int8: row scales of W_prev
  float* SK = SP + NLA * 2 * R;    // [NLA][S]   int8: row scales of W_skip
  u16* HX = reinterpret_cast<u16*>(SK + NLA * S);  // [NLA][NS][SR] history rows x_{j-1}[t + 1 - d], split
  u16* HH = HX + NLA * NS * SR;                    // [NLA][NS][SR] h_j[t], split
  __shared__ unsigned long long s_hb[NLA];         // stage(): history block (word offset) of each polled layer
  __shared__ unsigned s_ht[NLA];                   //          and the tag it must carry
  __shared__ int s_hl[NLA], s_nh;                  //          and its layer index; how many

  // wave v: row tiles 2v, 2v + 1 of W_prev and KS v .. KS v + KS - 1 of W_skip
  u32x4 wp[NLA][2][2], wk[NLA][KS][2];
  int dl[NLA], ho[NLA];
#pragma unroll
  for (int l = 0; l < NLA; ++l) {
    const size_t j = (size_t)ja + (l < nl ? l : 0);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const int col = 32 * kt + 8 * quad;
#pragma unroll
      for (int k = 0; k < 2; ++k) wp[l][k][kt] = wfrag<I8>(g.w.w_prev, j * 2 * R + 16 * (2 * wave + k) + n, R, col);
#pragma unroll
      for (int k = 0; k < KS; ++k) wk[l][k][kt] = wfrag<I8>(g.w.w_skip, j * S + 16 * (KS * wave + k) + n, R, col);
    }
    dl[l] = g.d.dil[ja + (l < nl ? l : 0)];
    ho[l] = g.d.hoff[ja + (l < nl ? l : 0)];
  }
  for (int i = tid; i < nl * 2 * R; i += NT) BG[i] = g.w.b_gate[(size_t)ja * 2 * R + i];
  if constexpr (I8) {
    for (int i = tid; i < nl * 2 * R; i += NT) SP[i] = g.w.s_prev[(size_t)ja * 2 * R + i];
    for (int i = tid; i < nl * S; i += NT) SK[i] = g.w.s_skip[(size_t)ja * S + i];
  }
  for (int i = tid; i < NLA * PW; i += NT) CD[i] = 0.f;  // padding columns stay zero
  __syncthreads();

  // this lane's words of row tile rt of a block
  auto lot = [&](int rt) { return rt * TW + (quad * NS + sn) * 4; };
  // Conditioning rows of step ts, CQ float4s per thread and layer: piece q holds rows 4 (q mod 32) ..
  // + 3 of column q / 32, i.e. tile (q mod 32) / 4, run (q mod 4, q / 32).  Columns past the
  // replica's streams read the last stream's row and never store it.
  constexpr int CQ = 2 * R * NS / 4 / NT;
  size_t cq_src[CQ];
  int cq_dst[CQ];
  bool cq_on[CQ];
#pragma unroll
  for (int k = 0; k < CQ; ++k) {
    const int q = tid + NT * k, cn = q >> 5, e4 = q & 31;
    cq_on[k] = cn < ns;
    cq_src[k] = (size_t)min(cn, ns - 1) * T * L * 2 * R + 4 * e4;  // + (step L + layer) 2R
    cq_dst[k] = (e4 >> 2) * TW + ((e4 & 3) * NS + cn) * 4;
  }
  const float* const cbase = g.io.cond + (size_t)b0 * T * L * 2 * R;
  // Stage the inputs of pre_j[ts]: the conditioning rows of every layer and the history rows
  // x_{j-1}[ts - d] of the layers with d >= 2 (final once step ts - d is over), or of every layer
  // (all_hist, the call's first step).  With d = 1 the row is written during step ts - 1 and is
  // waited for together with h_j.
  auto stage = [&](int64_t ts, bool all_hist) __attribute__((always_inline)) {
    // each row is read once: non-temporal loads, so that the stream does not evict the mailboxes
    f32x4 cq[NLA][CQ];
    const float* crow = cbase + ((size_t)(ts - tg0) * L + ja) * 2 * R;
#pragma unroll
    for (int l = 0; l < NLA; ++l)
#pragma unroll
      for (int k = 0; k < CQ; ++k)
        cq[l][k] = l < nl ? __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(crow + cq_src[k] + l * 2 * R))
                          : f32x4{0.f, 0.f, 0.f, 0.f};
    if (tid == 0) {
      int nh = 0;
#pragma unroll
      for (int l = 0; l < NLA; ++l) {
        if (l < nl && (all_hist || dl[l] >= 2)) {
          const int d = dl[l];
          const int64_t sl = ts % d;
          s_hb[nh] = ((unsigned long long)ho[l] + (unsigned long long)sl * R) * NS;
          s_ht[nh] = ts - d >= 0 ? (unsigned)(ts - d + 1) : 0u;
          s_hl[nh] = l;
          ++nh;
        }
      }
      s_nh = nh;
    }
    __syncthreads();
    poll_pairs<4, NT, 16>(
        g, rs, tid, s_nh * XW / 2, [&](int p) { return rgw + (unsigned)s_hb[(2 * p) / XW] + (2 * p) % XW; },
        [&](int i) { return s_ht[i / XW]; },
        [&](int i, int, float v) { split_into<NS>(HX + s_hl[i / XW] * NS * SR, i % XW, v); }, sy);
#pragma unroll
    for (int l = 0; l < NLA; ++l)
#pragma unroll
      for (int k = 0; k < CQ; ++k)
        if (l < nl && cq_on[k]) *reinterpret_cast<f32x4*>(CD + l * PW + cq_dst[k]) = cq[l][k];
    lds_barrier();
  };
  // pre_j[ts] = W_prev x_{j-1}[ts - d] + B + L[b, ts, j] of row tiles 2 wave, 2 wave + 1, j = ja + l,
  // posted with tag ts + 1
  auto post_pre = [&](int l, int64_t ts) __attribute__((always_inline)) {
    const unsigned tg = (unsigned)(ts + 1);
    const bool loc = lm(l);
    f32x4 pa[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
    prod2<PAIR>(pa[0], pa[1], wp[l][0][0], wp[l][0][1], wp[l][1][0], wp[l][1][1], HX + l * NS * SR + sn * SR, quad,
                part);
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int rt = 2 * wave + k;
      const f32x4 acc = PAIR ? fold8(pa[k]) : pa[k];
      const int mr = 16 * rt + 4 * quad;
      const float4 b = *reinterpret_cast<const float4*>(BG + l * 2 * R + mr);
      const float4 cd = *reinterpret_cast<const float4*>(CD + l * PW + lot(rt));
      float4 v;
      if constexpr (I8) {
        const float4 s4 = *reinterpret_cast<const float4*>(SP + l * 2 * R + mr);
        v = make_float4(s4.x * acc[0] + b.x + cd.x, s4.y * acc[1] + b.y + cd.y, s4.z * acc[2] + b.z + cd.z,
                        s4.w * acc[3] + b.w + cd.w);
      } else {
        v = make_float4(acc[0] + b.x + cd.x, acc[1] + b.y + cd.y, acc[2] + b.z + cd.z, acc[3] + b.w + cd.w);
      }
      post4<PAIR>(mb + (size_t)(ja + l) * PW + lot(rt), v, tg, loc, part);
    }
  };

  stage(tg0, true);
  if (sy.failed()) return;
#pragma unroll
  for (int l = 0; l < NLA; ++l)
    if (l < nl) post_pre(l, tg0);
  for (int64_t t = tg0; t < tg0 + T; ++t) {
    const bool more = t + 1 < tg0 + T;
    const unsigned tag = (unsigned)(t + 1);
    // A host abort request, read every WN_ABORT_CHECK steps by the replica's first aux CU, which works
    // a step ahead of the chain (the read's PCIe round trip stays off the critical path); every other
    // role sees the status word in its next wait and leaves too.
    if (ai == 0 && tid == 0 && ((t - tg0) & (WN_ABORT_CHECK - 1)) == 0 && abort_requested(g.io.abort_flag)) {
      atomicCAS(g.status, 0, (int)WN_EABORTED);
      *sy.flag = 1;
    }
    lds_barrier();
    if (sy.failed()) return;
    if (more) {
      stage(t + 1, false);
      if (sy.failed()) return;
    }
    // the skip sum of my layers (with paired columns unfolded until it is posted: the fold is linear)
    f32x4 qs[KS];
#pragma unroll
    for (int k = 0; k < KS; ++k) qs[k] = f32x4{0.f, 0.f, 0.f, 0.f};
    // The words each layer waits for: h_j[t] and, with d = 1, the history row x_{j-1}[t] that
    // pre_j[t + 1] reads.  Once h_j[t] is in, the chain has consumed pre_j[t], so posting pre_j[t + 1]
    // cannot overwrite a slot it has yet to read.  The next layer's loads are issued before this
    // layer's products, so their round trip overlaps them.
    auto lw_n = [&](int l) { return (more && dl[l] == 1) ? XW : XW / 2; };  // pairs
    auto lw_word = [&](int l) {
      const unsigned hw = mbw + g.off_h + (unsigned)(ja + l) * XW;
      const unsigned xw = rgw + (unsigned)ho[l] * NS;
      return [=](int p) { return 2 * p < XW ? hw + 2 * p : xw + (2 * p - XW); };
    };
    u32x4 pw[XW / NT];
    pairs_start(pw, rs, tid, lw_n(0), lw_word(0));
#pragma unroll
    for (int l = 0; l < NLA; ++l) {
      if (l < nl) {
        pairs_finish(
            g, pw, rs, tid, lw_n(l), lw_word(l), [&](int) { return tag; },
            [&](int i, int, float v) {
              if (i < XW) split_into<NS>(HH + l * NS * SR, i, v);
              else split_into<NS>(HX + l * NS * SR, i - XW, v);
            },
            sy);
        lds_barrier();
        if (sy.failed()) return;
        const bool posts = l == nsk - 1, more_l = l + 1 < NLA && l + 1 < nl;
        if (more_l) pairs_start(pw, rs, tid, lw_n(l + 1), lw_word(l + 1));
        if (l < nsk) {
          // q += W_skip h_j, row tiles KS wave ..
          const u16* hh = HH + l * NS * SR + sn * SR;
          f32x4 sa[KS];
#pragma unroll
          for (int k = 0; k < KS; ++k) sa[k] = I8 ? f32x4{0.f, 0.f, 0.f, 0.f} : qs[k];
#pragma unroll
          for (int k = 0; k < KS; k += 2)
            prod2<PAIR>(sa[k], sa[k + 1], wk[l][k][0], wk[l][k][1], wk[l][k + 1][0], wk[l][k + 1][1], hh, quad, part);
#pragma unroll
          for (int k = 0; k < KS; ++k) {
            const f32x4 acc = sa[k];
            if constexpr (I8) {
              const float4 s4 = *reinterpret_cast<const float4*>(SK + l * S + (KS * wave + k) * 16 + 4 * quad);
              qs[k] = f32x4{qs[k][0] + s4.x * acc[0], qs[k][1] + s4.y * acc[1], qs[k][2] + s4.z * acc[2],
                            qs[k][3] + s4.w * acc[3]};
            } else {
              qs[k] = acc;
            }
          }
          // the partial goes out as soon as its last layer is in (the head sums the partials)
          if (posts) {
            if constexpr (PAIR) {
#pragma unroll
              for (int k = 0; k < KS; ++k) qs[k] = fold8(qs[k]);
            }
            const bool loc = lm(16);
#pragma unroll
            for (int k = 0; k < KS; ++k)
              post4<PAIR>(mb + g.off_q + (size_t)ai * S * NS + lot(KS * wave + k), v4(qs[k]), tag, loc,
                          part);
          }
        }
      }
    }
    // the next step's pre-activations, once the skip partial is out (each layer's h_j[t] is in)
    if (more) {
#pragma unroll
      for (int l = 0; l < NLA; ++l)
        if (l < nl) post_pre(l, t + 1);
    }
    lds_barrier();
  }
}

// The head's products for the four row tiles of a wave: acc[k] = W[k] z over K inputs, row = this
// lane's part (hi or lo) of its stream's split row; folded.
template <int KT>
__device__ __forceinline__ void head_products(f32x4 (&acc)[4], const u32x4 (&w)[4][KT], const u16* row, int quad) {
  static_assert(KT % 4 == 0, "128-input blocks");
#pragma unroll
  for (int k = 0; k < 4; ++k) acc[k] = f32x4{0.f, 0.f, 0.f, 0.f};
  u32x4 xb[KT];  // every B operand first (one LDS round trip), then the MFMA blocks back to back
#pragma unroll
  for (int q = 0; q < KT; ++q) xb[q] = ld16(row + 32 * q + 8 * quad);
#pragma unroll
  for (int kb = 0; kb < KT; kb += 4) {
    const u32x4 x[4] = {xb[kb], xb[kb + 1], xb[kb + 2], xb[kb + 3]};
#pragma unroll
    for (int k = 0; k < 4; k += 2) {
      const u32x4 wa[4] = {w[k][kb], w[k][kb + 1], w[k][kb + 2], w[k][kb + 3]};
      const u32x4 wb[4] = {w[k + 1][kb], w[k + 1][kb + 1], w[k + 1][kb + 2], w[k + 1][kb + 3]};
      mfma_k128_2p(acc[k], acc[k + 1], wa, wb, x);
    }
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) acc[k] = fold8(acc[k]);
}

// ------------------------------------------------------------------------------------------
// head CU hh: columns 8 hh .. 8 hh + 7 of the replica's tiles (8 streams): the skip sum, the two head
// layers, the draw and the next step's x0
// ------------------------------------------------------------------------------------------
template <int S, bool TF, bool AX, bool I8, bool PAIR, class LM>
__device__ __forceinline__ void mc_head(const WnChainArgs& g, const int hh, const int rep, float* dyn, Sync sy,
                                        const int64_t tg0, const LM lm) {
  using C = Cols<PAIR>;
  constexpr int NS = C::NS;
  constexpr int KTH = S / 32, KTO = A / 32;
  constexpr int SS = 2 * S + 8, SA = 2 * A + 8, PA = A + 4;
  constexpr int QW = S * NS;           // words of a skip partial
  constexpr int QP = S * HG / 2;       // pairs of a partial in my 8 columns
  constexpr int NQP = QP / NT;         // of them per thread
  constexpr int NQ = 2 * NQP;          // skip-sum entries per thread
  constexpr int HT = A / 16 / 4;       // row tiles of W_relu and of W_out per wave
  static_assert(HT == 4 && NQP == 4, "four row tiles per wave, four pairs per partial and thread");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 15, quad = lane >> 4, sn = n & 7, part = n >> 3;
  const bool wl = part == 0;  // the lane that stores its stream's results (lanes n, n + 8 hold the same)
  const int T = g.io.T;
  const int c0 = HG * hh;                              // my first column of the replica's tiles
  const int nrs = min(g.G, g.io.B - rep * g.G);        // streams of the replica
  const int ns = max(0, min(HG, nrs - c0));            // mine
  const int b0 = rep * g.G + c0;
  const bool e2 = g.w.embed_prev != nullptr;
  u64* const mb = g.mb + (size_t)rep * g.mb_words;
  const wrsrc rs = tagged_region(g);
  const unsigned mbw = (unsigned)(mb - g.ring);
  u16* ZS = reinterpret_cast<u16*>(dyn);               // [HG][SS] z_s, split
  u16* ZA = ZS + HG * SS;                              // [HG][SA] z_a, split
  float* LG = reinterpret_cast<float*>(ZA + HG * SA);  // [HG][PA] logits
  float* BSK = LG + HG * PA;  // [S] B_skip
  float* BRL = BSK + S;       // [A] B_relu
  float* BO = BRL + A;        // [A] B_out
  float* BE = BO + A;         // [R] B_embed
  float* SRL = BE + R;        // [A] int8: row scales of W_relu, W_out and the two embedding tables
  float* SO = SRL + A;
  float* SE = SO + A;
  float* SEP = SE + A;
  u16* EMB = reinterpret_cast<u16*>(SEP + A);  // [A][R] the table of y_{t-1}: bf16, or int8 codes
  u16* EMBP = EMB + A * R;                     // [A][R] the table of y_{t-2} (two taps)
  __shared__ int s_y[HG], s_y2[HG];            // y_{t-1}, y_{t-2} (-1 before the first input)
  __shared__ float s_u[HG];
  __shared__ int s_yin[HG];

  // wave v: row tiles HT v .. HT v + HT - 1 of W_relu and of W_out
  u32x4 w1[HT][KTH], w2[HT][KTO];
#pragma unroll
  for (int k = 0; k < HT; ++k) {
    const size_t row = 16 * (HT * wave + k) + n;
#pragma unroll
    for (int kt = 0; kt < KTH; ++kt) w1[k][kt] = wfrag<I8>(g.w.w_relu, row, S, 32 * kt + 8 * quad);
#pragma unroll
    for (int kt = 0; kt < KTO; ++kt) w2[k][kt] = wfrag<I8>(g.w.w_out, row, A, 32 * kt + 8 * quad);
  }
  for (int i = tid; i < S; i += NT) BSK[i] = g.w.b_skip[i];
  for (int i = tid; i < A; i += NT) {
    BRL[i] = g.w.b_relu[i];
    BO[i] = g.w.b_out[i];
    if constexpr (I8) {
      SRL[i] = g.w.s_relu[i];
      SO[i] = g.w.s_out[i];
      SE[i] = g.w.s_embed[i];
      SEP[i] = e2 ? g.w.s_embed_prev[i] : 0.f;
    }
  }
  for (int i = tid; i < R; i += NT) BE[i] = g.w.b_embed[i];
  {
    // the tables as 32-bit words (bf16 pairs, or int8 quadruples)
    constexpr int TW = I8 ? A * R / 4 : A * R / 2;
    const unsigned* e = static_cast<const unsigned*>(g.w.embed);
    for (int i = tid; i < TW; i += NT) reinterpret_cast<unsigned*>(EMB)[i] = e[i];
    if (e2) {
      const unsigned* ep = static_cast<const unsigned*>(g.w.embed_prev);
      for (int i = tid; i < TW; i += NT) reinterpret_cast<unsigned*>(EMBP)[i] = ep[i];
    }
  }
  for (int i = tid; i < HG * SS; i += NT) ZS[i] = 0;  // padding streams' rows stay finite
  if (tid < HG) {
    int y = 0, y2 = -1;
    if (tid < ns) {
      const int64_t* st = g.state + WN_STATE_WORDS * (size_t)(b0 + tid);
      y = g.io.reset ? g.io.init_sample : (int)st[1];
      y2 = g.io.reset ? -1 : (int)st[2];
    }
    s_y[tid] = y < 0 ? 0 : (y > A - 1 ? A - 1 : y);
    s_y2[tid] = y2 < 0 ? -1 : (y2 > A - 1 ? A - 1 : y2);
  }
  __syncthreads();
  // row k of a table's entry y
  auto emb = [&](const u16* tab, const float* sc, int y, int k) __attribute__((always_inline)) -> float {
    if constexpr (I8) return (float)reinterpret_cast<const signed char*>(tab)[y * R + k] * sc[y];
    else return bf16_val(tab[y * R + k]);
  };
  // x0 of the call's first step in my columns (padding columns get zeros)
  for (int i = tid; i < R * HG; i += NT) {
    const int m = i >> 3, q = i & 7;
    float v = 0.f;
    if (q < ns) {
      v = emb(EMB, SE, s_y[q], m) + BE[m];
      if (e2 && s_y2[q] >= 0) v += emb(EMBP, SEP, s_y2[q], m);
    }
    stw(mb + g.off_x + tpos<NS>(m, c0 + q), pack(v, (unsigned)(tg0 + 1)), lm(0));
  }

  // skip partials per step: one from each aux CU that posts one, then the last layer's from the last
  // chain CU, summed in that order
  const int np = g.naux_q + (g.tail_on_chain ? 1 : 0);
  auto part_word = [&](int p) -> unsigned {
    if (p < g.naux_q) return mbw + g.off_q + (unsigned)p * QW;
    return mbw + g.off_qtail;
  };
  // pair r (0 .. QP - 1) of a partial in my columns: with paired columns the whole partial; else tile
  // r / 64, run (i / 8, c0 + i mod 8) with i = (r / 2) mod 32, words 2 (r mod 2), + 1 of that run
  auto pair_off = [&](int r) {
    if constexpr (PAIR) return (unsigned)(2 * r);
    const int i = (r >> 1) & 31;
    return (unsigned)((((r >> 6) << 6) + (i & 7) + c0 + ((i >> 3) << 4)) * 4 + 2 * (r & 1));
  };
  for (int64_t t = tg0; t < tg0 + T; ++t) {
    const unsigned tag = (unsigned)(t + 1);
    const bool more = t + 1 < tg0 + T;
    // this step's uniform (or teacher-forced sample) of each stream, staged after the wait below
    float uv = 0.f;
    int yv = 0;
    if (tid < ns) {
      const size_t at = (size_t)(b0 + tid) * T + (size_t)(t - tg0);
      if constexpr (TF) yv = g.io.y_in[at];
      else uv = g.io.u[at];
    }
    // the skip partials of the step, my columns, in batches of up to three partials: the early ones
    // while the chain still runs, then the last three (the aux CUs of the last layers and the chain's
    // tail).  In a batch, pair p = tid + NT k is pair tid + NT (k mod NQP) of partial k / NQP, entries
    // 2 (k mod NQP) (+ 1) of this thread, the same position in every partial.
    float qa[NQ];
#pragma unroll
    for (int e = 0; e < NQ; ++e) qa[e] = 0.f;
    for (int p0 = 0; p0 < np;) {
      const int p1 = np - p0 <= 3 ? np : min(p0 + 3, np - 3);
      constexpr int KP = 3 * NQP;
      u32x4 w[KP];
      auto word = [&](int p) { return part_word(p0 + p / QP) + pair_off(p % QP); };
      pairs_start<KP>(w, rs, tid, (p1 - p0) * QP, word);
      pairs_finish<KP>(
          g, w, rs, tid, (p1 - p0) * QP, word, [&](int) { return tag; }, [&](int, int q, float v) { qa[q % NQ] += v; },
          sy);
      if (sy.failed()) break;
      p0 = p1;
    }
    if (tid < HG) {
      if constexpr (TF) s_yin[tid] = yv < 0 ? 0 : (yv > A - 1 ? A - 1 : yv);
      else s_u[tid] = uv;
    }
    // z_s = relu(B_skip + sum of the partials); the two words of a pair are rows m, m + 1 (m even) of
    // one column, stored as one 32-bit word of hi parts and one of lo parts
#pragma unroll
    for (int e = 0; e < NQ; e += 2) {
      const unsigned wo = pair_off(tid + NT * (e >> 1));
      const int m = trow<NS>((int)wo), q = tcol<NS>((int)wo) - c0;
      const float z0 = fmaxf(qa[e] + BSK[m], 0.f), z1 = fmaxf(qa[e + 1] + BSK[m + 1], 0.f);
      const unsigned hi = pack_bf16(z0, z1);
      const unsigned lo = pack_bf16(z0 - low_bf16(hi), z1 - high_bf16(hi));
      *reinterpret_cast<unsigned*>(ZS + q * SS + m) = hi;
      *reinterpret_cast<unsigned*>(ZS + q * SS + S + m) = lo;
    }
    lds_barrier();
    if (sy.failed()) return;
    // z_a = relu(W_relu z_s + B_relu)
    {
      f32x4 za[HT];
      head_products<KTH>(za, w1, ZS + sn * SS + part * S, quad);
#pragma unroll
      for (int k = 0; k < HT; ++k) {
        f32x4 acc = za[k];
        const int mr = 16 * (HT * wave + k) + 4 * quad;
        const float4 b = *reinterpret_cast<const float4*>(BRL + mr);
        if constexpr (I8) {
          const float4 s4 = *reinterpret_cast<const float4*>(SRL + mr);
          acc = f32x4{s4.x * acc[0], s4.y * acc[1], s4.z * acc[2], s4.w * acc[3]};
        }
        if (wl)
          store_split4<A>(ZA + sn * SA, mr,
                          make_float4(fmaxf(acc[0] + b.x, 0.f), fmaxf(acc[1] + b.y, 0.f), fmaxf(acc[2] + b.z, 0.f),
                                      fmaxf(acc[3] + b.w, 0.f)));
      }
    }
    lds_barrier();
    // logits = W_out z_a + B_out
    {
      f32x4 lo[HT];
      head_products<KTO>(lo, w2, ZA + sn * SA + part * A, quad);
#pragma unroll
      for (int k = 0; k < HT; ++k) {
        f32x4 acc = lo[k];
        const int mr = 16 * (HT * wave + k) + 4 * quad;
        const float4 b = *reinterpret_cast<const float4*>(BO + mr);
        if constexpr (I8) {
          const float4 s4 = *reinterpret_cast<const float4*>(SO + mr);
          acc = f32x4{s4.x * acc[0], s4.y * acc[1], s4.z * acc[2], s4.w * acc[3]};
        }
        if (wl)
          *reinterpret_cast<float4*>(LG + sn * PA + mr) = make_float4(acc[0] + b.x, acc[1] + b.y, acc[2] + b.z, acc[3] + b.w);
      }
    }
    lds_barrier();
    // the draws of my streams HG / 4 wave .. (both at once, so that their steps interleave; a padding
    // stream's draw is made and dropped), then their x0 of the next step (row = lane)
    int ys[HG / 4];
    if constexpr (TF) {
#pragma unroll
      for (int k = 0; k < HG / 4; ++k) ys[k] = s_yin[(HG / 4) * wave + k];
    } else if (g.io.smode == WN_DRAW_DIRECT || g.io.smode == WN_DRAW_TEMPERATURE) {
      float4 lv[HG / 4];
      float uq[HG / 4];
#pragma unroll
      for (int k = 0; k < HG / 4; ++k) {
        const int q = (HG / 4) * wave + k;
        lv[k] = *reinterpret_cast<const float4*>(LG + q * PA + 4 * lane);
        uq[k] = s_u[q];
      }
      wave_draw_cdf<AX>(lv, uq, g.io.smode == WN_DRAW_TEMPERATURE ? g.io.inv_t : 1.0f, ys);
    } else {
#pragma unroll
      for (int k = 0; k < HG / 4; ++k) {
        const int q = (HG / 4) * wave + k;
        const float4 lv = *reinterpret_cast<const float4*>(LG + q * PA + 4 * lane);
        ys[k] = wave_draw<AX>(lv, s_u[q], g.io.smode, g.io.inv_t, g.io.top_k, lane);
      }
    }
#pragma unroll
    for (int k = 0; k < HG / 4; ++k) {
      const int q = (HG / 4) * wave + k;
      const int y = q < ns ? ys[k] : 0;
      if (q < ns) {
        const size_t at = (size_t)(b0 + q) * T + (size_t)(t - tg0);
        if constexpr (TF) reinterpret_cast<float4*>(g.io.logits + at * A)[lane] = *reinterpret_cast<const float4*>(LG + q * PA + 4 * lane);
        else if (lane == 0) g.io.y_out[at] = y;
      }
      const int yp = s_y[q];
      if (more) {
        float v = 0.f;
        if (q < ns) {
          v = emb(EMB, SE, y, lane) + BE[lane];
          if (e2) v += emb(EMBP, SEP, yp, lane);
        }
        stw(mb + g.off_x + tpos<NS>(lane, c0 + q), pack(v, tag + 1), lm(0));
      }
      if (lane == 0 && q < ns) {
        s_y2[q] = yp;
        s_y[q] = y;
      }
    }
    lds_barrier();
  }
  // after a timeout or an abort the state stays as it was (the next call must start from zero)
  if (!sy.failed() && tid < ns) {
    int64_t* st = g.state + WN_STATE_WORDS * (size_t)(b0 + tid);
    st[0] = tg0 + T;
    st[1] = s_y[tid];
    st[2] = s_y2[tid];
  }
}


template <int S, bool TF, bool AX, bool I8, bool PAIR>
__global__ __launch_bounds__(NT, 1) void wn_mchain_kernel(const WnChainArgs ga) {
  using C = Cols<PAIR>;
  // The argument block is read in place, through the kernel-argument segment: used as the by-value
  // parameter, the compiler copies all of it to scratch memory once the roles index it at run time.
#if __HIP_DEVICE_COMPILE__
  const WnChainArgs& g = *(const WnChainArgs*)__builtin_amdgcn_kernarg_segment_ptr();
#else
  const WnChainArgs& g = ga;  // the host pass only checks the body
#endif
  (void)ga;
  extern __shared__ __align__(16) float dyn[];
  __shared__ int s_abort;
  __shared__ unsigned char s_xcd[WN_MAX_CHAIN + 2 + WN_MAX_LAYERS];
  __shared__ unsigned char s_cof[WN_MAX_LAYERS], s_aof[WN_MAX_LAYERS];
  __shared__ int s_me;
  const int rb = g.role_of_block[blockIdx.x];
  if (rb == 0xffff) return;
  const int per = g.nch + C::NH + g.naux;  // roles of a replica: chain CUs, head CUs, aux CUs
  const int k = rb / per, role = rb - k * per;
  const int head = g.nch, aux0 = g.nch + C::NH;
  if (threadIdx.x == 0) s_abort = 0;
  // Which of this block's posts go to a reader on its own XCD in this launch: bit l of a chain CU for
  // the aux CU of its layer l (h and the history rows), bit 16 for the next chain CU, bit 17 for the
  // head CUs; bit l of an aux CU for the chain CU of its layer l, bit 16 for the head CUs; bit 0 of a
  // head CU for chain CU 0.  The map is read at the launch (grid_meet).  When every role of the
  // replica runs on the block's XCD, the roles run their all-local build.
  unsigned lm = 0;
  bool all_local = false;
  if (g.local_posts) {
    if (grid_meet(g.xmap, g.n_active, g.spin_limit, g.status, &s_me) < 0) return;  // WN_ETIMEOUT is in the status word
    for (int b = threadIdx.x; b < WN_CHAIN_GRID; b += NT) {
      const int r = g.role_of_block[b];
      if (r != 0xffff && r / per == k) s_xcd[r - k * per] = (unsigned char)ldw(g.xmap + b);
    }
    // the chain CU and the aux CU of every layer
    for (int c = threadIdx.x; c < g.nch; c += NT)
      for (int j = g.layer_begin[c]; j < g.layer_begin[c + 1]; ++j) s_cof[j] = (unsigned char)c;
    for (int a = threadIdx.x; a < g.naux; a += NT)
      for (int j = g.aux_begin[a]; j < g.aux_begin[a + 1]; ++j) s_aof[j] = (unsigned char)a;
    __syncthreads();
    const int me = s_me;
    auto same = [&](int r) { return s_xcd[r] == me; };
    const bool heads_same = same(head) && (C::NH == 1 || same(head + 1));
    all_local = true;
    for (int r = 0; r < per; ++r) all_local = all_local && same(r);
    if (role < head) {
      const int j0 = g.layer_begin[role], nl = g.layer_begin[role + 1] - j0;
      for (int l = 0; l < nl; ++l) lm |= (unsigned)same(aux0 + s_aof[j0 + l]) << l;
      if (role + 1 < g.nch) lm |= (unsigned)same(role + 1) << 16;
      lm |= (unsigned)heads_same << 17;
    } else if (role < aux0) {
      lm = same(0);
    } else {
      const int ai = role - aux0, ja = g.aux_begin[ai];
      for (int j = ja; j < g.aux_begin[ai + 1]; ++j) lm |= (unsigned)same(s_cof[j]) << (j - ja);
      lm |= (unsigned)heads_same << 16;
    }
  }
  // where this call starts: from zero, or where the previous call on this workspace stopped (the
  // head rewrites the state only after the whole call, when every role has started)
  const int64_t tg0 = g.io.reset ? 0 : g.state[WN_STATE_WORDS * (size_t)(k * g.G)];
  __syncthreads();
  Sync sy{&s_abort};
  auto run = [&](auto loc) {
    if (role < head) {
      // the all-local build also fixes the layer count of the common chain CUs at compile time
      const int nl = g.layer_begin[role + 1] - g.layer_begin[role];
      constexpr bool FIX = std::is_same<decltype(loc), Local<true>>::value;
      constexpr int K1 = FIX ? NLC : 0, K2 = (FIX && NLC > 1) ? NLC - 1 : 0;
      if (K1 > 0 && nl == K1) mc_chain<S, AX, I8, PAIR, K1>(g, role, k, dyn, sy, tg0, loc);
      else if (K2 > 0 && nl == K2) mc_chain<S, AX, I8, PAIR, K2>(g, role, k, dyn, sy, tg0, loc);
      else mc_chain<S, AX, I8, PAIR, 0>(g, role, k, dyn, sy, tg0, loc);
    }
    else if (role < aux0) mc_head<S, TF, AX, I8, PAIR>(g, role - head, k, dyn, sy, tg0, loc);
    else {
      // and the aux CUs' runs of the default l = 20 plan (5, 5, 5, 3, 2 layers)
      const int ai = role - aux0, na = g.aux_begin[ai + 1] - g.aux_begin[ai];
      constexpr bool FIX = std::is_same<decltype(loc), Local<true>>::value;
      constexpr int A1 = FIX ? NLA : 0, A2 = FIX ? 3 : 0, A3 = FIX ? 2 : 0;
      if (A1 > 0 && na == A1) mc_aux<S, AX, I8, PAIR, A1>(g, ai, k, dyn, sy, tg0, loc);
      else if (A2 > 0 && na == A2) mc_aux<S, AX, I8, PAIR, A2>(g, ai, k, dyn, sy, tg0, loc);
      else if (A3 > 0 && na == A3) mc_aux<S, AX, I8, PAIR, A3>(g, ai, k, dyn, sy, tg0, loc);
      else mc_aux<S, AX, I8, PAIR, 0>(g, ai, k, dyn, sy, tg0, loc);
    }
  };
  if (all_local) run(Local<true>{lm});
  else run(Local<false>{lm});
}

// Layers of each chain CU: runs of at most NLC, as even as possible.
int mchain_split(int L, int* layer_begin) {
  const int nch = (L + NLC - 1) / NLC;
  if (nch > WN_MAX_CHAIN) return nch;
  const int base = L / nch, extra = L % nch;
  layer_begin[0] = 0;
  for (int c = 0; c < nch; ++c) layer_begin[c + 1] = layer_begin[c] + base + (c < extra ? 1 : 0);
  return nch;
}

// Layers of each aux CU: uniform runs of nla, or front-loaded runs (the last two hold 2 and 3 layers,
// the others NLA, the first the remainder), so that the aux CUs of the last layers, which trail the
// chain by the most, have the fewest layers to catch up on.  Returns the number of aux CUs.
int aux_split(int L, int nla, bool front, int* begin) {
  int sizes[WN_MAX_LAYERS];
  int n = 0;
  if (front) {
    for (int rem = L; rem > 0; ++n) {
      sizes[n] = std::min(n == 0 ? 2 : (n == 1 ? 3 : NLA), rem);
      rem -= sizes[n];
    }
    std::reverse(sizes, sizes + n);
  } else {
    for (int j = 0; j < L; j += nla) sizes[n++] = std::min(nla, L - j);
  }
  begin[0] = 0;
  for (int a = 0; a < n; ++a) begin[a + 1] = begin[a] + sizes[a];
  return n;
}

constexpr size_t kMaxLds = 160 * 1024;

template <int S>
size_t mchain_lds() {
  return std::max({chain_lds<false>(S), chain_lds<true>(S), aux_lds<false>(S), aux_lds<true>(S), head_lds(S)});
}

template <int S, bool PAIR>
const void* mchain_kernel(bool teacher, bool ax, bool i8) {
  if (teacher) {
    if (i8) return ax ? reinterpret_cast<const void*>(wn_mchain_kernel<S, true, true, true, PAIR>)
                      : reinterpret_cast<const void*>(wn_mchain_kernel<S, true, false, true, PAIR>);
    return ax ? reinterpret_cast<const void*>(wn_mchain_kernel<S, true, true, false, PAIR>)
              : reinterpret_cast<const void*>(wn_mchain_kernel<S, true, false, false, PAIR>);
  }
  if (i8) return ax ? reinterpret_cast<const void*>(wn_mchain_kernel<S, false, true, true, PAIR>)
                    : reinterpret_cast<const void*>(wn_mchain_kernel<S, false, false, true, PAIR>);
  return ax ? reinterpret_cast<const void*>(wn_mchain_kernel<S, false, true, false, PAIR>)
            : reinterpret_cast<const void*>(wn_mchain_kernel<S, false, false, false, PAIR>);
}

template <int S>
hipError_t launch_mchain_s(const WnChainArgs& g, bool teacher, hipStream_t stream) {
  const size_t dyn = mchain_lds<S>();
  const bool ax = g.w.approx_nl != 0, i8 = g.w.i8 != 0;
  const void* k = g.pair ? mchain_kernel<S, true>(teacher, ax, i8) : mchain_kernel<S, false>(teacher, ax, i8);
  hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
  if (e != hipSuccess) return e;
  void* args[] = {const_cast<WnChainArgs*>(&g)};
  return hipLaunchCooperativeKernel(k, dim3(WN_CHAIN_GRID), dim3(NT), args, (unsigned)dyn, stream);
}

}  // namespace

bool wn_mchain_supported(int R_, int S_, int L) {
  if (R_ != R || S_ != 256 || L < 1 || L > WN_MAX_LAYERS) return false;
  int lb[WN_MAX_LAYERS + 2];
  const int nch = mchain_split(L, lb);
  const int naux = (L + NLA - 1) / NLA;
  return nch <= WN_MAX_CHAIN && nch + 1 + naux <= WN_CHAIN_GRID && mchain_lds<256>() <= kMaxLds;
}

bool wn_mchain_plan(int L, int R_, int S_, int B, WnChainPlan* p) {
  if (!p || B < 1 || !wn_mchain_supported(R_, S_, L)) return false;
  WnChainPlan q{};
  q.nch = mchain_split(L, q.layer_begin);
  q.tail_on_chain = 1;
  // Layouts in order of preference: paired columns (8 streams per replica, one head CU), then 16
  // streams per replica (two head CUs; WN_MFMA_COLUMNS=16 forces it); each with front-loaded aux
  // ranges, then uniform ones (WN_AUX_LAYERS=n forces uniform runs of n).  The first whose replicas
  // carry B streams (as few replicas as do, the streams spread evenly) is taken.
  const char* ce = std::getenv("WN_MFMA_COLUMNS");
  const bool force16 = ce && std::atoi(ce) == 16;
  int nla_forced = 0;
  if (const char* e = std::getenv("WN_AUX_LAYERS")) {
    const int v = std::atoi(e);
    if (v >= 1 && v <= NLA) nla_forced = v;
  }
  int per = 0, nrep = 0;
  for (int pair = force16 ? 0 : 1; pair >= 0 && nrep == 0; --pair) {
    for (int front = nla_forced ? 0 : 1; front >= 0; --front) {
      const int ns = pair ? 8 : 16;
      q.naux = aux_split(L, nla_forced ? nla_forced : NLA, front != 0, q.aux_begin);
      per = q.nch + (pair ? 1 : 2) + q.naux;
      const int nr = (B + ns - 1) / ns;
      if (nr <= WN_CHAIN_GRID / per) {
        q.pair = pair;
        nrep = nr;
        break;
      }
    }
  }
  if (nrep == 0) return false;
  q.nla = 0;
  for (int a = 0; a < q.naux; ++a) q.nla = std::max(q.nla, q.aux_begin[a + 1] - q.aux_begin[a]);
  // aux CUs that post a skip partial: all but one holding only the last layer
  q.naux_q = q.aux_begin[q.naux - 1] == L - 1 ? q.naux - 1 : q.naux;
  const int NS = q.pair ? 8 : 16, NH = q.pair ? 1 : 2;
  q.G = (B + nrep - 1) / nrep;
  q.nrep = (B + q.G - 1) / q.G;
  q.ub = 0;
  // mailboxes of one replica (one slot each), in words: pre [L][2R NS] at 0, h [L][R NS], skip
  // partials [naux][S NS], the tail's [S NS], x [nch][R NS]
  const long long xw = (long long)R * NS, pw = 2 * xw, qw = (long long)S_ * NS;
  q.off_h = (int)(L * pw);
  q.off_q = (int)(q.off_h + L * xw);
  q.off_qtail = (int)(q.off_q + q.naux * qw);
  q.off_x = (int)(q.off_qtail + qw);
  q.off_logit = 0;
  q.mb_words = ((long long)q.off_x + q.nch * xw + 31) / 32 * 32;
  // Placement: slot i of XCD x is block 8 i + x.  Each replica's chain CUs and head CUs go to its home
  // XCD first, then its aux CUs, last layers first, overflowing to the XCD with the most room.
  int used[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  constexpr int per_xcd = WN_CHAIN_GRID / 8;
  for (int b = 0; b < WN_CHAIN_GRID; ++b) q.role_of_block[b] = 0xffff;
  auto place = [&](int role, int home) {
    int x = home;
    if (used[x] >= per_xcd) {
      for (int y = 0; y < 8; ++y)
        if (used[y] < used[x]) x = y;
    }
    q.role_of_block[8 * used[x] + x] = (uint16_t)role;
    ++used[x];
  };
  for (int k = 0; k < q.nrep; ++k)
    for (int r = 0; r < q.nch + NH; ++r) place(k * per + r, k % 8);
  for (int k = 0; k < q.nrep; ++k)
    for (int a = q.naux - 1; a >= 0; --a) place(k * per + q.nch + NH + a, k % 8);
  *p = q;
  return true;
}

int wn_mchain_columns(const WnChainPlan& p) { return p.pair ? 8 : 16; }

hipError_t wn_mchain_launch(const WnChainArgs& g, bool teacher, hipStream_t stream) {
  if (g.d.R == R && g.d.S == 256) return launch_mchain_s<256>(g, teacher, stream);
  return hipErrorInvalidValue;
}
