// Multi-CU persistent generation kernel, fp32 weights, gfx950.
//
// One generated sample is a strictly serial chain: the previous sample's
// embedding, then l gated layers, then the skip sum and the two-layer head, then
// the draw that feeds the next step (Deep Voice, arXiv 1702.07825, Appendix A.1;
// Section 5 explains why inference must go one timestep and one layer at a time).
// The paper's GPU design keeps the weights in the register files of many SMs and
// passes control round-robin between them through L2 (Appendix D).  This kernel
// keeps that idea -- weights resident in VGPRs, nothing re-read from memory -- but
// takes the off-chain work off the critical path, as the paper's CPU design does
// with its auxiliary threads (Section 5.1):
//
//   chain CUs  hold W_cur and W_res of a contiguous run of layers in VGPRs and
//              compute, per layer, a = W_cur x + pre, h = tanh(a_h) sigmoid(a_g),
//              x += W_res h + B_res.  Chain CU 0 also holds the embedding table in
//              LDS, sums the head's partial logits and draws the sample.
//   aux CUs    (two consecutive layers each) hold W_prev and W_skip in VGPRs (at
//              r = 128 the first layer's W_skip in LDS).  For the NEXT step they
//              compute pre = W_prev x[t+1-d] + B + L[t+1] (so the dilated half, the
//              bias and the HBM read of the conditioning all happen a step early), and
//              for the current step the skip partial W_skip h summed over their layers.
//   head CUs   (four) hold 64 rows of W_relu and the matching 64 columns of W_out:
//              z_a = relu(W_relu relu(q) + B_relu) for their rows and the partial
//              logits W_out[:, rows] z_a[rows].
//
// Messages between CUs are vectors of 64-bit words (fp32 value in the low half,
// step + 1 in the high half), written with relaxed atomic stores (workgroup scope when
// the reader runs on the writer's XCD, else agent scope) and read in pairs with
// 128-bit agent-scope loads.
// Every word carries its own step tag, so a reader needs no fence: it re-reads a
// word until the tag it expects appears.  Each mailbox has one slot: per stream, a
// producer writes step t + 1 only after something that depends on its consumer's
// read of step t (an aux CU posts pre_j[t + 1] once h_j[t] is in, which the chain
// posts after reading pre_j[t]; every role's step t + 1 needs chain CU 0's draw of
// step t, which reads the head's logits, which need every skip partial of step t),
// and the tags keep the steps apart.  The dilation histories are rings of tagged
// words in the workspace: slot (t mod d) of layer j holds x_{j-1}[t] tagged t + 1.
//
// Several streams: the roles above form one replica.  Up to 256 / (roles per replica) replicas
// run side by side, each serving G streams, and every role of a replica takes its streams in
// turn within each step (stream i of step t after stream i - 1).  All messages are per stream,
// so the per-stream protocol is unchanged; while chain CU c works on stream i, chain CU c + 1
// works on stream i - 1, so the interleaved streams fill the chain's idle time.  Every role
// takes the (step, stream) pairs in the same order, and each input of a pair is produced at an
// earlier pair by its producer, so no role can wait on a role that waits on it.
//
// Every wait is bounded.  A block that times out stores WN_ETIMEOUT in the
// workspace status word; every waiting block polls that word and leaves, so the
// grid always drains.  The host gives each block its role: when blocks are dealt
// round-robin over the eight XCDs (block b on XCD b mod 8), a replica's chain and
// head CUs and as many of its aux CUs as fit (the last layers first) share one XCD.
// The protocol does not depend on that placement, only the hop latency does.
#include "wn_internal.h"
#include "wn_msg.h"
#include "wn_wave.h"

#include "wn.h"

#include <algorithm>
#include <cstdlib>
#include <type_traits>

namespace {

using namespace wnk;

typedef float f4v __attribute__((ext_vector_type(4)));
constexpr int NT = 512;
constexpr int A = WN_A;
constexpr int NHEAD = 4;
constexpr int HR = A / NHEAD;  // z_a rows per head CU

// A set of tagged words to wait for: item i lives at base + (i / len) * stride + i % len and
// its value goes to dst[i].
struct Items {
  const u64* base;
  int len, stride, n;
  float* dst;
  unsigned tag;  // the step tag the words must carry
};
__device__ __forceinline__ Items no_items() { return Items{nullptr, 1, 0, 0, nullptr, 0u}; }

// Wait until every item of `a` and `b` owned by this thread carries its descriptor's tag, writing
// the values to LDS (dst pointers lie in `lds`).  Items go in pairs (2p, 2p + 1), one 128-bit load
// each (wn_msg.h); pair p belongs to thread p mod NT, and up to K owned pairs are in flight together.
// Every descriptor's item count and segment length are even, so a pair never straddles two
// segments.  A thread that times out, or sees a nonzero status word, sets the block's abort flag and
// stops waiting.  Every polled word lies in the workspace's tagged region, which starts at g.ring;
// items are tracked as 32-bit word offsets from there.  With acc != nullptr the thread also adds the
// values of its pairs' first items to acc[0] and of their second items to acc[1], in pair order.
template <int K = 2>
__device__ void poll2(const WnChainArgs& g, const Items a, const Items b, float* lds, Sync s,
                      float* acc = nullptr) {
  const int np = (a.n + b.n) / 2;
  const u64* wbase = g.ring;
  const wrsrc rs = region_rsrc(g.ring, (size_t)(g.mb + (size_t)g.io.B * g.mb_words - g.ring));
  for (int base = threadIdx.x; base < np; base += K * NT) {
    u32x4 w[K];
    unsigned so[K], dofs[K];
    unsigned pend = 0, useb = 0;  // bit k: pair base + k * NT pending / belongs to descriptor b
    static_assert(K <= 32, "pending bits");
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int i = 2 * (base + k * NT);
      if (i < 2 * np) {
        const bool inb = (i >= a.n);
        const Items& it = inb ? b : a;
        const int ii = inb ? i - a.n : i;
        so[k] = (unsigned)((it.base - wbase) + (size_t)(ii / it.len) * it.stride + (ii % it.len));
        dofs[k] = (unsigned)((it.dst - lds) + ii);
        pend |= 1u << k;
        useb |= (inb ? 1u : 0u) << k;
        w[k] = ld_pair(rs, so[k]);
      }
    }
    int spins = 0;
    while (true) {
#pragma unroll
      for (int k = 0; k < K; ++k) {
        if (pend & (1u << k)) {
          const unsigned tg = (useb & (1u << k)) ? b.tag : a.tag;
          if (w[k][1] == tg && w[k][3] == tg) {
            pend &= ~(1u << k);
            lds[dofs[k]] = __uint_as_float(w[k][0]);
            lds[dofs[k] + 1] = __uint_as_float(w[k][2]);
          }
        }
      }
      if (!pend) {
        if (acc) {
#pragma unroll
          for (int k = 0; k < K; ++k) {
            if (base + k * NT < np) {
              acc[0] += __uint_as_float(w[k][0]);
              acc[1] += __uint_as_float(w[k][2]);
            }
          }
        }
        break;
      }
      if (++spins > g.spin_limit || ((spins & 63) == 0 && ld_status(g.status) != 0)) {
        if (ld_status(g.status) == 0) atomicCAS(g.status, 0, (int)WN_ETIMEOUT);
        *s.flag = 1;
        return;
      }
      // a compiler barrier between reloads: without one the compiler may hoist the loads out of the
      // loop (a 64-clock sleep here instead measured 0.3 us/step slower at l = 20, B = 1)
      asm volatile("" ::: "memory");
#pragma unroll
      for (int k = 0; k < K; ++k)
        if (pend & (1u << k)) w[k] = ld_pair(rs, so[k]);
    }
  }
}

template <int R>
struct ChainMap {
  static constexpr int LPR1 = NT / (2 * R);  // lanes per W_prev row (aux CUs)
  static constexpr int KC1 = R / LPR1;       // weights per lane per row
  static constexpr int LPRG = NT / R;        // lanes per gate pair (rows c and c + R of W_cur)
  static constexpr int KCG = R / LPRG;       // inputs per lane for each of the two rows
  static constexpr int LPR2 = NT / R;        // lanes per W_res row
  static constexpr int KC2 = R / LPR2;
  static_assert(LPR1 >= 1 && KC1 % 2 == 0 && KC2 >= 2 && KCG >= 2, "unsupported R");
  // r = 128 keeps W_res of one layer in VGPRs; a CU with two layers keeps both W_res in LDS
  static constexpr int WRV = (R == 128) ? 1 : 1 << 30;
  // r = 128 uses 8-lane groups instead: group q holds gate pairs 2q, 2q + 1 (W_cur) and rows
  // 2q, 2q + 1 (W_res); lane i of a group takes the inputs 4 (i + 8 m) .. + 3, m < R / 32.
  static constexpr bool G8 = (R == 128);
  static constexpr int CPL = R / 32;  // float4 input chunks per lane in the 8-lane layout
};

// Row stride (floats) of a matrix kept in LDS and read by 8-lane groups, lane i of a group taking
// the float4 chunks i, i + 8, ... of a row and group g + 1 reading the row `rows` after group g's:
// the two groups of a 16-lane access phase then hit the two halves of the 64 banks.
constexpr int lds_row_stride(int K, int rows) {
  int w = K;
  while ((rows * w) % 64 != 32) ++w;
  return w;
}


template <int K>
__device__ __forceinline__ float dot_lds(const float (&w)[K], const float* x, float init = 0.f) {
  float s0 = init, s1 = 0.f;
  if constexpr (K % 8 == 0) {
    float s2 = 0.f, s3 = 0.f;
#pragma unroll
    for (int i = 0; i < K; i += 4) {
      const float4 v = *reinterpret_cast<const float4*>(x + i);
      s0 = fmaf(w[i], v.x, s0);
      s1 = fmaf(w[i + 1], v.y, s1);
      s2 = fmaf(w[i + 2], v.z, s2);
      s3 = fmaf(w[i + 3], v.w, s3);
    }
    return (s0 + s1) + (s2 + s3);
  } else if constexpr (K % 4 == 0) {
#pragma unroll
    for (int i = 0; i < K; i += 4) {
      const float4 v = *reinterpret_cast<const float4*>(x + i);
      s0 = fmaf(w[i], v.x, s0);
      s1 = fmaf(w[i + 1], v.y, s1);
      s0 = fmaf(w[i + 2], v.z, s0);
      s1 = fmaf(w[i + 3], v.w, s1);
    }
  } else {
#pragma unroll
    for (int i = 0; i < K; i += 2) {
      const float2 v = *reinterpret_cast<const float2*>(x + i);
      s0 = fmaf(w[i], v.x, s0);
      s1 = fmaf(w[i + 1], v.y, s1);
    }
  }
  return s0 + s1;
}

// The same over a group of G lanes that share a row, in 16-byte chunks: this lane takes chunks
// c, c + G, c + 2 G, ... of the input vector (x points at its first chunk) and w holds its weights
// in that order.  Consecutive lanes read consecutive chunks, so the group's reads fall on distinct
// LDS banks (a lane-contiguous split with K >= 32 puts every other lane on the same banks).
template <int K, int G>
__device__ __forceinline__ float dot_lds_il(const float (&w)[K], const float* x) {
  static_assert(K % 4 == 0, "whole chunks");
  float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
#pragma unroll
  for (int m = 0; m < K / 4; ++m) {
    const float4 v = *reinterpret_cast<const float4*>(x + 4 * G * m);
    s0 = fmaf(w[4 * m], v.x, s0);
    s1 = fmaf(w[4 * m + 1], v.y, s1);
    s2 = fmaf(w[4 * m + 2], v.z, s2);
    s3 = fmaf(w[4 * m + 3], v.w, s3);
  }
  return (s0 + s1) + (s2 + s3);
}

// ------------------------------------------------------------------------------------------
// chain CU
// ------------------------------------------------------------------------------------------
// Two embedding tables fit chain CU 0's LDS beside its other buffers up to r = 64.
constexpr bool e2_in_lds(int R) { return R <= 64; }

// NLK > 0: this CU holds NLK layers, a compile-time count, so that no layer of the unrolled loop
// tests a run-time count (measured ~0.06 us per layer, in reloads of spilled masks and branches);
// NLK = 0: the count is read at run time.
template <int R, int S, int NLC, bool TF, bool MS, bool E2, bool AX, int NLK, class LM>
__device__ __forceinline__ void chain_role(const WnChainArgs& g, const int c, const int b0, const int ns, float* dyn, Sync sy,
                           const int64_t tg0, const LM lm) {
  constexpr bool E2L = E2 && e2_in_lds(R);
  using M = ChainMap<R>;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int L = g.d.L;
  const int j0 = g.layer_begin[c], nl = NLK > 0 ? NLK : g.layer_begin[c + 1] - j0;
  const bool first = (c == 0);
  const bool lastc = (c + 1 == g.nch);
  const bool tail = lastc && g.tail_on_chain;
  const int T = g.io.T;
  // streams per replica and staged steps per stream (a power of two); constants for one stream
  const int G = MS ? g.G : 1;
  const int ub = MS ? g.ub : 512, ubs = MS ? __builtin_ctz(g.ub) : 9;

  constexpr int NLCP = (NLC + 3) & ~3;
  constexpr int RPG = S / 64;                     // tail skip projection: rows per 8-lane group
  constexpr int WSK = lds_row_stride(R, RPG);     // W_skip row stride in LDS
  constexpr int WRS = lds_row_stride(R, 2);       // W_res row stride in LDS (r = 128)
  const int gq = tid >> 3, li = tid & 7;          // 8-lane group and lane in it
  const bool upper = (li & 4) != 0;
  // LDS: the part every chain CU uses, then a part that depends on the CU's place in the chain
  float* xs = dyn;                                  // R      x_{j-1}, updated in place
  float* hs = xs + R;                               // R
  float* pre = hs + R;                              // NLC*2R pre-activations of this step
  float* xbuf = pre + NLC * 2 * R;                  // NLC*R  x_{j-1} of this step (history writes)
  float* bres = xbuf + NLC * R;                     // NLC*R  B_res of my layers
  int* slotv = reinterpret_cast<int*>(bres + NLC * R);  // 2*NLCP history slot (t mod d) of each layer, by step parity
  // dilation and history offset of each of my layers (a kernel-argument array indexed at run time
  // would be read from memory, and the wait for that read also waits for this wave's stores)
  int* ldil = slotv + 2 * NLCP;                     // NLCP
  int* lhoff = ldil + NLCP;                         // NLCP
  float* var = reinterpret_cast<float*>(lhoff + NLCP);
  // chain CU 0: partial logits, staged inputs and samples, last samples, the embedding table
  float* lgp = var;                                 // NHEAD*A
  float* ubuf = lgp + NHEAD * A;                    // G*ub   uniforms / samples in, per stream
  int* ybuf = reinterpret_cast<int*>(ubuf + G * ub);  // G*ub drawn samples
  int* syv = ybuf + G * ub;                         // G      y_{t-1} of each stream
  int* syv2 = syv + ((G + 3) & ~3);                 // G      y_{t-2} (-1 before the first input)
  float* emb = reinterpret_cast<float*>(syv2 + ((G + 3) & ~3));  // A*R
  // the table of y_{t-2} (two taps, r <= 64; a global load instead at r = 128, where two tables
  // do not fit)
  float* emb2 = emb + A * R;                        // A*R when E2L
  // last chain CU: W_skip of layer l-1, S rows of stride WSK (after the tables if it is also CU 0)
  float* wsk = first ? emb2 + (E2L ? A * R : 0) : var;
  // a middle r = 128 CU with two layers: their W_res, R rows of stride WRS each
  float* wres = var;
  const bool wres_lds = nl > M::WRV;

  // resident weights
  // W_cur: lane group c (LPRG lanes) holds rows c and c + R, lane kq of it inputs kq*KCG .. +KCG
  const int g1 = tid / M::LPRG, kq = tid % M::LPRG;
  const int row2 = tid / M::LPR2, kk = tid % M::LPR2;
  constexpr int NWR = NLC < M::WRV ? NLC : M::WRV;
  float wc[NLC][2 * M::KCG], wr[NWR][M::KC2];
  const float* Wc = static_cast<const float*>(g.w.w_cur);
  const float* Wr = static_cast<const float*>(g.w.w_res);
#pragma unroll
  for (int l = 0; l < NLC; ++l) {
    const int j = j0 + (l < nl ? l : 0);
    if constexpr (M::G8) {
      // rows tanh 2q, sigmoid 2q, tanh 2q + 1, sigmoid 2q + 1; chunk m of each
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int row = 2 * gq + (rr >> 1) + (rr & 1) * R;
#pragma unroll
        for (int m = 0; m < M::CPL; ++m)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            wc[l][(rr * M::CPL + m) * 4 + e] = Wc[((size_t)j * 2 * R + row) * R + 4 * (li + 8 * m) + e];
      }
    } else {
#pragma unroll
      for (int i = 0; i < M::KCG; ++i) {
        wc[l][i] = Wc[((size_t)j * 2 * R + g1) * R + kq * M::KCG + i];
        wc[l][M::KCG + i] = Wc[((size_t)j * 2 * R + g1 + R) * R + kq * M::KCG + i];
      }
    }
  }
  if (wres_lds) {
    for (int i = tid; i < nl * R * R; i += NT) {
      const int l = i / (R * R), rr = (i / R) % R, k = i % R;
      wres[(l * R + rr) * WRS + k] = Wr[(size_t)j0 * R * R + i];
    }
  } else {
#pragma unroll
    for (int l = 0; l < NWR; ++l) {
      const int j = j0 + (l < nl ? l : 0);
      if constexpr (M::G8) {
#pragma unroll
        for (int rr = 0; rr < 2; ++rr)
#pragma unroll
          for (int m = 0; m < M::CPL; ++m)
#pragma unroll
            for (int e = 0; e < 4; ++e)
              wr[l][(rr * M::CPL + m) * 4 + e] = Wr[((size_t)j * R + 2 * gq + rr) * R + 4 * (li + 8 * m) + e];
      } else {
#pragma unroll
        for (int i = 0; i < M::KC2; ++i) wr[l][i] = Wr[((size_t)j * R + row2) * R + kk * M::KC2 + i];
      }
    }
  }
  for (int i = tid; i < nl * R; i += NT) bres[i] = g.w.b_res[(size_t)j0 * R + i];
  if (tid < nl) {
    slotv[(tg0 & 1) * NLCP + tid] = (int)(tg0 % g.d.dil[j0 + tid]);
    ldil[tid] = g.d.dil[j0 + tid];
    lhoff[tid] = g.d.hoff[j0 + tid];
  }
  float bemb = 0.f;
  // two-tap input convolution (E2): the table of y_{t-2}, copied to LDS when it fits (E2L)
  const float* const Eprev = E2 ? static_cast<const float*>(g.w.embed_prev) : nullptr;
  float4 bout4 = make_float4(0.f, 0.f, 0.f, 0.f);  // B_out of the 4 logits lane l of wave 0 draws from
  if (tail) {
    const float* Wk = static_cast<const float*>(g.w.w_skip) + (size_t)(L - 1) * S * R;
    for (int i = tid; i < S * R; i += NT) wsk[(i / R) * WSK + i % R] = Wk[i];
  }
  int64_t ub0 = tg0;  // first global step held in ubuf / ybuf
  // Stage steps ub0 .. ub0 + ub - 1 of every stream's uniforms (or teacher-forced samples).
  auto stage_inputs = [&]() {
    for (int idx = tid; idx < ns * ub; idx += NT) {
      const int i = idx >> ubs, k = idx & (ub - 1);
      const int64_t t = ub0 + k;
      if (t < tg0 + T) {
        const size_t at = (size_t)(b0 + i) * T + (size_t)(t - tg0);
        if constexpr (TF) reinterpret_cast<int*>(ubuf)[idx] = g.io.y_in[at];
        else ubuf[idx] = g.io.u[at];
      }
    }
  };
  if (first) {
    if (wave == 0) bout4 = *reinterpret_cast<const float4*>(g.w.b_out + 4 * lane);
    const float* E = static_cast<const float*>(g.w.embed);
    for (int i = tid; i < A * R; i += NT) emb[i] = E[i];
    if constexpr (E2L)
      for (int i = tid; i < A * R; i += NT) emb2[i] = Eprev[i];
    if (tid < R) bemb = g.w.b_embed[tid];
    for (int i = tid; i < ns; i += NT) {
      const int64_t* st = g.state + WN_STATE_WORDS * (size_t)(b0 + i);
      int y = g.io.reset ? g.io.init_sample : (int)st[1];
      syv[i] = y < 0 ? 0 : (y > A - 1 ? A - 1 : y);
      int y2 = g.io.reset ? -1 : (int)st[2];
      syv2[i] = y2 < 0 ? -1 : (y2 > A - 1 ? A - 1 : y2);
    }
    stage_inputs();
  }
  lds_barrier();

  // One wave sums the head's partial logits of global step ts of local stream i (lane l owns
  // logits 4l..4l+3), writes them out when teacher forcing, and draws (generation) or reads
  // (teacher forcing) the sample.
  // With r <= 64 (and the second embedding table, if any, in LDS) the drawing wave also forms the
  // next step's x0 = E[y] + B_embed (+ ep = E_prev[y_{t-2}]) from the sample in its registers.
  constexpr bool X0W = R <= 64 && (!E2 || E2L);
  auto sample_step = [&](int64_t ts, int i, float ep) {
    if (wave == 0) {
      float4 lv = bout4;
#pragma unroll
      for (int h = 0; h < NHEAD; ++h) {
        const float4 p = *reinterpret_cast<const float4*>(lgp + h * A + 4 * lane);
        lv.x += p.x;
        lv.y += p.y;
        lv.z += p.z;
        lv.w += p.w;
      }
      const int at = (i << ubs) + (int)(ts - ub0);
      int y;
      if constexpr (TF) {
        *reinterpret_cast<float4*>(g.io.logits + ((size_t)(b0 + i) * T + (size_t)(ts - tg0)) * A + 4 * lane) = lv;
        y = reinterpret_cast<const int*>(ubuf)[at];
        y = y < 0 ? 0 : (y > A - 1 ? A - 1 : y);
      } else if (g.io.smode == WN_DRAW_DIRECT || g.io.smode == WN_DRAW_TEMPERATURE) {
        const float4 lv1[1] = {lv};
        const float u1[1] = {ubuf[at]};
        int y1[1];
        wave_draw_cdf<AX>(lv1, u1, g.io.smode == WN_DRAW_TEMPERATURE ? g.io.inv_t : 1.0f, y1);
        y = y1[0];
      } else {
        y = wave_draw<AX>(lv, ubuf[at], g.io.smode, g.io.inv_t, g.io.top_k, lane);
      }
      if (lane == 0) {
        if constexpr (E2) syv2[i] = syv[i];
        syv[i] = y;
        ybuf[at] = y;
      }
      if constexpr (X0W) {
        if (lane < R) {
          if constexpr (E2) xs[lane] = emb[y * R + lane] + bemb + ep;
          else xs[lane] = emb[y * R + lane] + bemb;
        }
      }
    }
  };
  // The head's partial logits of step ts of stream b (tag ts + 1).
  auto logit_items = [&](int64_t ts, int b) {
    return Items{g.mb + (size_t)b * g.mb_words + g.off_logit, A, A, NHEAD * A, lgp, (unsigned)(ts + 1)};
  };
  // Move staged samples (steps before next0) to the output and stage the next block of inputs.
  auto roll_buffers = [&](int64_t next0) {
    if constexpr (!TF) {
      for (int idx = tid; idx < ns * ub; idx += NT) {
        const int i = idx >> ubs, k = idx & (ub - 1);
        const int64_t t = ub0 + k;
        if (t < next0 && t < tg0 + T) g.io.y_out[(size_t)(b0 + i) * T + (size_t)(t - tg0)] = ybuf[idx];
      }
    }
    lds_barrier();
    ub0 = next0;
    stage_inputs();
    lds_barrier();
  };

  for (int64_t t = tg0; t < tg0 + T; ++t) {
    const unsigned tag = (unsigned)(t + 1);
    const int par = (int)(t & 1);
    for (int i = 0; i < ns; ++i) {
      const int b = b0 + i;
      u64* const mbs = g.mb + (size_t)b * g.mb_words;
      u64* const rings = g.ring + (size_t)b * g.d.hist_len;
      // ---- inputs of this step, all waited for together: the pre-activations of my layers, and
      //      either x from the previous chain CU or (chain CU 0) the previous step's partial logits ----
      const Items pre_items{mbs + (size_t)j0 * 2 * R, 2 * R, 2 * R, nl * 2 * R, pre, tag};
      if (first) {
        // two-tap embedding: the row of y_{t-2}, known since the previous step, from LDS; at
        // r = 128 from global memory before the wait for the previous step's logits (the empty
        // asm keeps the compiler from sinking the load to its use after that wait).  A global
        // load here measured ~0.4 us of step time even when it hits in cache; the LDS read none.
        float ep = 0.f;
        if constexpr (E2) {
          const int y2 = t > tg0 ? syv[i] : syv2[i];
          if constexpr (E2L) {
            if (tid < R && y2 >= 0) ep = emb2[y2 * R + tid];
          } else {
            if (tid < R && y2 >= 0) ep = Eprev[(size_t)y2 * R + tid];
            asm volatile("" : "+v"(ep));
          }
        }
        bool x0_done = false;
        if (t > tg0) {
          poll2(g, logit_items(t - 1, b), pre_items, dyn, sy);
          lds_barrier();
          if (sy.failed()) return;
          if (i == 0 && t - 1 - ub0 >= ub) roll_buffers(t - 1);
          sample_step(t - 1, i, ep);
          x0_done = X0W;
        } else {
          poll2(g, pre_items, no_items(), dyn, sy);
        }
        if (!x0_done) {
          lds_barrier();
          if (sy.failed()) return;
          if (tid < R) {
            if constexpr (E2) xs[tid] = emb[syv[i] * R + tid] + bemb + ep;
            else xs[tid] = emb[syv[i] * R + tid] + bemb;
          }
        }
      } else {
        poll2(g, pre_items, Items{mbs + g.off_x + (size_t)c * R, R, R, R, xs, tag}, dyn, sy);
      }
      lds_barrier();
      if (sy.failed()) return;
      // history slots of step t + 1 (step t's stay readable until then: the slots of the other
      // parity were last read during step t - 1, which every thread has left)
      if (i == 0 && tid < nl) {
        const int sl = slotv[par * NLCP + tid] + 1;
        slotv[(par ^ 1) * NLCP + tid] = (sl == ldil[tid]) ? 0 : sl;
      }

      // h_j[t] -> layer j's aux CU (skip projection), posted by the lanes that computed it.  The
      // store data rotate over HPOST register pairs: a pair is written again HPOST layers after
      // its store was issued, by when that store has completed, so the wait the compiler places
      // before the overwrite costs nothing inside the layer loop.
      constexpr int HPOST = 3;
      u64 hpost[HPOST];
#pragma unroll
      for (int l = 0; l < HPOST; ++l) hpost[l] = 0;
      auto post_h = [&](int l, int j, int row, float h) __attribute__((always_inline)) {
        // an opaque row index keeps the compiler from hoisting one 64-bit address per layer out
        // of the step loop (they would not fit in registers)
        asm volatile("" : "+v"(row));
        hpost[l % HPOST] = pack(h, tag);
        stw(mbs + g.off_h + (size_t)j * R + row, hpost[l % HPOST], lm(l));
      };
      // x of this CU's last layer -> the next chain CU, posted by the lanes that computed it
      const bool handoff = c + 1 < g.nch;
      auto post_x = [&](int row, float v) __attribute__((always_inline)) {
        if (handoff) stw(mbs + g.off_x + (size_t)(c + 1) * R + row, pack(v, tag), lm(16));
      };
#pragma unroll
      for (int l = 0; l < NLC; ++l) {
        if (l < nl) {
          const int j = j0 + l;
          const bool last_layer = lastc && l == nl - 1;  // j == L - 1
          if (last_layer && tid < R) xbuf[l * R + tid] = xs[tid];
          // a = W_cur x + pre ; h = tanh(a[0:R]) * sigmoid(a[R:2R]).  Each lane ends with both rows
          // of a pair; the first lane of a group starts its partial sums from pre, so pre joins
          // the reduction.
          if constexpr (M::G8) {
            float p[4][2];
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) p[rr][0] = p[rr][1] = 0.f;
            if (li == 0) {
#pragma unroll
              for (int rr = 0; rr < 4; ++rr) p[rr][0] = pre[l * 2 * R + 2 * gq + (rr >> 1) + (rr & 1) * R];
            }
#pragma unroll
            for (int m = 0; m < M::CPL; ++m) {
              const float4 v = *reinterpret_cast<const float4*>(xs + 4 * (li + 8 * m));
#pragma unroll
              for (int rr = 0; rr < 4; ++rr) {
                const float* w = &wc[l][(rr * M::CPL + m) * 4];
                p[rr][0] = fmaf(w[0], v.x, p[rr][0]);
                p[rr][1] = fmaf(w[1], v.y, p[rr][1]);
                p[rr][0] = fmaf(w[2], v.z, p[rr][0]);
                p[rr][1] = fmaf(w[3], v.w, p[rr][1]);
              }
            }
            // lower four lanes: pair 2q, upper four: pair 2q + 1
            float ah, ag;
            xsplit8_2(p[0][0] + p[0][1], p[1][0] + p[1][1], p[2][0] + p[2][1], p[3][0] + p[3][1], upper, ah, ag);
            ah = gsum4(ah);
            ag = gsum4(ag);
            const float h = gate_nl<AX>(ah, ag, lane);  // lane pairs share (ah, ag)
            if ((li & 3) == 0) {
              int hr = 2 * gq + (upper ? 1 : 0);
              hs[hr] = h;
              post_h(l, j, hr, h);
            }
          } else {
            float sh0 = 0.f, sh1 = 0.f, sg0 = 0.f, sg1 = 0.f;
            if (kq == 0) {
              sh0 = pre[l * 2 * R + g1];
              sg0 = pre[l * 2 * R + g1 + R];
            }
            const float* xk = xs + kq * M::KCG;
            if constexpr (M::KCG % 4 == 0) {
#pragma unroll
              for (int i2 = 0; i2 < M::KCG; i2 += 4) {
                const float4 v = *reinterpret_cast<const float4*>(xk + i2);
                sh0 = fmaf(wc[l][i2], v.x, sh0);
                sh1 = fmaf(wc[l][i2 + 1], v.y, sh1);
                sh0 = fmaf(wc[l][i2 + 2], v.z, sh0);
                sh1 = fmaf(wc[l][i2 + 3], v.w, sh1);
                sg0 = fmaf(wc[l][M::KCG + i2], v.x, sg0);
                sg1 = fmaf(wc[l][M::KCG + i2 + 1], v.y, sg1);
                sg0 = fmaf(wc[l][M::KCG + i2 + 2], v.z, sg0);
                sg1 = fmaf(wc[l][M::KCG + i2 + 3], v.w, sg1);
              }
            } else {
              static_assert(M::KCG % 2 == 0, "inputs per lane must be even");
#pragma unroll
              for (int i2 = 0; i2 < M::KCG; i2 += 2) {
                const float2 v = *reinterpret_cast<const float2*>(xk + i2);
                sh0 = fmaf(wc[l][i2], v.x, sh0);
                sh1 = fmaf(wc[l][i2 + 1], v.y, sh1);
                sg0 = fmaf(wc[l][M::KCG + i2], v.x, sg0);
                sg1 = fmaf(wc[l][M::KCG + i2 + 1], v.y, sg1);
              }
            }
            const float ah = gsum<M::LPRG>(sh0 + sh1);
            const float ag = gsum<M::LPRG>(sg0 + sg1);
            const float h = gate_nl<AX>(ah, ag, lane);  // lane pairs share (ah, ag)
            if (kq == 0) {
              hs[g1] = h;
              post_h(l, j, g1, h);
            }
          }
          lds_barrier();
          // x_j = x_{j-1} + W_res h + B_res (x_l feeds nothing); x_{j-1} is kept for the history
          if (!last_layer) {
            if constexpr (M::G8) {
              // lower four lanes: row 2q, upper four: row 2q + 1.  x_{j-1} + B_res of the row joins
              // the reduction through lane 0 (row 2q) and lane 4 (row 2q + 1); every lane reads
              // it, so the read is issued with those of h rather than after the reduction
              const int row = 2 * gq + (upper ? 1 : 0);
              const float xo = xs[row];
              const float c0 = (li & 3) == 0 ? xo + bres[l * R + row] : 0.f;
              float r0 = upper ? 0.f : c0, r1 = upper ? c0 : 0.f;
              if (wres_lds) {
                const float* w0 = wres + (l * R + 2 * gq) * WRS;
#pragma unroll
                for (int m = 0; m < M::CPL; ++m) {
                  const int k = 4 * (li + 8 * m);
                  const float4 v = *reinterpret_cast<const float4*>(hs + k);
                  const float4 a = *reinterpret_cast<const float4*>(w0 + k);
                  const float4 b = *reinterpret_cast<const float4*>(w0 + WRS + k);
                  r0 = fmaf(a.x, v.x, fmaf(a.y, v.y, fmaf(a.z, v.z, fmaf(a.w, v.w, r0))));
                  r1 = fmaf(b.x, v.x, fmaf(b.y, v.y, fmaf(b.z, v.z, fmaf(b.w, v.w, r1))));
                }
              } else {
                const float* w = wr[l < NWR ? l : 0];
#pragma unroll
                for (int m = 0; m < M::CPL; ++m) {
                  const float4 v = *reinterpret_cast<const float4*>(hs + 4 * (li + 8 * m));
                  const float* a = w + m * 4;
                  const float* b = w + (M::CPL + m) * 4;
                  r0 = fmaf(a[0], v.x, fmaf(a[1], v.y, fmaf(a[2], v.z, fmaf(a[3], v.w, r0))));
                  r1 = fmaf(b[0], v.x, fmaf(b[1], v.y, fmaf(b[2], v.z, fmaf(b[3], v.w, r1))));
                }
              }
              const float r = gsum4(xsplit8_1(r0, r1, upper));
              if ((li & 3) == 0) {
                xbuf[l * R + row] = xo;
                xs[row] = r;
                if (l == nl - 1) post_x(row, r);
              }
            } else {
              // x_{j-1} + B_res joins the reduction through lane kk = 0 (read by every lane, so
              // it is issued with the reads of h)
              const float xo = xs[row2];
              const float c0 = kk == 0 ? xo + bres[l * R + row2] : 0.f;
              const float r = gsum<M::LPR2>(dot_lds<M::KC2>(wr[l < NWR ? l : 0], hs + kk * M::KC2, c0));
              if (kk == 0) {
                xbuf[l * R + row2] = xo;
                xs[row2] = r;
                if (l == nl - 1) post_x(row2, r);
              }
            }
            lds_barrier();
          }
          // the network's last layer has no residual (x_l feeds nothing): its x_{j-1} went to
          // xbuf before the first barrier, and the skip projection below reads h
        }
      }
      // The last chain CU adds the skip projection of the last layer itself (its W_skip is in
      // LDS), which saves the hop through that layer's aux CU on the way to the head.
      if (tail) {
        // group q: rows RPG q .. RPG q + RPG - 1; lane i: chunks i, i + 8, ... of each row
        float p[RPG];
#pragma unroll
        for (int rr = 0; rr < RPG; ++rr) p[rr] = 0.f;
#pragma unroll
        for (int m = 0; m < R / 32; ++m) {
          const int k = 4 * (li + 8 * m);
          const float4 v = *reinterpret_cast<const float4*>(hs + k);
#pragma unroll
          for (int rr = 0; rr < RPG; ++rr) {
            const float4 a = *reinterpret_cast<const float4*>(wsk + (RPG * gq + rr) * WSK + k);
            p[rr] = fmaf(a.x, v.x, fmaf(a.y, v.y, fmaf(a.z, v.z, fmaf(a.w, v.w, p[rr]))));
          }
        }
        const float q = xreduce8<RPG>(p, li);
        const int m = RPG * gq + (upper ? RPG / 2 : 0) + (RPG == 4 && (li & 2) ? 1 : 0);
        const int ks = (RPG == 4) ? (li & 1) : (li & 3);  // lanes holding the same row: post once
        if (ks == 0) stw(mbs + g.off_qtail + m, pack(q, tag), lm(17));
      }
      // Then x_{j-1} of each layer into the history slot (t mod d_j) that layer j's aux CU reads
      // again at t + d_j (the next chain CU's x went out in the last layer).
      for (int k = tid; k < nl * R; k += NT) {
        const int l = k / R, e = k % R;
        const int slot = slotv[par * NLCP + l];
        stw(rings + lhoff[l] + (size_t)slot * R + e, pack(xbuf[l * R + e], tag), lm(l));
      }
#pragma unroll
      for (int l = 0; l < HPOST; ++l) asm volatile("" ::"v"(hpost[l]));
    }
  }
  if (first) {
    if (T > 0) {
      const int64_t tl = tg0 + T - 1;
      for (int i = 0; i < ns; ++i) {
        poll2(g, logit_items(tl, b0 + i), no_items(), dyn, sy);
        lds_barrier();
        if (sy.failed()) return;
        if (i == 0 && tl - ub0 >= ub) roll_buffers(tl);
        sample_step(tl, i, 0.f);
        lds_barrier();
      }
      roll_buffers(tg0 + T);
    }
    if (!sy.failed()) {
      for (int i = tid; i < ns; i += NT) {
        int64_t* st = g.state + WN_STATE_WORDS * (size_t)(b0 + i);
        st[0] = tg0 + T;
        st[1] = syv[i];
        st[2] = syv2[i];
      }
    }
  }
}

// ------------------------------------------------------------------------------------------
// aux CU (nla consecutive layers): pre-activations of the next step and the skip partial
// ------------------------------------------------------------------------------------------
// Layers one aux CU holds: W_prev and W_skip of a layer take 48 floats per lane at r = 64,
// s = 256 (two layers fit the register file).  At r = 128 they take 128: the CU keeps both layers'
// W_prev (64 floats per lane each) and the second layer's W_skip in VGPRs and the first layer's
// W_skip in LDS (256 rows of 128 floats), so that an l = 20 replica (11 chain, 4 head, 10 aux CUs)
// fits one XCD's 32 CUs.
template <int R>
constexpr int aux_max_layers() { return 2; }
// r = 128: the aux CU's first layer's W_skip is read from LDS
template <int R>
constexpr bool aux_skip_in_lds() { return R == 128; }

template <int R, int S, bool TF, bool MS, class LM>
__device__ __forceinline__ void aux_role(const WnChainArgs& g, const int ai, const int b0, const int ns, float* dyn, Sync sy,
                         const int64_t tg0, const LM lm) {
  using M = ChainMap<R>;
  constexpr int NLA = aux_max_layers<R>();
  constexpr int LPRS = NT / S, KCS = R / LPRS;
  constexpr bool SKL = aux_skip_in_lds<R>();      // layer 0's W_skip in LDS
  constexpr int NWK = SKL ? NLA - 1 : NLA;        // W_skip blocks in VGPRs (layers SKL ..)
  constexpr int RPG = S / 64;                     // LDS skip product: rows per 8-lane group
  constexpr int WSKA = lds_row_stride(R, RPG);    // and its row stride
  constexpr int CQ = (WN_CHAIN_MAX_G * 2 * R / 4 + NT - 1) / NT;  // conditioning float4s per thread and layer
  const int tid = threadIdx.x;
  const int L = g.d.L;
  const int T = g.io.T;
  const int G = MS ? g.G : 1;
  const int ja = ai * g.nla, nl = min(g.nla, L - ja);  // my layers: ja .. ja + nl - 1
  // layers whose skip projection this CU computes (the last layer's runs on the last chain CU when
  // it has room for that W_skip); their sum goes to the head CUs as one partial per step
  const int nsk = (g.tail_on_chain && ja + nl == L) ? nl - 1 : nl;
  // LDS, carved for the plan's layers per aux CU (g.nla <= NLA)
  float* hs = dyn;                     // nla*R     h_j of the current stream, one row per layer
  float* xpg = hs + g.nla * R;         // nla*G*R   history reads x_{j-1}[ts - d] of every (layer, stream)
  float* clg = xpg + g.nla * G * R;    // nla*G*2R  conditioning rows L[b, ts, j] of every (layer, stream)
  float* wska = clg + g.nla * G * 2 * R;  // SKL: S rows of stride WSKA, W_skip of layer ja
  float* qsk = wska + S * WSKA;         // SKL: layer ja's skip projection of the current stream
  const int gq = tid >> 3, li = tid & 7;  // 8-lane groups of the LDS product

  const int rowp = tid / M::LPR1, kq = tid % M::LPR1;
  const int rows = tid / LPRS, ks = tid % LPRS;
  float wp[NLA][M::KC1], wk[NWK][KCS], bg[NLA];
  int dl[NLA], ho[NLA];  // dilation and history offset of each layer (uniform, kept in registers)
  const float* Wp = static_cast<const float*>(g.w.w_prev);
  const float* Wk = static_cast<const float*>(g.w.w_skip);
#pragma unroll
  for (int l = 0; l < NLA; ++l) {
    const int j = ja + (l < nl ? l : 0);
#pragma unroll
    for (int i = 0; i < M::KC1; ++i) wp[l][i] = Wp[((size_t)j * 2 * R + rowp) * R + kq * M::KC1 + i];
    if (l >= (SKL ? 1 : 0)) {
#pragma unroll
      for (int i = 0; i < KCS; ++i) wk[l - (SKL ? 1 : 0)][i] = Wk[((size_t)j * S + rows) * R + ks * KCS + i];
    }
    bg[l] = g.w.b_gate[j * 2 * R + rowp];
    dl[l] = g.d.dil[j];
    ho[l] = g.d.hoff[j];
  }

  if (SKL && nsk > 0)
    for (int i = tid; i < S * R; i += NT) wska[(i / R) * WSKA + i % R] = Wk[(size_t)ja * S * R + i];

  // The history slot that pre_j[ts] reads for every stream of the replica (consecutive streams'
  // histories are hist_len words apart), j = ja + l.
  auto hist_items = [&](int l, int64_t ts) {
    const int d = dl[l];
    const int slot = (d == 1) ? 0 : (int)(ts % d);
    const unsigned etag = (ts - d >= 0) ? (unsigned)(ts - d + 1) : 0u;
    return Items{g.ring + (size_t)b0 * g.d.hist_len + ho[l] + (size_t)slot * R, R, g.d.hist_len, ns * R,
                 xpg + l * G * R, etag};
  };
  // Stage the inputs of pre_j[ts] for every layer and stream at once: the conditioning rows (one HBM
  // round trip for all of them) and, when `all_hist`, every history read; otherwise the history reads
  // of the layers with d >= 2, which are final once step ts - d is over (with d = 1 the read waits for
  // the chain CU's step and is made per stream, together with h_j).
  auto stage = [&](int64_t ts, bool all_hist) {
    f4v cq[NLA][CQ];
#pragma unroll
    for (int l = 0; l < NLA; ++l) {
      if (l < nl) {
        const float* crow = g.io.cond + ((size_t)b0 * T + (size_t)(ts - tg0)) * L * 2 * R + (size_t)(ja + l) * 2 * R;
#pragma unroll
        for (int k = 0; k < CQ; ++k) {
          const int q = tid + k * NT;
          if (q < ns * (2 * R / 4)) {
            const int i = q / (2 * R / 4), e = q % (2 * R / 4);
            // each row is read once: a non-temporal load, so that the stream does not evict the mailboxes
            cq[l][k] = __builtin_nontemporal_load(reinterpret_cast<const f4v*>(crow + (size_t)i * T * L * 2 * R + 4 * e));
          }
        }
      }
    }
    const bool h0 = nl > 0 && (all_hist || dl[0] >= 2);
    const bool h1 = NLA > 1 && nl > 1 && (all_hist || dl[NLA > 1 ? 1 : 0] >= 2);
    if (h0 || h1)
      poll2(g, h0 ? hist_items(0, ts) : no_items(), h1 ? hist_items(NLA > 1 ? 1 : 0, ts) : no_items(), dyn, sy);
#pragma unroll
    for (int l = 0; l < NLA; ++l) {
      if (l < nl) {
#pragma unroll
        for (int k = 0; k < CQ; ++k) {
          const int q = tid + k * NT;
          if (q < ns * (2 * R / 4)) reinterpret_cast<f4v*>(clg + l * G * 2 * R)[q] = cq[l][k];
        }
      }
    }
    lds_barrier();
  };
  // pre_j[ts] of local stream i = W_prev x_{j-1}[ts - d] + B + L[b, ts], j = ja + l, tag ts + 1
  auto post_pre = [&](int l, int64_t ts, int i) {
    const float a = gsum<M::LPR1>(dot_lds<M::KC1>(wp[l], xpg + (l * G + i) * R + kq * M::KC1));
    if (kq == 0)
      stw(g.mb + (size_t)(b0 + i) * g.mb_words + (size_t)(ja + l) * 2 * R + rowp,
          pack(a + bg[l] + clg[(l * G + i) * 2 * R + rowp], (unsigned)(ts + 1)), lm(l));
  };

  stage(tg0, true);
  if (sy.failed()) return;
  for (int i = 0; i < ns; ++i)
#pragma unroll
    for (int l = 0; l < NLA; ++l)
      if (l < nl) post_pre(l, tg0, i);
  for (int64_t t = tg0; t < tg0 + T; ++t) {
    const bool more = (t + 1 < tg0 + T);
    // A host abort request, read every WN_ABORT_CHECK steps by the replica's first aux CU, which
    // works a step ahead of the chain, so the read's PCIe round trip stays off the critical path.
    // It stops here; every other role sees the status word in its next wait and leaves too.
    if (ai == 0 && threadIdx.x == 0 && ((t - tg0) & (WN_ABORT_CHECK - 1)) == 0 && abort_requested(g.io.abort_flag)) {
      atomicCAS(g.status, 0, (int)WN_EABORTED);
      *sy.flag = 1;
    }
    lds_barrier();
    if (sy.failed()) return;
    if (more) stage(t + 1, false);
    if (sy.failed()) return;
    for (int i = 0; i < ns; ++i) {
      const int b = b0 + i;
      u64* const mbs = g.mb + (size_t)b * g.mb_words;
      float q = 0.f;  // this thread's row of the skip partial, summed over my layers
#pragma unroll
      for (int l = 0; l < NLA; ++l) {
        if (l < nl) {
          const int j = ja + l;
          // Waiting for h_j[t] also paces this CU: once it has arrived the chain has consumed
          // pre_j[t], so posting pre_j[t + 1] below cannot overwrite a slot the chain has yet to read.
          const Items hi{mbs + g.off_h + (size_t)j * R, R, R, R, hs + l * R, (unsigned)(t + 1)};
          if (more && dl[l] == 1) {
            Items xi = hist_items(l, t + 1);
            xi.base += (size_t)i * g.d.hist_len;
            xi.n = R;
            xi.dst = xpg + (l * G + i) * R;
            poll2(g, hi, xi, dyn, sy);
          } else {
            poll2(g, hi, no_items(), dyn, sy);
          }
          lds_barrier();
          if (sy.failed()) return;
          // the partial goes out as soon as its last layer is in: a later layer of this CU (the
          // network's last, whose skip is on the chain) only paces the pre-activations
          if (SKL && l == 0 && l < nsk) {
            // W_skip from LDS: 8-lane group q takes rows RPG q .. RPG q + RPG - 1, lane i the
            // chunks i, i + 8, ... of each row; a full sum ends on a lane pair of every row
            float p[RPG];
#pragma unroll
            for (int rr = 0; rr < RPG; ++rr) p[rr] = 0.f;
#pragma unroll
            for (int m = 0; m < R / 32; ++m) {
              const int k = 4 * (li + 8 * m);
              const float4 v = *reinterpret_cast<const float4*>(hs + l * R + k);
#pragma unroll
              for (int rr = 0; rr < RPG; ++rr) {
                const float4 a = *reinterpret_cast<const float4*>(wska + (RPG * gq + rr) * WSKA + k);
                p[rr] = fmaf(a.x, v.x, fmaf(a.y, v.y, fmaf(a.z, v.z, fmaf(a.w, v.w, p[rr]))));
              }
            }
            const float qv = xreduce8<RPG>(p, li);
            const int m = RPG * gq + ((li & 4) ? RPG / 2 : 0) + (RPG == 4 && (li & 2) ? 1 : 0);
            if ((RPG == 4 ? (li & 1) : (li & 3)) == 0) {
              if (nsk == 1) stw(mbs + g.off_q + (size_t)ai * S + m, pack(qv, (unsigned)(t + 1)), lm(16));
              else qsk[m] = qv;  // read by the next layer's lanes of row m, after its barrier
            }
          } else if (l < nsk) {
            float qq = gsum<LPRS>(dot_lds<KCS>(wk[l - (SKL ? 1 : 0)], hs + l * R + ks * KCS));
            if (SKL && l == 1) qq += qsk[rows];
            q += qq;
            if (l == nsk - 1 && ks == 0)
              stw(mbs + g.off_q + (size_t)ai * S + rows, pack(q, (unsigned)(t + 1)), lm(16));
          }
        }
      }
      if (more) {
#pragma unroll
        for (int l = 0; l < NLA; ++l)
          if (l < nl) post_pre(l, t + 1, i);
      }
      lds_barrier();
    }
  }
}

// ------------------------------------------------------------------------------------------
// head CU: rows [64 h, 64 h + 64) of z_a and their share of the logits
// ------------------------------------------------------------------------------------------
template <int R, int S, bool TF, bool MS, class LM>
__device__ __forceinline__ void head_role(const WnChainArgs& g, const int hh, const int b0, const int ns, float* dyn, Sync sy,
                          const int64_t tg0, const LM lm) {
  constexpr int LPRH = NT / HR, KCH = S / LPRH;   // W_relu: 8 lanes per row
  constexpr int LPRO = NT / A, KCO = HR / LPRO;   // W_out: 2 lanes per output
  const int tid = threadIdx.x;
  const int L = g.d.L;
  const int T = g.io.T;
  const int nq = g.naux_q;      // skip partials that come from aux CUs (one per aux CU with a skip layer)
  float* qall = dyn;           // (nq + 1)*S skip partials of one step: the aux CUs', then the tail
  float* zs = qall + L * S;    // S
  float* za = zs + S;          // HR
  float* qpart = za + HR;      // 2 NT per-thread partial sums (two channels per thread)
  static_assert((2 * NT) % S == 0 && S % 2 == 0, "a thread's skip pairs share two channels");

  const int rl = tid / LPRH, kr = tid % LPRH;
  const int oo = tid / LPRO, ko = tid % LPRO;
  float wl[KCH], wo[KCO];
  const float* Wl = static_cast<const float*>(g.w.w_relu);
  const float* Wo = static_cast<const float*>(g.w.w_out);
#pragma unroll
  for (int i = 0; i < KCH; ++i) wl[i] = Wl[(size_t)(hh * HR + rl) * S + 4 * (kr + LPRH * (i / 4)) + i % 4];
#pragma unroll
  for (int i = 0; i < KCO; ++i) wo[i] = Wo[(size_t)oo * A + hh * HR + ko * KCO + i];
  const float bl = g.w.b_relu[hh * HR + rl];
  const float bsk = g.w.b_skip[tid % S];

  for (int64_t t = tg0; t < tg0 + T; ++t) {
    const unsigned tag = (unsigned)(t + 1);
    for (int i = 0; i < ns; ++i) {
      u64* const mbs = g.mb + (size_t)(b0 + i) * g.mb_words;
      // all skip partials of this step: sum_j W_skip_j h_j over each aux CU's layers and (when the
      // last chain CU computes it) the last layer's.  Item i is channel i mod S of partial i / S and
      // pair p (items 2p, 2p + 1) belongs to thread p mod NT, so thread tid polls channels
      // 2 tid mod S and 2 tid mod S + 1 of every (2 NT / S)-th partial, from partial 2 tid / S on,
      // and sums each channel's as they arrive; the 2 NT / S partial sums of a channel then meet in
      // LDS, in a fixed order.
      float part[2] = {0.f, 0.f};
      poll2<3>(g, Items{mbs + g.off_q, S, S, nq * S, qall, tag},
               g.tail_on_chain ? Items{mbs + g.off_qtail, S, S, S, qall + nq * S, tag} : no_items(),
               dyn, sy, part);
      qpart[(2 * tid / S) * S + (2 * tid) % S] = part[0];
      qpart[(2 * tid / S) * S + (2 * tid) % S + 1] = part[1];
      lds_barrier();
      if (sy.failed()) return;
      // z_s = relu(B_skip + sum_j q_j)
      if (tid < S) {
        float q = bsk;
#pragma unroll
        for (int p = 0; p < 2 * NT / S; ++p) q += qpart[p * S + tid];
        zs[tid] = fmaxf(q, 0.f);
      }
      lds_barrier();
      {
        const float v = gsum<LPRH>(dot_lds_il<KCH, LPRH>(wl, zs + 4 * kr));
        if (kr == 0) za[rl] = fmaxf(v + bl, 0.f);
      }
      lds_barrier();
      {
        const float v = gsum<LPRO>(dot_lds<KCO>(wo, za + ko * KCO));
        if (ko == 0) stw(mbs + g.off_logit + (size_t)hh * A + oo, pack(v, tag), lm(0));
      }
      lds_barrier();
    }
  }
}

template <int R, int S, int NLC, bool TF, bool MS, bool E2, bool AX>
__global__ __launch_bounds__(NT) void wn_chain_kernel(const WnChainArgs g) {
  extern __shared__ __align__(16) float dyn[];
  __shared__ int s_abort;
  const int rb = g.role_of_block[blockIdx.x];
  if (rb == 0xffff) return;
  const int per = g.nch + NHEAD + g.naux;
  const int k = MS ? rb / per : 0, role = rb - k * per;
  const int b0 = MS ? k * g.G : 0;
  const int ns = MS ? min(g.G, g.io.B - b0) : 1;  // streams of this replica
  if (ns <= 0) return;
  if (threadIdx.x == 0) s_abort = 0;
  // Which of this block's posts go to a reader on its own XCD (block b runs on XCD b mod 8, which
  // the host has checked on this device): bit l of a chain CU for the aux CU of its layer l (h
  // and the history rows), bit 16 for the next chain CU, bit 17 for the head CUs; bit l of an aux
  // CU for the chain CU of its layer l, bit 16 for the head CUs; bit 0 of a head CU for chain CU 0.
  // When every role of the replica runs on the block's XCD, the roles run their all-local build.
  __shared__ unsigned char s_xcd[WN_MAX_CHAIN + NHEAD + WN_MAX_LAYERS];
  __shared__ int s_me;
  unsigned lm = 0;
  bool all_local = false;  // every role of the replica on this block's XCD
  if (g.local_posts) {
    // The XCD of every block is read at each launch, not assumed: each block stores its XCC_ID, the
    // grid meets once (a cooperative launch keeps every block resident), and each block builds its
    // masks from the map it then reads, so a post is stored at workgroup scope only when its reader
    // runs on the writer's XCD in this launch.  (The host's placement assumes block b on XCD b mod 8;
    // a different map only costs hop latency.)
    if (grid_meet(g.xmap, g.n_active, g.spin_limit, g.status, &s_me) < 0) return;  // WN_ETIMEOUT is in the status word
    for (int b = threadIdx.x; b < WN_CHAIN_GRID; b += NT) {
      const int r = g.role_of_block[b];
      if (r != 0xffff && (MS ? r / per : 0) == k) s_xcd[r - k * per] = (unsigned char)ldw(g.xmap + b);
    }
    __syncthreads();
    const int me = s_me;
    auto same = [&](int r) { return s_xcd[r] == me; };
    const bool heads = same(g.nch) && same(g.nch + 1) && same(g.nch + 2) && same(g.nch + 3);
    all_local = true;
    for (int r = 0; r < per; ++r) all_local = all_local && same(r);
    if (role < g.nch) {
      const int j0 = g.layer_begin[role], nl = g.layer_begin[role + 1] - j0;
      for (int l = 0; l < nl; ++l) lm |= (unsigned)same(g.nch + NHEAD + (j0 + l) / g.nla) << l;
      if (role + 1 < g.nch) lm |= (unsigned)same(role + 1) << 16;
      lm |= (unsigned)heads << 17;
    } else if (role < g.nch + NHEAD) {
      lm = same(0);
    } else {
      const int ja = (role - g.nch - NHEAD) * g.nla;
      for (int l = 0; l < g.nla && ja + l < g.d.L; ++l) {
        int c = 0;
        while (g.layer_begin[c + 1] <= ja + l) ++c;
        lm |= (unsigned)same(c) << l;
      }
      lm |= (unsigned)heads << 16;
    }
  }
  // where this call starts: from zero, or where the previous call on this workspace stopped (the
  // replica's chain CU 0 rewrites its streams' state only after every role of it has started)
  const int64_t tg0 = g.io.reset ? 0 : g.state[WN_STATE_WORDS * (size_t)b0];
  __syncthreads();
  Sync sy{&s_abort};
  auto run = [&](auto loc) {
    if (role < g.nch) {
      // the all-local one-stream build also fixes the layer count of the common chain CUs at compile
      // time (with the stream loop, those builds spill)
      const int nl = g.layer_begin[role + 1] - g.layer_begin[role];
      constexpr bool FIX = std::is_same<decltype(loc), Local<true>>::value && !MS;
      constexpr int K1 = FIX ? NLC : 0, K2 = (FIX && NLC > 1) ? NLC - 1 : 0;
      if (K1 > 0 && nl == K1) chain_role<R, S, NLC, TF, MS, E2, AX, K1>(g, role, b0, ns, dyn, sy, tg0, loc);
      else if (K2 > 0 && nl == K2) chain_role<R, S, NLC, TF, MS, E2, AX, K2>(g, role, b0, ns, dyn, sy, tg0, loc);
      else chain_role<R, S, NLC, TF, MS, E2, AX, 0>(g, role, b0, ns, dyn, sy, tg0, loc);
    }
    else if (role < g.nch + NHEAD) head_role<R, S, TF, MS>(g, role - g.nch, b0, ns, dyn, sy, tg0, loc);
    else aux_role<R, S, TF, MS>(g, role - g.nch - NHEAD, b0, ns, dyn, sy, tg0, loc);
  };
  if (all_local) run(Local<true>{lm});
  else run(Local<false>{lm});
}

// Clears the tagged histories and mailboxes and the status word before a run from zero.
__global__ void wn_chain_reset_kernel(u64* words, size_t n, int* status) {
  const size_t i0 = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (size_t i = i0; i < n; i += (size_t)gridDim.x * blockDim.x) words[i] = 0ull;
  if (i0 == 0) *status = 0;
}

template <int R>
constexpr int chain_nlc() { return R == 128 ? 2 : (R == 64 ? 7 : 16); }

int nlc_for(int R) { return R == 128 ? chain_nlc<128>() : (R == 64 ? chain_nlc<64>() : chain_nlc<32>()); }

// Layers of each chain CU: runs of at most nlc layers, as even as possible.  With r = 128 the
// first CU (which also holds the embedding table) and the last (which holds the last layer's
// W_skip) take one layer each, since two layers' W_res only fit in the LDS of the CUs between.
int chain_split(int L, int R, int* layer_begin) {
  const int nlc = nlc_for(R);
  int first = 0, last = 0, mid = L;
  if (R == 128 && L >= 2) {
    first = 1;
    last = 1;
    mid = L - 2;
  }
  const int nmid = (mid + nlc - 1) / nlc;
  const int nch = (first ? 1 : 0) + nmid + (last ? 1 : 0);
  if (nch > WN_MAX_CHAIN) return nch;
  int c = 0;
  layer_begin[0] = 0;
  if (first) {
    layer_begin[1] = 1;
    c = 1;
  }
  const int base = nmid ? mid / nmid : 0, extra = nmid ? mid % nmid : 0;
  for (int k = 0; k < nmid; ++k, ++c) layer_begin[c + 1] = layer_begin[c] + base + (k < extra ? 1 : 0);
  if (last) layer_begin[c + 1] = layer_begin[c] + 1;
  return nch;
}

// Dynamic LDS floats of each role (the launch takes the largest); mirrors the carving in the roles.
size_t chain_lds_floats(int R, int S, int nlc, int G, int ub, int nch, int tail, bool e2) {
  const int nlcp = (nlc + 3) & ~3;
  const size_t common = (size_t)2 * R + (size_t)nlc * 2 * R + (size_t)2 * nlc * R + 4 * nlcp;
  const size_t wsk = (size_t)S * lds_row_stride(R, S / 64);
  size_t cu0 = (size_t)NHEAD * A + (size_t)2 * G * ub + 2 * ((G + 3) & ~3) + (size_t)A * R;
  if (e2 && e2_in_lds(R)) cu0 += (size_t)A * R;
  if (nch == 1 && tail) cu0 += wsk;
  size_t var = cu0;
  if (tail) var = std::max(var, wsk);
  if (R == 128) var = std::max(var, (size_t)2 * R * lds_row_stride(R, 2));
  return common + var;
}
size_t head_lds_floats(int L, int S) { return (size_t)L * S + S + HR + 2 * NT; }
size_t aux_lds_floats(int R, int S, int G, int nla) {
  const bool skl = R <= 64 ? aux_skip_in_lds<64>() : aux_skip_in_lds<128>();
  return (size_t)nla * ((size_t)R + (size_t)3 * R * G) + (skl ? (size_t)S * lds_row_stride(R, S / 64) + S : 0);
}
constexpr size_t kMaxLds = 160 * 1024;

template <int R, int S>
hipError_t launch_chain_rs(const WnChainArgs& g, bool teacher, hipStream_t stream) {
  constexpr int NLC = chain_nlc<R>();
  const size_t dyn = sizeof(float) * std::max(chain_lds_floats(R, S, NLC, g.G, g.ub, g.nch, g.tail_on_chain,
                                                                g.w.embed_prev != nullptr),
                                              std::max(head_lds_floats(g.d.L, S), aux_lds_floats(R, S, g.G, g.nla)));
  void* args[] = {const_cast<WnChainArgs*>(&g)};
  // one stream (no replicas) gets a build with the stream loops folded away, a one-table
  // embedding one without the second table's load; the approximate nonlinearities are built
  // only with the stream loops (they serve one stream too)
  const bool ax = g.w.approx_nl != 0, ms = g.io.B > 1 || ax, e2 = g.w.embed_prev != nullptr;
  auto pick = [&](auto tf, auto msc) -> const void* {
    constexpr bool TF = decltype(tf)::value, MS = decltype(msc)::value;
    if constexpr (MS) {
      if (ax)
        return e2 ? reinterpret_cast<const void*>(wn_chain_kernel<R, S, NLC, TF, true, true, true>)
                  : reinterpret_cast<const void*>(wn_chain_kernel<R, S, NLC, TF, true, false, true>);
    }
    return e2 ? reinterpret_cast<const void*>(wn_chain_kernel<R, S, NLC, TF, MS, true, false>)
              : reinterpret_cast<const void*>(wn_chain_kernel<R, S, NLC, TF, MS, false, false>);
  };
  using t_ = std::true_type;
  using f_ = std::false_type;
  const void* k = teacher ? (ms ? pick(t_{}, t_{}) : pick(t_{}, f_{})) : (ms ? pick(f_{}, t_{}) : pick(f_{}, f_{}));
  hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
  if (e != hipSuccess) return e;
  return hipLaunchCooperativeKernel(k, dim3(WN_CHAIN_GRID), dim3(NT), args, (unsigned)dyn, stream);
}

}  // namespace

bool wn_chain_supported(int R, int S, int L) {
  if (!((R == 128 && S == 256) || (R == 64 && (S == 256 || S == 128)) || (R == 32 && S == 128))) return false;
  if (L < 1 || L > WN_MAX_LAYERS) return false;
  int lb[WN_MAX_LAYERS + 2];
  const int nch = chain_split(L, R, lb);
  const int nla = R <= 64 ? aux_max_layers<64>() : aux_max_layers<128>();
  return L >= 1 && L <= WN_MAX_LAYERS && nch <= WN_MAX_CHAIN && nch + NHEAD + (L + nla - 1) / nla <= WN_CHAIN_GRID &&
         head_lds_floats(L, S) * sizeof(float) <= kMaxLds;
}

bool wn_chain_plan(int L, int R, int S, int B, bool two_taps, WnChainPlan* p) {
  if (!p || B < 1 || !wn_chain_supported(R, S, L)) return false;
  WnChainPlan q{};
  const int nlc = nlc_for(R);
  q.nch = chain_split(L, R, q.layer_begin);
  // layers per aux CU: as many as fit its registers (WN_AUX_LAYERS=1 keeps one layer each), fewer
  // where the aux CUs' staging of more streams per replica would not fit their LDS (r = 128)
  int nla_max = R <= 64 ? aux_max_layers<64>() : aux_max_layers<128>();
  if (const char* e = std::getenv("WN_AUX_LAYERS")) {
    const int v = std::atoi(e);
    if (v >= 1 && v <= nla_max) nla_max = v;
  }
  int per = 0;
  for (q.nla = nla_max; q.nla >= 1; --q.nla) {
    q.naux = (L + q.nla - 1) / q.nla;
    // as many replicas as the grid holds, the streams spread evenly over them
    per = q.nch + NHEAD + q.naux;
    const int max_rep = WN_CHAIN_GRID / per;
    if (max_rep < 1) continue;
    q.G = (B + std::min(B, max_rep) - 1) / std::min(B, max_rep);
    q.nrep = (B + q.G - 1) / q.G;
    if (q.G <= WN_CHAIN_MAX_G && aux_lds_floats(R, S, q.G, q.nla) * sizeof(float) <= kMaxLds) break;
  }
  if (q.nla < 1) return false;
  int gp = 1;
  while (gp < q.G) gp *= 2;
  q.ub = std::max(16, 512 / gp);
  q.tail_on_chain = 1;
  if (chain_lds_floats(R, S, nlc, q.G, q.ub, q.nch, 1, two_taps) * sizeof(float) > kMaxLds) q.tail_on_chain = 0;
  if (chain_lds_floats(R, S, nlc, q.G, q.ub, q.nch, q.tail_on_chain, two_taps) * sizeof(float) > kMaxLds)
    return false;
  // aux CUs that post a skip partial: all but one holding only the last layer when the last chain
  // CU computes that layer's skip projection
  q.naux_q = (q.tail_on_chain && (L - 1) % q.nla == 0) ? q.naux - 1 : q.naux;
  // mailboxes of one stream: pre, h, q, x, logits, tail (see WnChainArgs)
  const long long pre_w = (long long)L * 2 * R;
  q.off_h = (int)pre_w;
  q.off_q = q.off_h + L * R;
  q.off_x = q.off_q + q.naux * S;
  q.off_logit = q.off_x + q.nch * R;
  q.off_qtail = q.off_logit + NHEAD * A;
  q.mb_words = ((long long)q.off_qtail + S + 31) / 32 * 32;
  // Placement: slot i of XCD x is block 8 i + x.  Each replica's chain and head CUs go to its home
  // XCD first, then its aux CUs, last layers first (their skip partials are the last ones the head
  // waits for), overflowing to the XCD with the most room.
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
    for (int r = 0; r < q.nch + NHEAD; ++r) place(k * per + r, k % 8);
  for (int k = 0; k < q.nrep; ++k)
    for (int a = q.naux - 1; a >= 0; --a) place(k * per + q.nch + NHEAD + a, k % 8);
  *p = q;
  return true;
}

// XCD of every block of a cooperative launch of the multi-CU kernel's grid.
__global__ void wn_xcc_probe_kernel(int* ids) {
  if (threadIdx.x == 0) {
    unsigned v;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
    ids[blockIdx.x] = (int)(v & 0xf);
  }
}

bool wn_chain_xcd_map_ok() {
  int* d = nullptr;
  if (hipMalloc(&d, WN_CHAIN_GRID * sizeof(int)) != hipSuccess) return false;
  void* args[] = {&d};
  bool ok = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(wn_xcc_probe_kernel), dim3(WN_CHAIN_GRID),
                                       dim3(64), args, 0, nullptr) == hipSuccess &&
            hipDeviceSynchronize() == hipSuccess;
  int h[WN_CHAIN_GRID];
  ok = ok && hipMemcpy(h, d, sizeof(h), hipMemcpyDeviceToHost) == hipSuccess;
  for (int b = 0; ok && b < WN_CHAIN_GRID; ++b) ok = h[b] == b % 8;
  (void)hipFree(d);
  return ok;
}

__global__ void wn_status_clear_kernel(int* status) { *status = 0; }

hipError_t wn_status_clear(int* status, hipStream_t stream) {
  hipLaunchKernelGGL(wn_status_clear_kernel, dim3(1), dim3(1), 0, stream, status);
  return hipGetLastError();
}

hipError_t wn_chain_reset(unsigned long long* words, size_t n, int* status, hipStream_t stream) {
  hipLaunchKernelGGL(wn_chain_reset_kernel, dim3(256), dim3(256), 0, stream, words, n, status);
  return hipGetLastError();
}

hipError_t wn_chain_launch(const WnChainArgs& g, bool teacher, hipStream_t stream) {
  const int R = g.d.R, S = g.d.S;
  if (R == 128 && S == 256) return launch_chain_rs<128, 256>(g, teacher, stream);
  if (R == 64 && S == 256) return launch_chain_rs<64, 256>(g, teacher, stream);
  if (R == 64 && S == 128) return launch_chain_rs<64, 128>(g, teacher, stream);
  if (R == 32 && S == 128) return launch_chain_rs<32, 128>(g, teacher, stream);
  return hipErrorInvalidValue;
}
