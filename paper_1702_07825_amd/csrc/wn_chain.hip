// Multi-CU persistent generation kernel for one stream (B = 1), fp32, gfx950.
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
//   aux CUs    (one per layer) hold W_prev and W_skip in VGPRs.  For the NEXT step
//              they compute pre = W_prev x[t+1-d] + B + L[t+1] (so the dilated half,
//              the bias and the HBM read of the conditioning all happen a step
//              early), and for the current step the skip partial W_skip h.
//   head CUs   (four) hold 64 rows of W_relu and the matching 64 columns of W_out:
//              z_a = relu(W_relu relu(q) + B_relu) for their rows and the partial
//              logits W_out[:, rows] z_a[rows].
//
// Messages between CUs are vectors of 64-bit words (fp32 value in the low half,
// step + 1 in the high half) written and read with relaxed agent-scope atomics.
// Every word carries its own step tag, so a reader needs no fence: it re-reads a
// word until the tag it expects appears.  Each mailbox has two slots (step
// parity); the dependency chain keeps every producer at most one step ahead of
// its consumer.  The dilation histories are rings of tagged words in the
// workspace: slot (t mod d) of layer j holds x_{j-1}[t] tagged t + 1.
//
// Every wait is bounded.  A block that times out stores WN_ETIMEOUT in the
// workspace status word; every waiting block polls that word and leaves, so the
// grid always drains.  Block b takes role (b mod 8) * 32 + b / 8, which puts
// roles 0..31 (the chain and head CUs and the first aux CUs) on one XCD when
// blocks are dealt round-robin over the eight XCDs; the protocol does not depend
// on that placement, only the hop latency does.
#include "wn_internal.h"
#include "wn_wave.h"

#include "wn.h"

#include <algorithm>

namespace {

using namespace wnk;

constexpr int NT = 512;
constexpr int A = WN_A;
constexpr int NHEAD = 4;
constexpr int HR = A / NHEAD;  // z_a rows per head CU
constexpr int UB = 512;        // per-step host inputs / outputs staged in LDS

typedef unsigned long long u64;

__device__ __forceinline__ u64 pack(float v, unsigned tag) {
  return ((u64)tag << 32) | (u64)__float_as_uint(v);
}
__device__ __forceinline__ float wval(u64 w) { return __uint_as_float((unsigned)w); }
__device__ __forceinline__ unsigned wtag(u64 w) { return (unsigned)(w >> 32); }
__device__ __forceinline__ u64 ldw(const u64* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void stw(u64* p, u64 w) {
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int ld_status(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Block-uniform abort flag kept in LDS.
struct Sync {
  int* flag;
  __device__ bool failed() const { return *flag != 0; }
};

// A set of tagged words to wait for: item i lives at base + (i / len) * stride + i % len and
// its value goes to dst[i].
struct Items {
  const u64* base;
  int len, stride, n;
  float* dst;
  unsigned tag;  // the step tag the words must carry
};
__device__ __forceinline__ Items no_items() { return Items{nullptr, 1, 0, 0, nullptr, 0u}; }

// Wait until every item of `a` and `b` owned by this thread (item i belongs to thread i mod NT)
// carries its descriptor's tag, writing the values to LDS (dst pointers lie in `lds`).  All owned
// loads are in flight together.  A thread that times out, or sees a nonzero status word, sets the
// block's abort flag and stops waiting.  Every polled word lies in the workspace's tagged region,
// which starts at g.ring; items are tracked as 32-bit word offsets from there.
__device__ void poll2(const WnChainArgs& g, const Items a, const Items b, float* lds, Sync s) {
  const int n = a.n + b.n;
  const u64* wbase = g.ring;
  for (int base = threadIdx.x; base < n; base += 4 * NT) {
    u64 w[4];
    unsigned so[4], dofs[4];
    unsigned pend = 0, useb = 0;  // bit k: item base + k * NT pending / belongs to descriptor b
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int i = base + k * NT;
      if (i < n) {
        const bool inb = (i >= a.n);
        const Items& it = inb ? b : a;
        const int ii = inb ? i - a.n : i;
        so[k] = (unsigned)((it.base - wbase) + (size_t)(ii / it.len) * it.stride + (ii % it.len));
        dofs[k] = (unsigned)((it.dst - lds) + ii);
        pend |= 1u << k;
        useb |= (inb ? 1u : 0u) << k;
        w[k] = ldw(wbase + so[k]);
      }
    }
    int spins = 0;
    while (true) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (pend & (1u << k)) {
          if (wtag(w[k]) == ((useb & (1u << k)) ? b.tag : a.tag)) {
            pend &= ~(1u << k);
            lds[dofs[k]] = wval(w[k]);
          }
        }
      }
      if (!pend) break;
      if (++spins > g.spin_limit || ((spins & 63) == 0 && ld_status(g.status) != 0)) {
        if (ld_status(g.status) == 0) atomicCAS(g.status, 0, (int)WN_ETIMEOUT);
        *s.flag = 1;
        return;
      }
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (pend & (1u << k)) w[k] = ldw(wbase + so[k]);
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
};

template <int K>
__device__ __forceinline__ float dot_lds(const float (&w)[K], const float* x) {
  float s0 = 0.f, s1 = 0.f;
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

// ------------------------------------------------------------------------------------------
// chain CU
// ------------------------------------------------------------------------------------------
template <int R, int S, int NLC, bool TF>
__device__ void chain_role(const WnChainArgs& g, const int c, float* dyn, Sync sy, const int64_t tg0, const int yprev0) {
  using M = ChainMap<R>;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int L = g.d.L;
  const int j0 = g.layer_begin[c], nl = g.layer_begin[c + 1] - j0;
  const bool first = (c == 0);
  const int T = g.io.T;

  float* xs = dyn;                    // R      x_{j-1}, updated in place
  float* hs = xs + R;                 // R
  float* pre = hs + R;                // NLC*2R pre-activations of this step
  float* lgp = pre + NLC * 2 * R;     // NHEAD*A partial logits (chain CU 0)
  float* ubuf = lgp + NHEAD * A;      // UB uniforms (generation) / samples in (teacher forcing)
  int* ybuf = reinterpret_cast<int*>(ubuf + UB);  // UB drawn samples
  float* xbuf = reinterpret_cast<float*>(ybuf + UB);  // NLC*R x_{j-1} of this step (history writes)
  float* emb = xbuf + NLC * R;                         // A*R embedding table (chain CU 0)
  float* wsk = emb + A * R;                            // S*R W_skip of layer l-1 (last chain CU)
  float* bres = wsk + S * R;                           // NLC*R B_res of my layers
  __shared__ int s_y;
  const bool lastc = (c + 1 == g.nch);

  // resident weights
  // W_cur: lane group c (LPRG lanes) holds rows c and c + R, lane kq of it inputs kq*KCG .. +KCG
  const int g1 = tid / M::LPRG, kq = tid % M::LPRG;
  const int row2 = tid / M::LPR2, kk = tid % M::LPR2;
  float wc[NLC][2 * M::KCG], wr[NLC][M::KC2];
  const float* Wc = static_cast<const float*>(g.w.w_cur);
  const float* Wr = static_cast<const float*>(g.w.w_res);
#pragma unroll
  for (int l = 0; l < NLC; ++l) {
    const int j = j0 + (l < nl ? l : 0);
#pragma unroll
    for (int i = 0; i < M::KCG; ++i) {
      wc[l][i] = Wc[((size_t)j * 2 * R + g1) * R + kq * M::KCG + i];
      wc[l][M::KCG + i] = Wc[((size_t)j * 2 * R + g1 + R) * R + kq * M::KCG + i];
    }
#pragma unroll
    for (int i = 0; i < M::KC2; ++i) wr[l][i] = Wr[((size_t)j * R + row2) * R + kk * M::KC2 + i];
  }
  for (int i = tid; i < nl * R; i += NT) bres[i] = g.w.b_res[(size_t)j0 * R + i];
  float bemb = 0.f;
  float4 bout4 = make_float4(0.f, 0.f, 0.f, 0.f);  // B_out of the 4 logits lane l of wave 0 draws from
  if (lastc) {
    const float* Wk = static_cast<const float*>(g.w.w_skip) + (size_t)(L - 1) * S * R;
    for (int i = tid; i < S * R; i += NT) wsk[i] = Wk[i];
  }
  if (first) {
    if (wave == 0) bout4 = *reinterpret_cast<const float4*>(g.w.b_out + 4 * lane);
    const float* E = static_cast<const float*>(g.w.embed);
    for (int i = tid; i < A * R; i += NT) emb[i] = E[i];
    if (tid < R) bemb = g.w.b_embed[tid];
    if (tid == 0) s_y = yprev0;
  }
  int64_t ub0 = tg0;  // first global step held in ubuf / ybuf
  if (first) {
    for (int i = tid; i < UB; i += NT) {
      const int64_t t = tg0 + i;
      if (t < tg0 + T) {
        if constexpr (TF) reinterpret_cast<int*>(ubuf)[i] = g.io.y_in[t - tg0];
        else ubuf[i] = g.io.u[t - tg0];
      }
    }
  }
  lds_barrier();

  // One wave sums the head's partial logits of global step ts (lane l owns logits 4l..4l+3),
  // writes them out when teacher forcing, and draws (generation) or reads (teacher forcing)
  // the sample.
  auto sample_step = [&](int64_t ts) {
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
      int y;
      if constexpr (TF) {
        *reinterpret_cast<float4*>(g.io.logits + (size_t)(ts - tg0) * A + 4 * lane) = lv;
        y = reinterpret_cast<const int*>(ubuf)[ts - ub0];
        y = y < 0 ? 0 : (y > A - 1 ? A - 1 : y);
      } else {
        const float l0 = lv.x, l1 = lv.y, l2 = lv.z, l3 = lv.w;
        const float m = wave_max(fmaxf(fmaxf(l0, l1), fmaxf(l2, l3)));
        const float e0 = expf_fast(l0 - m), e1 = expf_fast(l1 - m), e2 = expf_fast(l2 - m), e3 = expf_fast(l3 - m);
        const float s0 = e0, s1 = s0 + e1, s2 = s1 + e2, s3 = s2 + e3;
        const float incl = wave_incl_scan(s3);
        const float excl = wave_shr1(incl);
        const float Z = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, incl), 63));
        const float iz = 1.0f / Z;
        const float u = ubuf[ts - ub0];
        int cnt = ((excl + s0) * iz <= u) + ((excl + s1) * iz <= u) + ((excl + s2) * iz <= u);
        if (lane != 63) cnt += ((excl + s3) * iz <= u);
        y = wave_sum_int(cnt);
      }
      if (lane == 0) {
        s_y = y;
        ybuf[ts - ub0] = y;
      }
    }
  };
  // The head's partial logits of step ts (tag ts + 1).
  auto logit_items = [&](int64_t ts) {
    return Items{g.mb_logit + (size_t)(ts & 1) * A, A, 2 * A, NHEAD * A, lgp, (unsigned)(ts + 1)};
  };
  // Move staged samples to the output and stage the next block of inputs.
  auto roll_buffers = [&](int64_t next0) {
    if constexpr (!TF) {
      for (int i = tid; i < UB; i += NT) {
        const int64_t t = ub0 + i;
        if (t < next0 && t < tg0 + T) g.io.y_out[t - tg0] = ybuf[i];
      }
    }
    lds_barrier();
    ub0 = next0;
    for (int i = tid; i < UB; i += NT) {
      const int64_t t = ub0 + i;
      if (t < tg0 + T) {
        if constexpr (TF) reinterpret_cast<int*>(ubuf)[i] = g.io.y_in[t - tg0];
        else ubuf[i] = g.io.u[t - tg0];
      }
    }
    lds_barrier();
  };

  for (int64_t t = tg0; t < tg0 + T; ++t) {
    const unsigned tag = (unsigned)(t + 1);
    const int par = (int)(t & 1);
    // ---- inputs of this step, all waited for together: the pre-activations of my layers, and
    //      either x from the previous chain CU or (chain CU 0) the previous step's partial logits ----
    const Items pre_items{g.mb_pre + ((size_t)j0 * 2 + par) * 2 * R, 2 * R, 2 * 2 * R, nl * 2 * R, pre, tag};
    if (first) {
      if (t > tg0) {
        poll2(g, logit_items(t - 1), pre_items, dyn, sy);
        lds_barrier();
        if (sy.failed()) return;
        if (t - 1 - ub0 >= UB) roll_buffers(t - 1);
        sample_step(t - 1);
      } else {
        poll2(g, pre_items, no_items(), dyn, sy);
      }
      lds_barrier();
      if (sy.failed()) return;
      if (tid < R) xs[tid] = emb[s_y * R + tid] + bemb;
    } else {
      poll2(g, pre_items, Items{g.mb_x + ((size_t)c * 2 + par) * R, R, R, R, xs, tag}, dyn, sy);
    }
    lds_barrier();
    if (sy.failed()) return;

    // Store data of the per-layer h posts, rotating over HPOST register pairs: a pair is written
    // again HPOST layers after its store was issued, by when that store has completed, so the
    // wait the compiler places before the overwrite costs nothing inside the layer loop.
    constexpr int HPOST = 3;
    u64 hpost[HPOST];
#pragma unroll
    for (int l = 0; l < HPOST; ++l) hpost[l] = 0;
#pragma unroll
    for (int l = 0; l < NLC; ++l) {
      if (l < nl) {
        const int j = j0 + l;
        // a = W_cur x + pre ; h = tanh(a[0:R]) * sigmoid(a[R:2R]).  Each lane has both rows of its
        // pair; lane 0 of the group starts its partial sums from pre, so pre joins the reduction.
        float ah, ag;
        {
          float sh0 = 0.f, sh1 = 0.f, sg0 = 0.f, sg1 = 0.f;
          if (kq == 0) {
            sh0 = pre[l * 2 * R + g1];
            sg0 = pre[l * 2 * R + g1 + R];
          }
          const float* xk = xs + kq * M::KCG;
          if constexpr (M::KCG % 4 == 0) {
#pragma unroll
            for (int i = 0; i < M::KCG; i += 4) {
              const float4 v = *reinterpret_cast<const float4*>(xk + i);
              sh0 = fmaf(wc[l][i], v.x, sh0);
              sh1 = fmaf(wc[l][i + 1], v.y, sh1);
              sh0 = fmaf(wc[l][i + 2], v.z, sh0);
              sh1 = fmaf(wc[l][i + 3], v.w, sh1);
              sg0 = fmaf(wc[l][M::KCG + i], v.x, sg0);
              sg1 = fmaf(wc[l][M::KCG + i + 1], v.y, sg1);
              sg0 = fmaf(wc[l][M::KCG + i + 2], v.z, sg0);
              sg1 = fmaf(wc[l][M::KCG + i + 3], v.w, sg1);
            }
          } else {
            static_assert(M::KCG % 2 == 0, "inputs per lane must be even");
#pragma unroll
            for (int i = 0; i < M::KCG; i += 2) {
              const float2 v = *reinterpret_cast<const float2*>(xk + i);
              sh0 = fmaf(wc[l][i], v.x, sh0);
              sh1 = fmaf(wc[l][i + 1], v.y, sh1);
              sg0 = fmaf(wc[l][M::KCG + i], v.x, sg0);
              sg1 = fmaf(wc[l][M::KCG + i + 1], v.y, sg1);
            }
          }
          ah = gsum<M::LPRG>(sh0 + sh1);
          ag = gsum<M::LPRG>(sg0 + sg1);
        }
        const float h = tanh_f(ah) * sigmoid_f(ag);
        if (kq == 0) {
          hs[g1] = h;
        }
        lds_barrier();
        // h_j[t] -> layer j's aux CU (skip projection)
        if (wave == NT / 64 - 1 && lane < R) {
          // an opaque lane index keeps the compiler from hoisting one 64-bit address per layer
          // out of the step loop (they would not fit in registers)
          int ln = lane;
          asm volatile("" : "+v"(ln));
          hpost[l % HPOST] = pack(hs[ln], tag);
          stw(g.mb_h + ((size_t)j * 2 + par) * R + ln, hpost[l % HPOST]);
        }
        // x_j = x_{j-1} + W_res h + B_res (x_l feeds nothing); x_{j-1} is kept for the history
        if (j < L - 1) {
          const float xo = xs[row2], bo = bres[l * R + row2];
          const float r = gsum<M::LPR2>(dot_lds<M::KC2>(wr[l], hs + kk * M::KC2));
          if (kk == 0) {
            xbuf[l * R + row2] = xo;
            xs[row2] = xo + r + bo;
          }
        } else if (tid < R) {
          xbuf[l * R + tid] = xs[tid];
        }
        lds_barrier();
      }
    }
    // The last chain CU adds the skip projection of the last layer itself (its W_skip is in LDS),
    // which saves the hop through that layer's aux CU on the way to the head.
    if (lastc) {
      constexpr int LPRS = NT / S, KCS = R / LPRS;
      const int m = tid / LPRS, ks = tid % LPRS;
      float acc0 = 0.f, acc1 = 0.f;
      const float* wrow = wsk + m * R + ks * KCS;
      const float* hk = hs + ks * KCS;
#pragma unroll
      for (int i = 0; i < KCS; i += 4) {
        const float4 w4 = *reinterpret_cast<const float4*>(wrow + i);
        const float4 h4 = *reinterpret_cast<const float4*>(hk + i);
        acc0 = fmaf(w4.x, h4.x, acc0);
        acc1 = fmaf(w4.y, h4.y, acc1);
        acc0 = fmaf(w4.z, h4.z, acc0);
        acc1 = fmaf(w4.w, h4.w, acc1);
      }
      const float q = gsum<LPRS>(acc0 + acc1);
      if (ks == 0) stw(g.mb_qtail + (size_t)par * S + m, pack(q, tag));
    }
    // Then, one or two words per lane: x for the next chain CU, and x_{j-1} into the history
    // slot (t mod d_j) that layer j's aux CU reads again at t + d_j.
    {
      const int nx = (c + 1 < g.nch) ? R : 0;
      for (int i = tid; i < nx + nl * R; i += NT) {
        if (i < nx) {
          stw(g.mb_x + ((size_t)(c + 1) * 2 + par) * R + i, pack(xs[i], tag));
        } else {
          const int k = i - nx, l = k / R, e = k % R, j = j0 + l;
          const int slot = (int)(t % g.d.dil[j]);
          stw(g.ring + g.d.hoff[j] + (size_t)slot * R + e, pack(xbuf[l * R + e], tag));
        }
      }
    }
#pragma unroll
    for (int l = 0; l < HPOST; ++l) asm volatile("" ::"v"(hpost[l]));
  }
  if (first) {
    if (T > 0) {
      const int64_t tl = tg0 + T - 1;
      poll2(g, logit_items(tl), no_items(), dyn, sy);
      lds_barrier();
      if (sy.failed()) return;
      if (tl - ub0 >= UB) roll_buffers(tl);
      sample_step(tl);
      lds_barrier();
      roll_buffers(tg0 + T);
    }
    if (tid == 0 && !sy.failed()) {
      g.state[0] = tg0 + T;
      g.state[1] = s_y;
    }
  }
}

// ------------------------------------------------------------------------------------------
// aux CU (one per layer): pre-activations of the next step and the skip partial
// ------------------------------------------------------------------------------------------
template <int R, int S, bool TF>
__device__ void aux_role(const WnChainArgs& g, const int j, float* dyn, Sync sy, const int64_t tg0) {
  using M = ChainMap<R>;
  constexpr int LPRS = NT / S, KCS = R / LPRS;
  const int tid = threadIdx.x;
  const int L = g.d.L, d = g.d.dil[j];
  const int T = g.io.T;
  float* xp = dyn;        // R   history read
  float* hs = xp + R;     // R
  float* cl = hs + R;     // 2R  conditioning of the target step

  const int rowp = tid / M::LPR1, kq = tid % M::LPR1;
  const int rows = tid / LPRS, ks = tid % LPRS;
  float wp[M::KC1], wk[KCS];
  const float* Wp = static_cast<const float*>(g.w.w_prev);
  const float* Wk = static_cast<const float*>(g.w.w_skip);
#pragma unroll
  for (int i = 0; i < M::KC1; ++i) wp[i] = Wp[((size_t)j * 2 * R + rowp) * R + kq * M::KC1 + i];
#pragma unroll
  for (int i = 0; i < KCS; ++i) wk[i] = Wk[((size_t)j * S + rows) * R + ks * KCS + i];
  const float bg = g.w.b_gate[j * 2 * R + rowp];

  // pre_j[ts] = W_prev x_{j-1}[ts - d] + B + L[ts], posted with tag ts + 1
  auto make_pre = [&](int64_t ts) {
    const int slot = (int)(ts % d);
    const unsigned etag = (ts - d >= 0) ? (unsigned)(ts - d + 1) : 0u;
    poll2(g, Items{g.ring + g.d.hoff[j] + (size_t)slot * R, R, R, R, xp, etag}, no_items(), dyn, sy);
    if (tid >= 64 && tid < 64 + 2 * R)
      cl[tid - 64] = g.io.cond[((size_t)(ts - tg0) * L + j) * 2 * R + (tid - 64)];
    lds_barrier();
    if (sy.failed()) return;
    const float a = gsum<M::LPR1>(dot_lds<M::KC1>(wp, xp + kq * M::KC1));
    if (kq == 0)
      stw(g.mb_pre + ((size_t)j * 2 + (ts & 1)) * 2 * R + rowp, pack(a + bg + cl[rowp], (unsigned)(ts + 1)));
    lds_barrier();
  };

  make_pre(tg0);
  const bool skip_here = (j < L - 1);  // the last layer's skip projection runs on the last chain CU
  for (int64_t t = tg0; t < tg0 + T; ++t) {
    if (sy.failed()) return;
    // Waiting for h_j[t] also paces this CU: once it has arrived the chain has consumed pre_j[t],
    // so posting pre_j[t + 1] below cannot overwrite a slot the chain has yet to read.
    poll2(g, Items{g.mb_h + ((size_t)j * 2 + (t & 1)) * R, R, R, R, hs, (unsigned)(t + 1)}, no_items(), dyn, sy);
    lds_barrier();
    if (sy.failed()) return;
    if (skip_here) {
      const float q = gsum<LPRS>(dot_lds<KCS>(wk, hs + ks * KCS));
      if (ks == 0) stw(g.mb_q + ((size_t)j * 2 + (t & 1)) * S + rows, pack(q, (unsigned)(t + 1)));
    }
    lds_barrier();
    if (t + 1 < tg0 + T) make_pre(t + 1);
  }
}

// ------------------------------------------------------------------------------------------
// head CU: rows [64 h, 64 h + 64) of z_a and their share of the logits
// ------------------------------------------------------------------------------------------
template <int R, int S, bool TF>
__device__ void head_role(const WnChainArgs& g, const int hh, float* dyn, Sync sy, const int64_t tg0) {
  constexpr int LPRH = NT / HR, KCH = S / LPRH;   // W_relu: 8 lanes per row
  constexpr int LPRO = NT / A, KCO = HR / LPRO;   // W_out: 2 lanes per output
  const int tid = threadIdx.x;
  const int L = g.d.L;
  const int T = g.io.T;
  float* qall = dyn;           // L*S skip partials of one step: layers 0..L-2, then the tail
  float* zs = qall + L * S;    // S
  float* za = zs + S;          // HR

  const int rl = tid / LPRH, kr = tid % LPRH;
  const int oo = tid / LPRO, ko = tid % LPRO;
  float wl[KCH], wo[KCO];
  const float* Wl = static_cast<const float*>(g.w.w_relu);
  const float* Wo = static_cast<const float*>(g.w.w_out);
#pragma unroll
  for (int i = 0; i < KCH; ++i) wl[i] = Wl[(size_t)(hh * HR + rl) * S + kr * KCH + i];
#pragma unroll
  for (int i = 0; i < KCO; ++i) wo[i] = Wo[(size_t)oo * A + hh * HR + ko * KCO + i];
  const float bl = g.w.b_relu[hh * HR + rl];
  const float bsk = g.w.b_skip[tid % S];

  for (int64_t t = tg0; t < tg0 + T; ++t) {
    const unsigned tag = (unsigned)(t + 1);
    const int par = (int)(t & 1);
    // all skip partials of this step: W_skip_j h_j from the aux CUs (j < l-1) and the last
    // layer's from the last chain CU
    poll2(g, Items{g.mb_q + (size_t)par * S, S, 2 * S, (L - 1) * S, qall, tag},
          Items{g.mb_qtail + (size_t)par * S, S, S, S, qall + (L - 1) * S, tag}, dyn, sy);
    lds_barrier();
    if (sy.failed()) return;
    // z_s = relu(B_skip + sum_j q_j), summed in layer order
    if (tid < S) {
      float q = bsk;
      for (int j = 0; j < L; ++j) q += qall[j * S + tid];
      zs[tid] = fmaxf(q, 0.f);
    }
    lds_barrier();
    {
      const float v = gsum<LPRH>(dot_lds<KCH>(wl, zs + kr * KCH));
      if (kr == 0) za[rl] = fmaxf(v + bl, 0.f);
    }
    lds_barrier();
    {
      const float v = gsum<LPRO>(dot_lds<KCO>(wo, za + ko * KCO));
      if (ko == 0) stw(g.mb_logit + ((size_t)hh * 2 + par) * A + oo, pack(v, tag));
    }
    lds_barrier();
  }
}

template <int R, int S, int NLC, bool TF>
__global__ __launch_bounds__(NT) void wn_chain_kernel(const WnChainArgs g) {
  extern __shared__ __align__(16) float dyn[];
  __shared__ int s_abort;
  const int b = blockIdx.x;
  const int role = (b % 8) * 32 + b / 8;
  if (role >= g.nch + NHEAD + g.d.L) return;
  if (threadIdx.x == 0) s_abort = 0;
  // where this call starts: from zero, or where the previous call on this workspace stopped
  const int64_t tg0 = g.io.reset ? 0 : g.state[0];
  int yprev0 = g.io.reset ? g.io.init_sample : (int)g.state[1];
  yprev0 = yprev0 < 0 ? 0 : (yprev0 > A - 1 ? A - 1 : yprev0);
  __syncthreads();
  Sync sy{&s_abort};
  if (role < g.nch) chain_role<R, S, NLC, TF>(g, role, dyn, sy, tg0, yprev0);
  else if (role < g.nch + NHEAD) head_role<R, S, TF>(g, role - g.nch, dyn, sy, tg0);
  else aux_role<R, S, TF>(g, role - g.nch - NHEAD, dyn, sy, tg0);
}

// Clears the tagged histories and mailboxes and the status word before a run from zero.
__global__ void wn_chain_reset_kernel(u64* words, size_t n, int* status) {
  const size_t i0 = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (size_t i = i0; i < n; i += (size_t)gridDim.x * blockDim.x) words[i] = 0ull;
  if (i0 == 0) *status = 0;
}

template <int R>
constexpr int chain_nlc() { return R == 64 ? 7 : 16; }

template <int R, int S>
hipError_t launch_chain_rs(const WnChainArgs& g, bool teacher, hipStream_t stream) {
  constexpr int NLC = chain_nlc<R>();
  const size_t chain_lds =
      ((size_t)2 * R + NLC * 2 * R + NHEAD * A + 2 * UB + 2 * NLC * R + (size_t)A * R + (size_t)S * R) *
      sizeof(float);
  const size_t head_lds = ((size_t)g.d.L * S + S + HR) * sizeof(float);
  const size_t aux_lds = (size_t)4 * R * sizeof(float);
  const size_t dyn = std::max(chain_lds, std::max(head_lds, aux_lds));
  void* args[] = {const_cast<WnChainArgs*>(&g)};
  const void* k = teacher ? reinterpret_cast<const void*>(wn_chain_kernel<R, S, NLC, true>)
                          : reinterpret_cast<const void*>(wn_chain_kernel<R, S, NLC, false>);
  hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
  if (e != hipSuccess) return e;
  return hipLaunchCooperativeKernel(k, dim3(WN_CHAIN_GRID), dim3(NT), args, (unsigned)dyn, stream);
}

}  // namespace

int wn_chain_layers_per_cu(int R) { return R == 64 ? chain_nlc<64>() : (R == 32 ? chain_nlc<32>() : 0); }

bool wn_chain_supported(int R, int S, int L) {
  if (!((R == 64 && (S == 256 || S == 128)) || (R == 32 && S == 128))) return false;
  const int nlc = wn_chain_layers_per_cu(R);
  const int nch = (L + nlc - 1) / nlc;
  return L >= 1 && L <= WN_MAX_LAYERS && nch <= WN_MAX_CHAIN && nch + NHEAD + L <= WN_CHAIN_GRID;
}

int wn_chain_num_cus(int L, int R) {
  const int nlc = wn_chain_layers_per_cu(R);
  return (L + nlc - 1) / nlc + NHEAD + L;
}

size_t wn_chain_mailbox_words(int L, int R, int S) {
  const int nlc = wn_chain_layers_per_cu(R);
  const int nch = (L + nlc - 1) / nlc;
  return (size_t)L * 2 * 2 * R + (size_t)L * 2 * R + (size_t)L * 2 * S + (size_t)nch * 2 * R + (size_t)NHEAD * 2 * A +
         (size_t)2 * S;
}

hipError_t wn_chain_reset(unsigned long long* words, size_t n, int* status, hipStream_t stream) {
  hipLaunchKernelGGL(wn_chain_reset_kernel, dim3(256), dim3(256), 0, stream, words, n, status);
  return hipGetLastError();
}

hipError_t wn_chain_launch(const WnChainArgs& g, bool teacher, hipStream_t stream) {
  const int R = g.d.R, S = g.d.S;
  if (R == 64 && S == 256) return launch_chain_rs<64, 256>(g, teacher, stream);
  if (R == 64 && S == 128) return launch_chain_rs<64, 128>(g, teacher, stream);
  if (R == 32 && S == 128) return launch_chain_rs<32, 128>(g, teacher, stream);
  return hipErrorInvalidValue;
}
