// Persistent per-stream generation kernel for gfx950.
//
// One 1024-thread workgroup (16 wave64s) owns one stream for the whole call and
// loops over its T steps.  Each step evaluates the autoregressive WaveNet of
// Deep Voice (arXiv 1702.07825), Appendix A.1, in the order of the paper's
// CPU-inference section (Section 5.1): sample embedding, then per layer the two
// halves of the width-2 dilated convolution (W_prev on the history slot, W_cur
// on the current input), the gated activation, the residual and skip 1x1
// projections, then the relu head, the softmax and the draw.
//
// Data placement:
//  - weights stay in HBM and are re-read every step through the L2 (each row is
//    read by LPR adjacent lanes, 4 weights per load (16 int8 codes), so a wave
//    instruction covers contiguous row segments); fp32, bf16 or int8 codes with a
//    per-row scale that multiplies the row's dot product;
//  - activations (x, h, q, z_a, logits) and the step's conditioning and history
//    reads live in LDS;
//  - each layer's dilation history is a ring of d_j slots of r floats in the
//    workspace: slot (tg mod d_j) holds x_{j-1}[tg - d_j] when step tg starts and
//    receives x_{j-1}[tg] during it.
// Matrix-vector products reduce across the LPR lanes of a row with cross-lane
// shuffles.  The draw is a single-wave max / exp / inclusive scan / count.
#include "wn_internal.h"
#include "wn_wave.h"

#include "wn.h"

namespace {

constexpr int NT = 1024;
constexpr int A = WN_A;

__device__ __forceinline__ float ex2(float v) { return __builtin_amdgcn_exp2f(v); }
__device__ __forceinline__ float rcp(float v) { return __builtin_amdgcn_rcpf(v); }
__device__ __forceinline__ float expf_fast(float v) { return ex2(v * 1.4426950408889634f); }
// tanh(v) = 1 - 2 / (1 + e^{2v}); saturates correctly at both ends.
__device__ __forceinline__ float tanh_f(float v) { return 1.0f - 2.0f * rcp(1.0f + expf_fast(2.0f * v)); }
__device__ __forceinline__ float sigmoid_f(float v) { return rcp(1.0f + expf_fast(-v)); }

__device__ __forceinline__ float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 ld4(const uint16_t* p) {
  const uint2 v = *reinterpret_cast<const uint2*>(p);
  return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                     __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u));
}
// Scale of row `row` of a matrix stored as WT: the int8 codes' per-row scale, else 1.
template <typename WT>
__device__ __forceinline__ float row_scale(const float* s, size_t row) {
  if constexpr (sizeof(WT) == 1) return s[row];
  else return 1.0f;
}
__device__ __forceinline__ float dot4(float4 w, float4 x, float acc) {
  acc = fmaf(w.x, x.x, acc);
  acc = fmaf(w.y, x.y, acc);
  acc = fmaf(w.z, x.z, acc);
  return fmaf(w.w, x.w, acc);
}

// Unpacks 16 int8 codes (one 16-byte load) and adds their dot product with 16 inputs to acc.
__device__ __forceinline__ float dot16_i8(const int8_t* p, const float4* x, float acc) {
  const int4 v = *reinterpret_cast<const int4*>(p);
  const int w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    acc = fmaf((float)((w[q] << 24) >> 24), x[q].x, acc);
    acc = fmaf((float)((w[q] << 16) >> 24), x[q].y, acc);
    acc = fmaf((float)((w[q] << 8) >> 24), x[q].z, acc);
    acc = fmaf((float)(w[q] >> 24), x[q].w, acc);
  }
  return acc;
}

// Inputs one lane takes from a row per load: 4 fp32 or bf16 weights, or 16 int8 codes.
template <typename WT>
constexpr int kChunk = sizeof(WT) == 1 ? 16 : 4;

// Dot products of K-long rows stored as WT: LPR adjacent lanes share a row, each handling NV
// chunks of CH inputs (chunk index lane + i*LPR), then reduce across the LPR lanes.
template <int K, typename WT>
struct RowDot {
  static constexpr int CH = kChunk<WT>;
  static constexpr int LPR = (K / CH < 16) ? K / CH : 16;
  static constexpr int NV = K / CH / LPR;
  static constexpr int NX = NV * CH / 4;  // float4s of the input a lane holds
  static constexpr int G = NT / LPR;      // rows per pass over the workgroup
  __device__ static float partial(const WT* row, const float4 (&x4)[NX], int li) {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      if constexpr (CH == 16) s = dot16_i8(row + CH * (li + i * LPR), x4 + 4 * i, s);
      else s = dot4(ld4(row + CH * (li + i * LPR)), x4[i], s);
    }
    return s;
  }
  __device__ static void load_x(const float* x, float4 (&x4)[NX], int li) {
#pragma unroll
    for (int i = 0; i < NV; ++i)
#pragma unroll
      for (int q = 0; q < CH / 4; ++q) x4[i * (CH / 4) + q] = reinterpret_cast<const float4*>(x)[(li + i * LPR) * (CH / 4) + q];
  }
  __device__ static float reduce(float v) {
#pragma unroll
    for (int o = LPR / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
  }
};

template <int R, int S, typename WT, bool TF>
__global__ __launch_bounds__(NT) void wn_stream_kernel(const WnStreamArgs args) {
  const WnDims& D = args.d;
  const int L = D.L;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int T = args.io.T;

  extern __shared__ float dyn[];
  float* xr = dyn;              // [L][R] history reads of this step
  float* cs = dyn + L * R;      // [L][2R] conditioning of this step
  __shared__ float xs[R];       // x_{j-1}, updated in place to x_j
  __shared__ float hs[R];
  __shared__ float qs[S];
  __shared__ float zas[A];
  __shared__ __align__(16) float lgs[A];
  __shared__ int yprev_s;   // y_{t-1}
  __shared__ int yprev2_s;  // y_{t-2}, -1 before the first input
  __shared__ int abort_s;   // 1 once this block has seen an abort request

  const WT* embed = static_cast<const WT*>(args.w.embed);
  const WT* embed_prev = static_cast<const WT*>(args.w.embed_prev);  // null with one tap
  const WT* w_prev = static_cast<const WT*>(args.w.w_prev);
  const WT* w_cur = static_cast<const WT*>(args.w.w_cur);
  const WT* w_res = static_cast<const WT*>(args.w.w_res);
  const WT* w_skip = static_cast<const WT*>(args.w.w_skip);
  const WT* w_relu = static_cast<const WT*>(args.w.w_relu);
  const WT* w_out = static_cast<const WT*>(args.w.w_out);

  float* hist = args.ws.hist + (size_t)b * D.hist_len;
  int64_t* state = args.ws.state + WN_STATE_WORDS * (size_t)b;

  int64_t tg0;
  if (args.io.reset) {
    for (int i = tid; i < D.hist_len / 4; i += NT) reinterpret_cast<float4*>(hist)[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    tg0 = 0;
    if (tid == 0) {
      yprev_s = args.io.init_sample;
      yprev2_s = -1;
    }
  } else {
    tg0 = state[0];
    if (tid == 0) {
      yprev_s = (int)state[1];
      yprev2_s = (int)state[2];
    }
  }
  if (tid == 0) abort_s = 0;
  __syncthreads();

  for (int t = 0; t < T; ++t) {
    const int64_t tg = tg0 + t;
    const size_t bt = (size_t)b * T + t;
    // a host abort request, read every WN_ABORT_CHECK steps; the decision is taken block-wide after
    // the barrier below
    if (tid == 0 && (t & (WN_ABORT_CHECK - 1)) == 0 && wnk::abort_requested(args.io.abort_flag)) {
      atomicCAS(args.ws.status, 0, (int)WN_EABORTED);
      abort_s = 1;
    }
    // ---- step inputs: history slots, conditioning, embedding, q = B_skip ----
    {
      const float* cond_t = args.io.cond + bt * (size_t)(L * 2 * R);
      for (int i = tid; i < L * 2 * R / 4; i += NT)
        reinterpret_cast<float4*>(cs)[i] = reinterpret_cast<const float4*>(cond_t)[i];
      for (int i = tid; i < L * R / 4; i += NT) {
        const int j = i / (R / 4), c4 = i % (R / 4);
        const int slot = (int)(tg % D.dil[j]);
        reinterpret_cast<float4*>(xr)[i] = reinterpret_cast<const float4*>(hist + D.hoff[j] + slot * R)[c4];
      }
      const int yp = yprev_s, yp2 = yprev2_s;
      if (tid < R) {
        auto ld = [&](const WT* e) {
          if constexpr (sizeof(WT) == 2) return __uint_as_float((uint32_t)e[tid] << 16);
          else return (float)e[tid];
        };
        float ev = ld(embed + (size_t)yp * R) * row_scale<WT>(args.w.s_embed, yp) + args.w.b_embed[tid];
        if (embed_prev && yp2 >= 0) ev += ld(embed_prev + (size_t)yp2 * R) * row_scale<WT>(args.w.s_embed_prev, yp2);
        xs[tid] = ev;
      }
      for (int m = tid; m < S; m += NT) qs[m] = args.w.b_skip[m];
    }
    __syncthreads();
    if (abort_s) break;

    for (int j = 0; j < L; ++j) {
      // ---- a = W_prev x[t-d] + W_cur x[t] + B + L ; h = tanh(a[:R]) * sigmoid(a[R:]) ----
      {
        using RD = RowDot<R, WT>;
        const int li = tid % RD::LPR, grp = tid / RD::LPR;
        float4 xp4[RD::NX], xc4[RD::NX];
        RD::load_x(xr + j * R, xp4, li);
        RD::load_x(xs, xc4, li);
        const WT* wp = w_prev + (size_t)j * 2 * R * R;
        const WT* wc = w_cur + (size_t)j * 2 * R * R;
        constexpr int P = (R + RD::G - 1) / RD::G;
#pragma unroll
        for (int p = 0; p < P; ++p) {
          const int c = p * RD::G + grp;
          if (c < R) {
            const size_t r0 = (size_t)j * 2 * R + c, r1 = r0 + R;  // rows c (tanh) and c + R (sigmoid)
            float s0 = RD::partial(wp + (size_t)c * R, xp4, li) * row_scale<WT>(args.w.s_prev, r0) +
                       RD::partial(wc + (size_t)c * R, xc4, li) * row_scale<WT>(args.w.s_cur, r0);
            float s1 = RD::partial(wp + (size_t)(c + R) * R, xp4, li) * row_scale<WT>(args.w.s_prev, r1) +
                       RD::partial(wc + (size_t)(c + R) * R, xc4, li) * row_scale<WT>(args.w.s_cur, r1);
            s0 = RD::reduce(s0);
            s1 = RD::reduce(s1);
            if (li == 0) {
              const float* bg = args.w.b_gate + j * 2 * R;
              const float a0 = s0 + bg[c] + cs[j * 2 * R + c];
              const float a1 = s1 + bg[c + R] + cs[j * 2 * R + c + R];
              hs[c] = args.w.approx_nl ? wnk::tanh_paper(a0) * wnk::sigmoid_paper(a1) : tanh_f(a0) * sigmoid_f(a1);
            }
          }
        }
        // x_{j-1}[tg] goes into the slot whose old value (x_{j-1}[tg - d]) was read above
        if (tid < R) hist[D.hoff[j] + (int)(tg % D.dil[j]) * R + tid] = xs[tid];
      }
      __syncthreads();
      // ---- x += W_res h + B_res (rows 0..R-1) ; q += W_skip h (rows R..R+S-1) ----
      {
        using RD = RowDot<R, WT>;
        const int li = tid % RD::LPR, grp = tid / RD::LPR;
        float4 h4[RD::NX];
        RD::load_x(hs, h4, li);
        const bool last = (j == L - 1);  // x_L feeds nothing
        const WT* wr = w_res + (size_t)j * R * R;
        const WT* wk = w_skip + (size_t)j * S * R;
        constexpr int P = (R + S + RD::G - 1) / RD::G;
#pragma unroll
        for (int p = 0; p < P; ++p) {
          const int row = p * RD::G + grp;
          if (row < R) {
            if (!last) {
              const float v = RD::reduce(RD::partial(wr + (size_t)row * R, h4, li)) *
                              row_scale<WT>(args.w.s_res, (size_t)j * R + row);
              if (li == 0) xs[row] += v + args.w.b_res[j * R + row];
            }
          } else if (row < R + S) {
            const int m = row - R;
            const float v = RD::reduce(RD::partial(wk + (size_t)m * R, h4, li)) *
                            row_scale<WT>(args.w.s_skip, (size_t)j * S + m);
            if (li == 0) qs[m] += v;
          }
        }
      }
      __syncthreads();
    }

    // ---- z_a = relu(W_relu relu(q) + B_relu) ----
    {
      using RD = RowDot<S, WT>;
      const int li = tid % RD::LPR, grp = tid / RD::LPR;
      float4 z4[RD::NX];
      RD::load_x(qs, z4, li);
#pragma unroll
      for (int i = 0; i < RD::NX; ++i) {
        z4[i].x = fmaxf(z4[i].x, 0.f); z4[i].y = fmaxf(z4[i].y, 0.f);
        z4[i].z = fmaxf(z4[i].z, 0.f); z4[i].w = fmaxf(z4[i].w, 0.f);
      }
      constexpr int P = (A + RD::G - 1) / RD::G;  // int8 rows of s = 32 take 2 lanes: one pass covers 512 rows
#pragma unroll
      for (int p = 0; p < P; ++p) {
        const int i = p * RD::G + grp;
        if (i >= A) break;  // uniform over the lanes of a row
        const float v = RD::reduce(RD::partial(w_relu + (size_t)i * S, z4, li)) * row_scale<WT>(args.w.s_relu, i);
        if (li == 0) zas[i] = fmaxf(v + args.w.b_relu[i], 0.f);
      }
    }
    __syncthreads();
    // ---- logits = W_out z_a + B_out ----
    {
      using RD = RowDot<A, WT>;
      const int li = tid % RD::LPR, grp = tid / RD::LPR;
      float4 z4[RD::NX];
      RD::load_x(zas, z4, li);
      constexpr int P = A / RD::G;
#pragma unroll
      for (int p = 0; p < P; ++p) {
        const int i = p * RD::G + grp;
        const float v = RD::reduce(RD::partial(w_out + (size_t)i * A, z4, li)) * row_scale<WT>(args.w.s_out, i);
        if (li == 0) {
          const float lg = v + args.w.b_out[i];
          if constexpr (TF) args.io.logits[bt * A + i] = lg;
          else lgs[i] = lg;
        }
      }
    }
    if constexpr (TF) {
      if (tid == 0) {
        int y = args.io.y_in[bt];
        yprev2_s = yprev_s;
        yprev_s = y < 0 ? 0 : (y > A - 1 ? A - 1 : y);
      }
    } else {
      __syncthreads();
      // ---- the draw from p = softmax(logits) (one wave) ----
      if (tid < 64) {
        const int lane = tid;
        const float4 lv = *reinterpret_cast<const float4*>(lgs + 4 * lane);
        const int y = args.w.approx_nl
                          ? wnk::wave_draw<true>(lv, args.io.u[bt], args.io.smode, args.io.inv_t, args.io.top_k, lane)
                          : wnk::wave_draw<false>(lv, args.io.u[bt], args.io.smode, args.io.inv_t, args.io.top_k, lane);
        if (lane == 0) {
          args.io.y_out[bt] = y;
          yprev2_s = yprev_s;
          yprev_s = y;
        }
      }
    }
    __syncthreads();
  }
  // after an abort the state stays as it was (the next call must start from zero)
  if (tid == 0 && !abort_s) {
    state[0] = tg0 + T;
    state[1] = yprev_s;
    state[2] = yprev2_s;
  }
}

template <int R, int S>
hipError_t launch_rs(const WnStreamArgs& args, bool teacher, hipStream_t stream) {
  const size_t dyn = (size_t)args.d.L * 3 * R * sizeof(float);
  const dim3 grid(args.io.B), block(NT);
  hipError_t e;
#define WN_LAUNCH(WT, TF)                                                                            \
  do {                                                                                               \
    auto k = wn_stream_kernel<R, S, WT, TF>;                                                         \
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn); \
    if (e != hipSuccess) return e;                                                                   \
    hipLaunchKernelGGL(k, grid, block, dyn, stream, args);                                           \
  } while (0)
  if (args.w.bf16) {
    if (teacher) WN_LAUNCH(uint16_t, true); else WN_LAUNCH(uint16_t, false);
  } else if (args.w.i8) {
    if (teacher) WN_LAUNCH(int8_t, true); else WN_LAUNCH(int8_t, false);
  } else {
    if (teacher) WN_LAUNCH(float, true); else WN_LAUNCH(float, false);
  }
#undef WN_LAUNCH
  return hipGetLastError();
}

}  // namespace

bool wn_stream_supported(int R, int S) {
  return (R == 16 && S == 32) || (R == 32 && S == 128) || (R == 64 && S == 128) || (R == 64 && S == 256) ||
         (R == 128 && S == 256);
}

hipError_t wn_stream_launch(const WnStreamArgs& args, bool teacher, hipStream_t stream) {
  const int R = args.d.R, S = args.d.S;
  if (R == 16 && S == 32) return launch_rs<16, 32>(args, teacher, stream);
  if (R == 32 && S == 128) return launch_rs<32, 128>(args, teacher, stream);
  if (R == 64 && S == 128) return launch_rs<64, 128>(args, teacher, stream);
  if (R == 64 && S == 256) return launch_rs<64, 256>(args, teacher, stream);
  if (R == 128 && S == 256) return launch_rs<128, 256>(args, teacher, stream);
  return hipErrorInvalidValue;
}
