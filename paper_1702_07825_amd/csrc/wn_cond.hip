// Conditioning network on gfx950 (Deep Voice, arXiv 1702.07825, Appendix A.2): two
// bidirectional fo-pooling QRNN layers with width-2 convolutions, the two directions' channels
// interleaved, and upsampling to the audio rate by repetition.  Declarations and contracts are
// in include/wn_cond.h.
//
// Each layer is two kernels.  The gate pre-activations of all frames at once are a dense
// contraction, [B*Tf x 2 cin] . [2 cin x 3h] per direction (the width-2 convolution: inputs
// 0..cin-1 are the direction's previous frame, cin..2cin-1 the current one), run on fp32 MFMA
// (v_mfma_f32_16x16x4_f32) in 64 x 64 tiles staged through LDS.  The fo-pool is a linear
// recurrence along the frames, independent per (stream, direction, channel): one thread each,
// with the gate pre-activations of 16 frames loaded ahead of the dependent chain.  The second
// layer's pool writes its output interleaved, and a last kernel repeats every frame over its
// audio steps with coalesced float4 stores (bound by the HBM write of [B][T][2 h2]).
#include "wn_cond.h"
#include "wn.h"
#include "wn_internal.h"
#include "wn_wave.h"

#include <algorithm>
#include <cstring>
#include <vector>

struct wn_cond {
  int device = 0;
  int F = 0, h1 = 0, h2 = 0, fr = 1, ar = 1;
  void* dmem = nullptr;
  const float *w1 = nullptr, *b1 = nullptr, *w2 = nullptr, *b2 = nullptr;
};

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int TM = 64, TN = 64, TK = 16;  // output tile (frames x gate rows) and K chunk
constexpr int NTG = 256;                  // four waves, each a 32 x 32 sub-tile

struct GateArgs {
  const float* x;  // [B][Tf][cin]
  const float* w;  // [2][N][2 cin]
  const float* b;  // [2][N]
  float* p;        // [B][Tf][2][N]
  int B, Tf, cin, N;
};

// Gate pre-activations p[b][t][dir][n] = b[dir][n] + sum_k w[dir][n][k] x2[b][t][k], where
// x2[b][t] = [x[b][t'], x[b][t]] with t' = t - 1 (forward) or t + 1 (backward), zero outside.
__global__ __launch_bounds__(NTG) void qrnn_gate_gemm(const GateArgs a) {
  const int dir = blockIdx.z;
  const int m0 = blockIdx.x * TM, n0 = blockIdx.y * TN;
  const int M = a.B * a.Tf, K = 2 * a.cin;
  __shared__ float As[TM][TK + 1];
  __shared__ float Bs[TN][TK + 1];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = (wave >> 1) * 32, wn = (wave & 1) * 32;
  const int row = lane & 15, kq = lane >> 4;  // MFMA operand: row / column of the 16, k of the 4
  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const float* wd = a.w + (size_t)dir * a.N * K;
  for (int k0 = 0; k0 < K; k0 += TK) {
    for (int i = tid; i < TM * TK; i += NTG) {
      const int r = i / TK, kk = i % TK;
      const int m = m0 + r, k = k0 + kk;
      float v = 0.f;
      if (m < M && k < K) {
        const int bb = m / a.Tf, t = m % a.Tf;
        const bool prev = k < a.cin;
        const int tt = prev ? (dir == 0 ? t - 1 : t + 1) : t;
        if (tt >= 0 && tt < a.Tf) v = a.x[((size_t)bb * a.Tf + tt) * a.cin + (prev ? k : k - a.cin)];
      }
      As[r][kk] = v;
    }
    for (int i = tid; i < TN * TK; i += NTG) {
      const int r = i / TK, kk = i % TK;
      const int n = n0 + r, k = k0 + kk;
      Bs[r][kk] = (n < a.N && k < K) ? wd[(size_t)n * K + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < TK; ks += 4) {
      float av[2], bv[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) av[i] = As[wm + i * 16 + row][ks + kq];
#pragma unroll
      for (int j = 0; j < 2; ++j) bv[j] = Bs[wn + j * 16 + row][ks + kq];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
  // result (i, j): lane holds rows 4 kq .. 4 kq + 3 of column `row`
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int n = n0 + wn + j * 16 + row;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = m0 + wm + i * 16 + 4 * kq + v;
        if (m < M && n < a.N) a.p[((size_t)m * 2 + dir) * a.N + n] = acc[i][j][v] + a.b[(size_t)dir * a.N + n];
      }
    }
}

struct PoolArgs {
  const float* p;  // [B][Tf][2][3H]: blocks h~, o, f
  float* out;      // [B][Tf][2H]: stacked (forward then backward) or interleaved (2k + dir)
  int B, Tf, H, interleave;
};

// fo-pool h_t = f_t h_{t-1} + (1 - f_t) tanh(a_h), z_t = sigmoid(a_o) h_t, over the frames in the
// direction's own order; one thread per (stream, direction, channel).
__global__ __launch_bounds__(256) void qrnn_pool(const PoolArgs a) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  const int b = blockIdx.y >> 1, dir = blockIdx.y & 1;
  if (k >= a.H) return;
  const size_t fstride = (size_t)6 * a.H;  // floats per frame of p
  const float* base = a.p + (size_t)b * a.Tf * fstride + (size_t)dir * 3 * a.H + k;
  float* ob = a.out + (size_t)b * a.Tf * 2 * a.H + (a.interleave ? 2 * k + dir : dir * a.H + k);
  constexpr int U = 16;
  float h = 0.f;
  for (int s0 = 0; s0 < a.Tf; s0 += U) {
    float ah[U], ao[U], af[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = s0 + u;
      if (s < a.Tf) {
        const int t = dir ? a.Tf - 1 - s : s;
        const float* q = base + (size_t)t * fstride;
        ah[u] = q[0];
        ao[u] = q[a.H];
        af[u] = q[2 * a.H];
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = s0 + u;
      if (s < a.Tf) {
        const int t = dir ? a.Tf - 1 - s : s;
        const float f = wnk::sigmoid_f(af[u]);
        h = f * h + (1.f - f) * wnk::tanh_f(ah[u]);
        ob[(size_t)t * 2 * a.H] = wnk::sigmoid_f(ao[u]) * h;
      }
    }
  }
}

// cond[b][tau][c] = src[b][floor(tau * fr / ar)][c] for c < C (C % 4 == 0: float4 copies).
__global__ __launch_bounds__(256) void cond_upsample4(const float4* src, float4* cond, int Tf, long long T, int C4,
                                                      long long n4, int fr, int ar) {
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (long long)gridDim.x * blockDim.x) {
    const long long row = i / C4, c = i - row * C4;
    const long long b = row / T, tau = row - b * T;
    const long long t = tau * fr / ar;
    cond[i] = src[((size_t)b * Tf + t) * C4 + c];
  }
}
__global__ __launch_bounds__(256) void cond_upsample1(const float* src, float* cond, int Tf, long long T, int C,
                                                      long long n, int fr, int ar) {
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x) {
    const long long row = i / C, c = i - row * C;
    const long long b = row / T, tau = row - b * T;
    const long long t = tau * fr / ar;
    cond[i] = src[((size_t)b * Tf + t) * C + c];
  }
}

size_t align_up(size_t v, size_t al) { return (v + al - 1) / al * al; }

struct CondLayout {
  size_t p_off, z1_off, c_off, total;
};
CondLayout cond_layout(const wn_cond* c, int B, int Tf) {
  CondLayout l;
  const size_t frames = (size_t)B * Tf;
  l.p_off = 0;
  l.z1_off = align_up(l.p_off + frames * 6 * (size_t)std::max(c->h1, c->h2) * 4, 256);
  l.c_off = align_up(l.z1_off + frames * 2 * (size_t)c->h1 * 4, 256);
  l.total = align_up(l.c_off + frames * 2 * (size_t)c->h2 * 4, 256);
  return l;
}

class DeviceScope {
 public:
  explicit DeviceScope(int dev) {
    ok_ = hipGetDevice(&prev_) == hipSuccess;
    if (ok_ && prev_ != dev) ok_ = hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceScope() {
    int cur = -1;
    if (hipGetDevice(&cur) == hipSuccess && cur != prev_) (void)hipSetDevice(prev_);
  }
  bool ok() const { return ok_; }

 private:
  int prev_ = 0;
  bool ok_ = false;
};

hipError_t run_layer(const float* x, int B, int Tf, int cin, int H, const float* w, const float* b, float* p,
                     float* out, int interleave, hipStream_t st) {
  GateArgs g{x, w, b, p, B, Tf, cin, 3 * H};
  const dim3 grid((unsigned)((B * Tf + TM - 1) / TM), (unsigned)((3 * H + TN - 1) / TN), 2);
  hipLaunchKernelGGL(qrnn_gate_gemm, grid, dim3(NTG), 0, st, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  PoolArgs pa{p, out, B, Tf, H, interleave};
  hipLaunchKernelGGL(qrnn_pool, dim3((unsigned)((H + 255) / 256), (unsigned)(2 * B)), dim3(256), 0, st, pa);
  return hipGetLastError();
}

}  // namespace

extern "C" {

int wn_cond_create(const wn_cond_config* cfg, const wn_cond_weights* w, wn_cond** out) {
  wn_clear_last_error();
  if (!cfg || !w || !out || !w->w1 || !w->b1 || !w->w2 || !w->b2) return wn_set_last_error(WN_EINVAL, "null argument");
  if (cfg->n_features < 1 || cfg->n_features > 4096) return wn_set_last_error(WN_EINVAL, "n_features must be 1..4096");
  if (cfg->h1 < 1 || cfg->h1 > 4096) return wn_set_last_error(WN_EINVAL, "h1 must be 1..4096");
  if (cfg->n_layers < 1 || cfg->r < 1 || (long long)cfg->n_layers * cfg->r > 8192)
    return wn_set_last_error(WN_EINVAL, "n_layers * r must be 1..8192");
  if (cfg->frame_rate < 1 || cfg->audio_rate < 1) return wn_set_last_error(WN_EINVAL, "rates must be >= 1");
  wn_cond* c = new (std::nothrow) wn_cond();
  if (!c) return wn_set_last_error(WN_ENOMEM, "host allocation");
  c->F = cfg->n_features;
  c->h1 = cfg->h1;
  c->h2 = cfg->n_layers * cfg->r;
  c->fr = cfg->frame_rate;
  c->ar = cfg->audio_rate;
  if (hipGetDevice(&c->device) != hipSuccess) {
    delete c;
    return wn_set_last_error(WN_EHIP, "hipGetDevice failed");
  }
  const size_t n_w1 = (size_t)2 * 3 * c->h1 * 2 * c->F, n_b1 = (size_t)2 * 3 * c->h1;
  const size_t n_w2 = (size_t)2 * 3 * c->h2 * 2 * 2 * c->h1, n_b2 = (size_t)2 * 3 * c->h2;
  const size_t o_b1 = align_up(n_w1 * 4, 256), o_w2 = align_up(o_b1 + n_b1 * 4, 256);
  const size_t o_b2 = align_up(o_w2 + n_w2 * 4, 256), total = align_up(o_b2 + n_b2 * 4, 256);
  hipError_t e = hipMalloc(&c->dmem, total);
  if (e != hipSuccess) {
    delete c;
    return e == hipErrorOutOfMemory ? wn_set_last_error(WN_ENOMEM, "hipMalloc of weights")
                                    : wn_set_last_error(WN_EHIP, hipGetErrorString(e));
  }
  char* d = static_cast<char*>(c->dmem);
  const struct { const float* src; size_t n, off; } parts[] = {
      {w->w1, n_w1, 0}, {w->b1, n_b1, o_b1}, {w->w2, n_w2, o_w2}, {w->b2, n_b2, o_b2}};
  for (const auto& pt : parts) {
    if (e == hipSuccess) e = hipMemcpy(d + pt.off, pt.src, pt.n * 4, hipMemcpyHostToDevice);
  }
  if (e != hipSuccess) {
    (void)hipFree(c->dmem);
    delete c;
    return wn_set_last_error(WN_EHIP, hipGetErrorString(e));
  }
  c->w1 = reinterpret_cast<const float*>(d);
  c->b1 = reinterpret_cast<const float*>(d + o_b1);
  c->w2 = reinterpret_cast<const float*>(d + o_w2);
  c->b2 = reinterpret_cast<const float*>(d + o_b2);
  *out = c;
  return WN_OK;
}

size_t wn_cond_workspace_bytes(const wn_cond* c, int32_t B, int32_t n_frames) {
  if (!c || B < 1 || n_frames < 1) return 0;
  return cond_layout(c, B, n_frames).total;
}

int wn_condition(wn_cond* c, int32_t B, int32_t n_frames, const float* features, int32_t T, float* cond,
                 void* workspace, size_t ws_bytes, void* stream) {
  wn_clear_last_error();
  if (!c) return wn_set_last_error(WN_EINVAL, "null handle");
  if (B < 1 || n_frames < 1 || T < 0) return wn_set_last_error(WN_EINVAL, "B and n_frames must be >= 1, T >= 0");
  if (T == 0) return WN_OK;
  if (!features || !cond || !workspace) return wn_set_last_error(WN_EINVAL, "null pointer");
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
    return wn_set_last_error(WN_EINVAL, "workspace must be 256-byte aligned");
  if ((long long)B * n_frames > (1LL << 31) - 1) return wn_set_last_error(WN_EINVAL, "B * n_frames too large");
  if ((long long)(T - 1) * c->fr / c->ar >= n_frames)
    return wn_set_last_error(WN_EINVAL, "audio steps beyond the last frame");
  const CondLayout l = cond_layout(c, B, n_frames);
  if (ws_bytes < l.total) return wn_set_last_error(WN_EINVAL, "workspace too small");
  DeviceScope scope(c->device);
  if (!scope.ok()) return wn_set_last_error(WN_EHIP, "cannot select the handle's device");
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  float* p = reinterpret_cast<float*>(ws + l.p_off);
  float* z1 = reinterpret_cast<float*>(ws + l.z1_off);
  float* cf = reinterpret_cast<float*>(ws + l.c_off);
  hipError_t e = run_layer(features, B, n_frames, c->F, c->h1, c->w1, c->b1, p, z1, 0, st);
  if (e == hipSuccess) e = run_layer(z1, B, n_frames, 2 * c->h1, c->h2, c->w2, c->b2, p, cf, 1, st);
  if (e == hipSuccess) {
    const int C = 2 * c->h2;
    const long long n = (long long)B * T * C;
    if (C % 4 == 0) {
      const long long n4 = n / 4;
      const unsigned blocks = (unsigned)std::min<long long>((n4 + 255) / 256, 65536);
      hipLaunchKernelGGL(cond_upsample4, dim3(blocks), dim3(256), 0, st, reinterpret_cast<const float4*>(cf),
                         reinterpret_cast<float4*>(cond), n_frames, (long long)T, C / 4, n4, c->fr, c->ar);
    } else {
      const unsigned blocks = (unsigned)std::min<long long>((n + 255) / 256, 65536);
      hipLaunchKernelGGL(cond_upsample1, dim3(blocks), dim3(256), 0, st, cf, cond, n_frames, (long long)T, C, n,
                         c->fr, c->ar);
    }
    e = hipGetLastError();
  }
  if (e != hipSuccess) return wn_set_last_error(WN_EHIP, hipGetErrorString(e));
  return WN_OK;
}

void wn_cond_destroy(wn_cond* c) {
  if (!c) return;
  {
    DeviceScope scope(c->device);
    if (c->dmem) (void)hipFree(c->dmem);
  }
  delete c;
}

}  // extern "C"
