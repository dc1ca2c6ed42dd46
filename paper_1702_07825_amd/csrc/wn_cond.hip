// Conditioning network on gfx950 (Deep Voice, arXiv 1702.07825, Appendix A.2): two
// bidirectional fo-pooling QRNN layers with width-2 convolutions, the two directions' channels
// interleaved, and upsampling to the audio rate by repetition.  Declarations and contracts are
// in include/wn_cond.h.
//
// Each layer is two kernels.  The gate pre-activations of all frames at once are a dense
// contraction, [3h x 2 cin] . [2 cin x B*Tf] per direction (the width-2 convolution: tap 0 is the
// direction's previous frame, tap 1 the current one), run on fp32 MFMA (v_mfma_f32_16x16x4f32) in
// 128 x 128 tiles staged through double-buffered LDS; the weights are stored with each tap padded
// to a multiple of 32 inputs so that K chunks never straddle the taps.  The fo-pool is a linear
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
#include <mutex>
#include <vector>

struct wn_cond {
  int device = 0;
  int F = 0, h1 = 0, h2 = 0, fr = 1, ar = 1;
  int cinp1 = 0, cinp2 = 0;  // per-tap input widths of the two layers rounded up to 32
  void* dmem = nullptr;
  const float *w1 = nullptr, *b1 = nullptr, *w2 = nullptr, *b2 = nullptr;
  void* scratch = nullptr;  // device address of this device's copy of `scratch` (wn_condition_static)
};

// Scratch of wn_condition_static: one copy per device, held until the process ends.  Host code
// never uses the array's name as an address (on the host it is only a stand-in for the symbol);
// wn_cond_create looks up each device's address of it once, with that device current.
static __device__ __align__(256) unsigned char scratch[WN_COND_SCRATCH_BYTES];

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

struct GateArgs {
  const float* x;  // [B][Tf][cin]
  const float* w;  // [2][N][2 cinp]: tap 0 (previous frame) inputs 0..cin-1, tap 1 at cinp.., zeros past cin
  const float* b;  // [2][N]
  float* p;        // [B][Tf][2][N]
  int B, Tf, cin, cinp, N;
};

// Gate pre-activations of every frame of a layer, both directions (grid.z):
//   p[b][t][dir][n] = b[dir][n] + sum_k w[dir][n][0][k] x[b][t'][k] + w[dir][n][1][k] x[b][t][k]
// with t' = t - 1 (forward) or t + 1 (backward) and x = 0 outside the frames: the width-2
// convolution as one dense contraction [N x 2 cinp] . [2 cinp x B Tf] on fp32 MFMA
// (v_mfma_f32_16x16x4f32).  128 x 128 output tiles (gate rows x frames) per 256 threads, each wave
// a 64 x 64 quarter; K in chunks of 32 that never straddle the two taps (cinp is a multiple of
// 32).  LDS is double-buffered, one barrier per chunk, with the next chunk's global loads in
// flight during the current chunk's products.  The MFMA A operand is the weight rows and B the
// frames, so each lane ends with four consecutive gate rows of one frame.  Within a chunk the k
// index is permuted (lane group q of MFMA step e takes k = 4q + e of each 16), identically for
// both operands, so one b128 LDS read feeds four MFMA steps.  VX: the input rows are float4
// aligned (cin % 4 == 0), else they are read one float at a time.
constexpr int NTG = 256;
constexpr int VM = 128, VN = 128, VK = 32, VLD = VK + 8;  // tile, K chunk, LDS row (floats)

template <bool VX>
__global__ __launch_bounds__(NTG, 2) void qrnn_gate_gemm(const GateArgs a) {
  const int dir = blockIdx.z;
  const int m0 = blockIdx.x * VM, n0 = blockIdx.y * VN;
  const int M = a.B * a.Tf, K = 2 * a.cinp, N = a.N;
  __shared__ __align__(16) float Ws[2][VN][VLD];
  __shared__ __align__(16) float Xs[2][VM][VLD];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wn = (wave >> 1) * 64, wm = (wave & 1) * 64;
  const int r16 = lane & 15, q = lane >> 4;
  // global -> LDS assignment: rows tid/8 + 32 i, float4 column tid % 8 of the chunk
  const int lr = tid >> 3, lc = (tid & 7) * 4;
  const float* wd = a.w + (size_t)dir * N * K;
  const float* xcur[4];
  const float* xprev[4];
  const float* wrow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + lr + 32 * i;
    xcur[i] = xprev[i] = nullptr;
    if (m < M) {
      const int bb = m / a.Tf, t = m - bb * a.Tf;
      const int tp = dir == 0 ? t - 1 : t + 1;
      xcur[i] = a.x + ((size_t)bb * a.Tf + t) * a.cin;
      if (tp >= 0 && tp < a.Tf) xprev[i] = a.x + ((size_t)bb * a.Tf + tp) * a.cin;
    }
    const int n = n0 + lr + 32 * i;
    wrow[i] = n < N ? wd + (size_t)n * K + lc : nullptr;
  }
  f32x4 gx[4], gw[4];
  auto load = [&](int k0) {
    const bool prev = k0 < a.cinp;
    const int kk = (prev ? k0 : k0 - a.cinp) + lc;  // input index of this thread's first float
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float* xp = prev ? xprev[i] : xcur[i];
      if (VX) {
        gx[i] = xp && kk < a.cin ? *reinterpret_cast<const f32x4*>(xp + kk) : f32x4{0.f, 0.f, 0.f, 0.f};
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) gx[i][e] = xp && kk + e < a.cin ? xp[kk + e] : 0.f;
      }
      gw[i] = wrow[i] ? *reinterpret_cast<const f32x4*>(wrow[i] + k0) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *reinterpret_cast<f32x4*>(&Xs[buf][lr + 32 * i][lc]) = gx[i];
      *reinterpret_cast<f32x4*>(&Ws[buf][lr + 32 * i][lc]) = gw[i];
    }
  };
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  load(0);
  stash(0);
  __syncthreads();
  const int nk = K / VK;
  for (int c = 0; c < nk; ++c) {
    const int buf = c & 1;
    if (c + 1 < nk) load((c + 1) * VK);
#pragma unroll
    for (int h = 0; h < VK; h += 16) {
      f32x4 wa[4], xb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) wa[i] = *reinterpret_cast<const f32x4*>(&Ws[buf][wn + 16 * i + r16][h + 4 * q]);
#pragma unroll
      for (int j = 0; j < 4; ++j) xb[j] = *reinterpret_cast<const f32x4*>(&Xs[buf][wm + 16 * j + r16][h + 4 * q]);
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[i][e], xb[j][e], acc[i][j], 0, 0, 0);
    }
    if (c + 1 < nk) stash(buf ^ 1);
    __syncthreads();
  }
  // acc[i][j]: lane holds gate rows wn + 16 i + 4 q .. +3 of frame wm + 16 j + r16
  const float* bd = a.b + (size_t)dir * N;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int n = n0 + wn + 16 * i + 4 * q;
    if (n >= N) continue;
    const bool whole = (N & 3) == 0;  // then n + 3 < N and the row offsets are float4 aligned
    f32x4 bias;
#pragma unroll
    for (int v = 0; v < 4; ++v) bias[v] = n + v < N ? bd[n + v] : 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + wm + 16 * j + r16;
      if (m >= M) continue;
      float* dst = a.p + ((size_t)m * 2 + dir) * N + n;
      const f32x4 v4 = acc[i][j] + bias;
      if (whole) {
        *reinterpret_cast<f32x4*>(dst) = v4;
      } else {
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (n + v < N) dst[v] = v4[v];
      }
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

// Upsampling by repetition: cond[b][tau][:] = src[b][floor(tau fr / ar)][:].  One block per source
// frame (b, t); the frame covers the audio steps ceil(t ar / fr) <= tau < ceil((t + 1) ar / fr)
// (clipped to T), so its row is read once and stored to each of them (plain stores: nontemporal
// ones measured 4% slower here).
__global__ __launch_bounds__(256) void cond_repeat4(const f32x4* src, f32x4* cond, int Tf, long long T, int C4,
                                                    int fr, int ar) {
  const long long b = blockIdx.x / Tf, t = blockIdx.x - b * Tf;
  const long long tau0 = (t * ar + fr - 1) / fr;
  const long long tau1 = std::min<long long>(T, ((t + 1) * ar + fr - 1) / fr);
  const f32x4* s = src + (size_t)blockIdx.x * C4;
  f32x4* o = cond + (size_t)b * T * C4;
  for (int c = threadIdx.x; c < C4; c += 256) {
    const f32x4 v = s[c];
    for (long long tau = tau0; tau < tau1; ++tau) o[tau * C4 + c] = v;
  }
}
__global__ __launch_bounds__(256) void cond_repeat1(const float* src, float* cond, int Tf, long long T, int C, int fr,
                                                    int ar) {
  const long long b = blockIdx.x / Tf, t = blockIdx.x - b * Tf;
  const long long tau0 = (t * ar + fr - 1) / fr;
  const long long tau1 = std::min<long long>(T, ((t + 1) * ar + fr - 1) / fr);
  const float* s = src + (size_t)blockIdx.x * C;
  float* o = cond + (size_t)b * T * C;
  for (int c = threadIdx.x; c < C; c += 256) {
    const float v = s[c];
    for (long long tau = tau0; tau < tau1; ++tau) o[tau * C + c] = v;
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

hipError_t run_layer(const float* x, int B, int Tf, int cin, int cinp, int H, const float* w, const float* b,
                     float* p, float* out, int interleave, hipStream_t st) {
  GateArgs g{x, w, b, p, B, Tf, cin, cinp, 3 * H};
  const dim3 grid((unsigned)((B * Tf + VM - 1) / VM), (unsigned)((3 * H + VN - 1) / VN), 2);
  if (cin % 4 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0)
    hipLaunchKernelGGL(qrnn_gate_gemm<true>, grid, dim3(NTG), 0, st, g);
  else
    hipLaunchKernelGGL(qrnn_gate_gemm<false>, grid, dim3(NTG), 0, st, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  PoolArgs pa{p, out, B, Tf, H, interleave};
  hipLaunchKernelGGL(qrnn_pool, dim3((unsigned)((H + 255) / 256), (unsigned)(2 * B)), dim3(256), 0, st, pa);
  return hipGetLastError();
}

// [2][n][2][cin] -> [2][n][2][cinp], zeros in inputs cin..cinp-1 of each tap.
std::vector<float> pad_taps(const float* w, int n, int cin, int cinp) {
  std::vector<float> out((size_t)2 * n * 2 * cinp, 0.f);
  for (size_t row = 0; row < (size_t)2 * n * 2; ++row)
    std::memcpy(out.data() + row * cinp, w + row * cin, (size_t)cin * sizeof(float));
  return out;
}

// Device address of `scratch` on device dev (the current device), looked up once per device.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};

int scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return wn_set_last_error(WN_EUNSUPPORTED, "device index beyond 63");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return wn_set_last_error(WN_EHIP, "hipGetSymbolAddress of the scratch array failed");
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return WN_OK;
}

// The three kernels of one call, with the scratch at ws (cond_layout(c, B, n_frames) bytes).
int run_condition(wn_cond* c, int B, int n_frames, const float* features, int T, float* cond, char* ws,
                  hipStream_t st) {
  const CondLayout l = cond_layout(c, B, n_frames);
  float* p = reinterpret_cast<float*>(ws + l.p_off);
  float* z1 = reinterpret_cast<float*>(ws + l.z1_off);
  float* cf = reinterpret_cast<float*>(ws + l.c_off);
  hipError_t e = run_layer(features, B, n_frames, c->F, c->cinp1, c->h1, c->w1, c->b1, p, z1, 0, st);
  if (e == hipSuccess) e = run_layer(z1, B, n_frames, 2 * c->h1, c->cinp2, c->h2, c->w2, c->b2, p, cf, 1, st);
  if (e == hipSuccess) {
    const int C = 2 * c->h2;
    const unsigned blocks = (unsigned)((long long)B * n_frames);
    if (C % 4 == 0 && reinterpret_cast<uintptr_t>(cond) % 16 == 0)
      hipLaunchKernelGGL(cond_repeat4, dim3(blocks), dim3(256), 0, st, reinterpret_cast<const f32x4*>(cf),
                         reinterpret_cast<f32x4*>(cond), n_frames, (long long)T, C / 4, c->fr, c->ar);
    else
      hipLaunchKernelGGL(cond_repeat1, dim3(blocks), dim3(256), 0, st, cf, cond, n_frames, (long long)T, C, c->fr,
                         c->ar);
    e = hipGetLastError();
  }
  if (e != hipSuccess) return wn_set_last_error(WN_EHIP, hipGetErrorString(e));
  return WN_OK;
}

// Checks shared by wn_condition and wn_condition_static (all but the workspace).
int check_condition(const wn_cond* c, int B, int n_frames, const float* features, int T, const float* cond) {
  if (!c) return wn_set_last_error(WN_EINVAL, "null handle");
  if (B < 1 || n_frames < 1 || T < 0) return wn_set_last_error(WN_EINVAL, "B and n_frames must be >= 1, T >= 0");
  if (T == 0) return WN_OK;
  if (!features || !cond) return wn_set_last_error(WN_EINVAL, "null pointer");
  if ((long long)B * n_frames > (1LL << 31) - 1) return wn_set_last_error(WN_EINVAL, "B * n_frames too large");
  if ((long long)(T - 1) * c->fr / c->ar >= n_frames)
    return wn_set_last_error(WN_EINVAL, "audio steps beyond the last frame");
  return WN_OK;
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
  {
    const int rc = scratch_address(c->device, &c->scratch);
    if (rc != WN_OK) {
      delete c;
      return rc;
    }
  }
  c->cinp1 = (c->F + 31) / 32 * 32;
  c->cinp2 = (2 * c->h1 + 31) / 32 * 32;
  std::vector<float> w1p, w2p;
  try {
    w1p = pad_taps(w->w1, 3 * c->h1, c->F, c->cinp1);
    w2p = pad_taps(w->w2, 3 * c->h2, 2 * c->h1, c->cinp2);
  } catch (const std::bad_alloc&) {
    delete c;
    return wn_set_last_error(WN_ENOMEM, "host allocation");
  }
  const size_t n_b1 = (size_t)2 * 3 * c->h1, n_b2 = (size_t)2 * 3 * c->h2;
  const size_t o_b1 = align_up(w1p.size() * 4, 256), o_w2 = align_up(o_b1 + n_b1 * 4, 256);
  const size_t o_b2 = align_up(o_w2 + w2p.size() * 4, 256), total = align_up(o_b2 + n_b2 * 4, 256);
  hipError_t e = hipMalloc(&c->dmem, total);
  if (e != hipSuccess) {
    delete c;
    return e == hipErrorOutOfMemory ? wn_set_last_error(WN_ENOMEM, "hipMalloc of weights")
                                    : wn_set_last_error(WN_EHIP, hipGetErrorString(e));
  }
  char* d = static_cast<char*>(c->dmem);
  const struct { const float* src; size_t n, off; } parts[] = {
      {w1p.data(), w1p.size(), 0}, {w->b1, n_b1, o_b1}, {w2p.data(), w2p.size(), o_w2}, {w->b2, n_b2, o_b2}};
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
  int rc = check_condition(c, B, n_frames, features, T, cond);
  if (rc != WN_OK || T == 0) return rc;
  if (!workspace) return wn_set_last_error(WN_EINVAL, "null pointer");
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
    return wn_set_last_error(WN_EINVAL, "workspace must be 256-byte aligned");
  if (ws_bytes < cond_layout(c, B, n_frames).total) return wn_set_last_error(WN_EINVAL, "workspace too small");
  DeviceScope scope(c->device);
  if (!scope.ok()) return wn_set_last_error(WN_EHIP, "cannot select the handle's device");
  return run_condition(c, B, n_frames, features, T, cond, static_cast<char*>(workspace),
                       static_cast<hipStream_t>(stream));
}

int wn_condition_static(wn_cond* c, int32_t B, int32_t n_frames, const float* features, int32_t T, float* cond,
                        void* stream) {
  wn_clear_last_error();
  int rc = check_condition(c, B, n_frames, features, T, cond);
  if (rc != WN_OK || T == 0) return rc;
  if (cond_layout(c, B, n_frames).total > WN_COND_SCRATCH_BYTES)
    return wn_set_last_error(WN_EINVAL, "B * n_frames needs more scratch than the static array holds "
                                        "(wn_cond_workspace_bytes > WN_COND_SCRATCH_BYTES)");
  DeviceScope scope(c->device);
  if (!scope.ok()) return wn_set_last_error(WN_EHIP, "cannot select the handle's device");
  return run_condition(c, B, n_frames, features, T, cond, static_cast<char*>(c->scratch),
                       static_cast<hipStream_t>(stream));
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
