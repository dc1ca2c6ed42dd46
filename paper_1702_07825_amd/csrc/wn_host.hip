// Host side of the libwn C ABI: argument checks, weight packing, workspace
// layout and kernel selection.  Declarations and contracts are in include/wn.h.
#include "wn.h"
#include "wn_internal.h"

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

enum WnVariant { WN_VARIANT_STREAM = 0, WN_VARIANT_CHAIN = 1, WN_VARIANT_GROUP = 2, WN_VARIANT_MCHAIN = 3 };

struct wn_handle {
  int device = 0;
  int L = 0, R = 0, S = 0, A = 0;
  int init_sample = 128;
  int dtype = WN_F32;
  std::vector<int> dil;
  void* dmem = nullptr;
  WnDims dims{};
  WnDevWeights w{};
  bool chain_ok = false;  // the multi-CU kernel can serve this model (fp32, supported shape)
  bool xcd_map = false;   // blocks of the multi-CU kernel's grid run on XCD (block mod 8)
  bool group_ok = false;  // the batched MFMA kernel serves every B
  bool mchain_ok = false; // the multi-CU MFMA kernel can serve this model (bf16 or int8, supported shape)
  // WN_KERNEL at wn_create: the one kernel family calls may use ("" = the default choice); a call the
  // family cannot serve runs on the per-stream kernel
  std::string force;
  void* dpack = nullptr;  // its packed bf16 weight tiles
  // int8 models on the multi-CU kernel: the matrices as fp32 values code * scale (that kernel holds
  // its weights in registers and LDS for a whole call, so it takes them in fp32 and reads them once)
  void* dmem_f32 = nullptr;
  WnDevWeights w_chain{};
  // wn_abort's request word: coherent pinned host memory the kernels read at system scope
  int* abort_host = nullptr;
  int* abort_dev = nullptr;
};

namespace {
thread_local std::string g_err;
}  // namespace

int wn_set_last_error(int code, const char* msg) {
  g_err = msg;
  return code;
}
void wn_clear_last_error() { g_err.clear(); }

// Round fp32 to bfloat16, nearest even (NaN stays NaN).
uint16_t wn_to_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u) {
    if (u & 0x007fffffu) u |= 0x00400000u;
    return (uint16_t)(u >> 16);
  }
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

namespace {

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  g_err = std::string(what) + ": " + hipGetErrorString(e);
  return WN_EHIP;
}

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// int8 storage of a row-major [rows][cols] matrix: per row s = max|w| / 127 rounded to fp32, codes
// w / s (in double) rounded to nearest, ties to even, clamped to [-127, 127]; a zero row has s = 0
// and zero codes.
void quantize_rows_i8(const float* w, size_t rows, size_t cols, int8_t* codes, float* scale) {
  for (size_t i = 0; i < rows; ++i) {
    const float* row = w + i * cols;
    double mx = 0.0;
    for (size_t k = 0; k < cols; ++k) mx = std::max(mx, std::fabs((double)row[k]));
    const float s = (float)(mx / 127.0);
    scale[i] = s;
    for (size_t k = 0; k < cols; ++k) {
      const double q = s > 0.0f ? std::nearbyint((double)row[k] / (double)s) : 0.0;
      codes[i * cols + k] = (int8_t)std::min(127.0, std::max(-127.0, q));
    }
  }
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

// The multi-CU kernels poll their tagged words (histories, then mailboxes) through a buffer
// resource, whose byte offsets are 32-bit: the region must stay under 2 GiB.
bool tagged_region_fits(unsigned long long words) { return words * 8 + 4096 < (1ull << 31); }

// The multi-CU kernel's layout of B streams, if it serves them.
bool chain_plan_for(const wn_handle* h, int B, WnChainPlan* p) {
  if (!h->chain_ok || !wn_chain_plan(h->L, h->R, h->S, B, h->w.embed_prev != nullptr, p)) return false;
  return tagged_region_fits((unsigned long long)B * ((unsigned long long)h->dims.hist_len + (unsigned long long)p->mb_words));
}

// The multi-CU MFMA kernel's layout of B streams, if it serves them.
bool mchain_plan_for(const wn_handle* h, int B, WnChainPlan* p) {
  if (!h->mchain_ok || !wn_mchain_plan(h->L, h->R, h->S, B, p)) return false;
  return tagged_region_fits((unsigned long long)p->nrep *
                            ((unsigned long long)h->dims.hist_len * wn_mchain_columns(*p) + (unsigned long long)p->mb_words));
}

int variant_for(const wn_handle* h, int B) {
  WnChainPlan p;
  const std::string& f = h->force;
  if (f == "stream") return WN_VARIANT_STREAM;
  if (f == "multi_cu_mfma") return mchain_plan_for(h, B, &p) ? WN_VARIANT_MCHAIN : WN_VARIANT_STREAM;
  if (f == "multi_cu_chain") return chain_plan_for(h, B, &p) ? WN_VARIANT_CHAIN : WN_VARIANT_STREAM;
  if (f == "mfma_group") return h->group_ok ? WN_VARIANT_GROUP : WN_VARIANT_STREAM;
  // fp32 models: the fp32 multi-CU kernel while its replicas carry the batch.  bf16 and int8 models run
  // it on their exact fp32 copy while a replica carries at most 2 streams, and the MFMA one beyond
  // (measured at l = 20, r = 64, bf16: 11.7 / 14.7 / 18.6 / 24.8 us/step at 1 / 2 / 3 / 4 streams per
  // replica, against a flat 18.1 on the MFMA kernel; int8 the same within 0.2 us), then the batched
  // kernel (bf16); the fp32 one again for the shapes that neither MFMA kernel serves.
  // fp32 at r <= 64 goes to the per-stream kernel from 14 streams per replica on (measured at l = 20,
  // r = 64: 74.3 against 80.0 us/step at 12 streams per replica, 86.5 against ~83.6 at 14, 99.0
  // against 87.2 at 16); at r = 128 the per-stream kernel reads its weights from the MALL and
  // stays far behind (197 against 28 us/step at B = 32).
  const bool chain = chain_plan_for(h, B, &p);
  if (h->dtype == WN_F32) return chain && (h->R > 64 || p.G <= 13) ? WN_VARIANT_CHAIN : WN_VARIANT_STREAM;
  if (chain && p.G <= 2) return WN_VARIANT_CHAIN;
  WnChainPlan q;
  if (mchain_plan_for(h, B, &q)) return WN_VARIANT_MCHAIN;
  if (h->group_ok) return WN_VARIANT_GROUP;
  return chain ? WN_VARIANT_CHAIN : WN_VARIANT_STREAM;
}

// Workspace: status word, per-stream state, then either fp32 histories (per-stream and batched
// kernels) or tagged 64-bit histories followed by the inter-CU mailboxes and the launch-time
// block -> XCD map with its grid-barrier words (multi-CU kernel).
struct WsLayout {
  size_t status_off, state_off, hist_off, mb_off, mb_words, map_off, total;
};

WsLayout ws_layout(const wn_handle* h, int B) {
  WsLayout l;
  l.status_off = 0;
  l.state_off = 256;
  l.hist_off = align_up(l.state_off + (size_t)B * WN_STATE_WORDS * sizeof(int64_t), 256);
  WnChainPlan p;
  const int v = variant_for(h, B);
  if (v == WN_VARIANT_MCHAIN && mchain_plan_for(h, B, &p)) {
    // tagged histories of each replica's column blocks, then the replicas' mailboxes and the map
    l.mb_off = align_up(l.hist_off + (size_t)p.nrep * h->dims.hist_len * wn_mchain_columns(p) * 8, 256);
    l.mb_words = (size_t)p.nrep * p.mb_words;
    l.map_off = l.mb_off + l.mb_words * 8;
    l.total = align_up(l.map_off + (size_t)WN_CHAIN_MAP_WORDS * 8, 256);
  } else if (v == WN_VARIANT_CHAIN && chain_plan_for(h, B, &p)) {
    l.mb_off = align_up(l.hist_off + (size_t)B * h->dims.hist_len * 8, 256);
    l.mb_words = (size_t)B * p.mb_words;
    l.map_off = l.mb_off + l.mb_words * 8;
    l.total = align_up(l.map_off + (size_t)WN_CHAIN_MAP_WORDS * 8, 256);
  } else {
    l.mb_off = 0;
    l.mb_words = 0;
    l.map_off = 0;
    l.total = align_up(l.hist_off + (size_t)B * h->dims.hist_len * sizeof(float), 256);
  }
  return l;
}

const wn_sampler kDirect = {WN_SAMPLE_DIRECT, 1.0f, WN_A};

void set_sampler(WnIO& io, const wn_sampler& sp) {
  io.smode = sp.mode;
  io.inv_t = sp.mode == WN_SAMPLE_TEMPERATURE ? 1.0f / sp.temperature : 1.0f;
  io.top_k = sp.mode == WN_SAMPLE_TOPK ? sp.top_k : WN_A;
}

int check_sampler(const wn_sampler& sp) {
  if (sp.mode < WN_SAMPLE_DIRECT || sp.mode > WN_SAMPLE_MEAN) return fail(WN_EINVAL, "unknown sampling mode");
  if (sp.mode == WN_SAMPLE_TEMPERATURE && !(std::isfinite(sp.temperature) && sp.temperature > 0.0f))
    return fail(WN_EINVAL, "temperature must be finite and > 0");
  if (sp.mode == WN_SAMPLE_TEMPERATURE && !std::isfinite(1.0f / sp.temperature))
    return fail(WN_EINVAL, "temperature too small");
  if (sp.mode == WN_SAMPLE_TOPK && (sp.top_k < 1 || sp.top_k > WN_A)) return fail(WN_EINVAL, "top_k must be 1..a");
  return WN_OK;
}

int check_call(wn_handle* h, int B, int T, const void* cond, const void* a1, const void* a2, void* ws,
               size_t ws_bytes, int reset) {
  if (!h) return fail(WN_EINVAL, "null handle");
  if (B < 1) return fail(WN_EINVAL, "B must be >= 1");
  if (T < 0) return fail(WN_EINVAL, "T must be >= 0");
  if (reset != 0 && reset != 1) return fail(WN_EINVAL, "reset must be 0 or 1");
  if (T == 0) return WN_OK;
  if (!cond || !a1 || !a2) return fail(WN_EINVAL, "null input or output pointer");
  if (!ws) return fail(WN_EINVAL, "null workspace");
  if (reinterpret_cast<uintptr_t>(ws) % 256 != 0) return fail(WN_EINVAL, "workspace must be 256-byte aligned");
  if (ws_bytes < ws_layout(h, B).total) return fail(WN_EINVAL, "workspace too small");
  if ((size_t)B * (size_t)T > (size_t)1 << 40) return fail(WN_EINVAL, "B*T too large");
  return WN_OK;
}

int launch(wn_handle* h, int B, int T, const float* cond, const float* u, const int32_t* y_in, int32_t* y_out,
           float* logits, void* ws, int reset, void* stream, bool teacher, const wn_sampler& sp) {
  DeviceScope scope(h->device);
  if (!scope.ok()) return fail(WN_EHIP, "cannot select the handle's device");
  const WsLayout l = ws_layout(h, B);
  char* base = static_cast<char*>(ws);
  hipStream_t st = static_cast<hipStream_t>(stream);
  WnChainPlan plan;
  const int variant = variant_for(h, B);
  const bool mchain = variant == WN_VARIANT_MCHAIN && mchain_plan_for(h, B, &plan);
  if (mchain || (variant == WN_VARIANT_CHAIN && chain_plan_for(h, B, &plan))) {
    WnChainArgs g{};
    g.d = h->dims;
    // the fp32 multi-CU kernel takes an int8 model's fp32 copy; the MFMA one the int8 codes
    g.w = (h->dmem_f32 && !mchain) ? h->w_chain : h->w;
    g.io.cond = cond;
    g.io.u = u;
    g.io.y_in = y_in;
    g.io.y_out = y_out;
    g.io.logits = logits;
    g.io.B = B;
    g.io.T = T;
    g.io.reset = reset;
    g.io.init_sample = h->init_sample;
    g.io.abort_flag = h->abort_dev;
    set_sampler(g.io, sp);
    g.status = reinterpret_cast<int32_t*>(base + l.status_off);
    g.state = reinterpret_cast<int64_t*>(base + l.state_off);
    g.ring = reinterpret_cast<unsigned long long*>(base + l.hist_off);
    g.mb = reinterpret_cast<unsigned long long*>(base + l.mb_off);
    g.xmap = reinterpret_cast<unsigned long long*>(base + l.map_off);
    g.n_active = 0;
    for (int b = 0; b < WN_CHAIN_GRID; ++b) g.n_active += plan.role_of_block[b] != 0xffff;
    g.mb_words = plan.mb_words;
    g.off_h = plan.off_h;
    g.off_q = plan.off_q;
    g.off_x = plan.off_x;
    g.off_logit = plan.off_logit;
    g.off_qtail = plan.off_qtail;
    g.nch = plan.nch;
    for (int c = 0; c <= plan.nch; ++c) g.layer_begin[c] = plan.layer_begin[c];
    // polls before a wait gives up (seconds of spinning); WN_SPIN_LIMIT overrides it so that tests
    // can force the timeout path from the host
    g.spin_limit = 1 << 22;
    if (const char* sl = std::getenv("WN_SPIN_LIMIT")) {
      const long v = std::strtol(sl, nullptr, 10);
      if (v > 0 && v < (1L << 30)) g.spin_limit = (int)v;
    }
    g.nrep = plan.nrep;
    g.G = plan.G;
    g.ub = plan.ub;
    g.tail_on_chain = plan.tail_on_chain;
    g.nla = plan.nla;
    g.naux = plan.naux;
    g.naux_q = plan.naux_q;
    g.pair = plan.pair;
    for (int a = 0; a <= plan.naux; ++a) g.aux_begin[a] = plan.aux_begin[a];
    // posts to same-XCD readers stop at the XCD's L2 when the block -> XCD map is the expected
    // one; WN_LOCAL_POSTS=0 writes every post through
    const char* lp = std::getenv("WN_LOCAL_POSTS");
    g.local_posts = h->xcd_map && !(lp && lp[0] == '0');
    std::memcpy(g.role_of_block, plan.role_of_block, sizeof(g.role_of_block));
    if (reset) {
      const size_t words = (l.mb_off - l.hist_off) / 8 + l.mb_words + WN_CHAIN_MAP_WORDS;
      const hipError_t e = wn_chain_reset(g.ring, words, g.status, st);
      if (e != hipSuccess) return hip_fail(e, "reset kernel launch");
    }
    const hipError_t e = mchain ? wn_mchain_launch(g, teacher, st) : wn_chain_launch(g, teacher, st);
    if (e != hipSuccess) return hip_fail(e, "multi-CU kernel launch");
    return WN_OK;
  }
  if (variant == WN_VARIANT_GROUP) {
    WnGroupArgs g{};
    g.d = h->dims;
    g.w = h->w;
    g.packed = h->dpack;
    g.io.cond = cond;
    g.io.u = u;
    g.io.y_in = y_in;
    g.io.y_out = y_out;
    g.io.logits = logits;
    g.io.B = B;
    g.io.T = T;
    g.io.reset = reset;
    g.io.init_sample = h->init_sample;
    g.io.abort_flag = h->abort_dev;
    set_sampler(g.io, sp);
    g.ws.status = reinterpret_cast<int32_t*>(base + l.status_off);
    g.ws.state = reinterpret_cast<int64_t*>(base + l.state_off);
    g.ws.hist = reinterpret_cast<float*>(base + l.hist_off);
    g.gs = wn_group_streams(B);
    if (reset) {
      const hipError_t e = wn_status_clear(g.ws.status, st);
      if (e != hipSuccess) return hip_fail(e, "status clear launch");
    }
    const hipError_t e = wn_group_launch(g, teacher, st);
    if (e != hipSuccess) return hip_fail(e, "batched kernel launch");
    return WN_OK;
  }
  WnStreamArgs args{};
  args.d = h->dims;
  args.w = h->w;
  args.io.cond = cond;
  args.io.u = u;
  args.io.y_in = y_in;
  args.io.y_out = y_out;
  args.io.logits = logits;
  args.io.B = B;
  args.io.T = T;
  args.io.reset = reset;
  args.io.init_sample = h->init_sample;
  args.io.abort_flag = h->abort_dev;
  set_sampler(args.io, sp);
  args.ws.status = reinterpret_cast<int32_t*>(base + l.status_off);
  args.ws.state = reinterpret_cast<int64_t*>(base + l.state_off);
  args.ws.hist = reinterpret_cast<float*>(base + l.hist_off);
  if (reset) {
    const hipError_t se = wn_status_clear(args.ws.status, st);
    if (se != hipSuccess) return hip_fail(se, "status clear launch");
  }
  const hipError_t e = wn_stream_launch(args, teacher, st);
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return WN_OK;
}

}  // namespace

extern "C" {

int wn_create(const wn_config* c, const wn_weights* w, wn_handle** out) {
  g_err.clear();
  if (!c || !w || !out) return fail(WN_EINVAL, "null argument");
  if (c->n_layers < 1 || c->n_layers > WN_MAX_LAYERS) return fail(WN_EINVAL, "n_layers must be 1..64");
  if (!c->dilations) return fail(WN_EINVAL, "null dilations");
  if (c->r < 1 || c->s < 1 || c->a < 1) return fail(WN_EINVAL, "r, s, a must be >= 1");
  if (c->weight_dtype != WN_F32 && c->weight_dtype != WN_BF16 && c->weight_dtype != WN_I8)
    return fail(WN_EINVAL, "unknown weight_dtype");
  if (c->initial_sample < 0 || c->initial_sample >= c->a) return fail(WN_EINVAL, "initial_sample out of range");
  if (c->embed_taps < 1 || c->embed_taps > 2) return fail(WN_EINVAL, "embed_taps must be 1 or 2");
  if (c->nonlinearity != WN_NONLIN_EXACT && c->nonlinearity != WN_NONLIN_PAPER)
    return fail(WN_EINVAL, "unknown nonlinearity");
  long long hist_steps = 0;
  for (int j = 0; j < c->n_layers; ++j) {
    if (c->dilations[j] < 1 || c->dilations[j] > 65536) return fail(WN_EINVAL, "dilations must be 1..65536");
    hist_steps += c->dilations[j];
  }
  const void* need[] = {w->embed, w->b_embed, w->w_prev, w->w_cur, w->b_gate, w->w_res, w->b_res,
                        w->w_skip, w->b_skip, w->w_relu, w->b_relu, w->w_out, w->b_out};
  for (const void* p : need)
    if (!p) return fail(WN_EINVAL, "null weight array");
  if (c->a != WN_A) return fail(WN_EUNSUPPORTED, "a must be 256");
  if (!wn_stream_supported(c->r, c->s)) return fail(WN_EUNSUPPORTED, "unsupported (r, s) pair");

  wn_handle* h = new (std::nothrow) wn_handle();
  if (!h) return fail(WN_ENOMEM, "host allocation");
  h->L = c->n_layers;
  h->R = c->r;
  h->S = c->s;
  h->A = c->a;
  h->init_sample = c->initial_sample;
  h->dtype = c->weight_dtype;
  h->dil.assign(c->dilations, c->dilations + c->n_layers);
  if (hipGetDevice(&h->device) != hipSuccess) {
    delete h;
    return fail(WN_EHIP, "hipGetDevice failed");
  }
  const int L = h->L, R = h->R, S = h->S, A = h->A;
  h->dims.L = L;
  h->dims.R = R;
  h->dims.S = S;
  h->dims.hist_len = (int)(hist_steps * R);
  {
    int off = 0;
    for (int j = 0; j < L; ++j) {
      h->dims.dil[j] = h->dil[j];
      h->dims.hoff[j] = off;
      off += h->dil[j] * R;
    }
  }

  // Pack every array into one device allocation, each 256-byte aligned.  int8 storage adds one fp32
  // scale per matrix row (`cols` inputs per row).
  const bool bf = (h->dtype == WN_BF16), i8 = (h->dtype == WN_I8);
  const size_t we = bf ? 2 : (i8 ? 1 : 4);
  struct Arr { const float* src; size_t n; bool matrix; size_t cols; size_t off, soff; };
  Arr arrs[] = {
      {w->embed, (size_t)c->embed_taps * A * R, true, (size_t)R, 0, 0},
      {w->w_prev, (size_t)L * 2 * R * R, true, (size_t)R, 0, 0},
      {w->w_cur, (size_t)L * 2 * R * R, true, (size_t)R, 0, 0},
      {w->w_res, (size_t)L * R * R, true, (size_t)R, 0, 0},
      {w->w_skip, (size_t)L * S * R, true, (size_t)R, 0, 0},
      {w->w_relu, (size_t)A * S, true, (size_t)S, 0, 0},
      {w->w_out, (size_t)A * A, true, (size_t)A, 0, 0},
      {w->b_embed, (size_t)R, false, 0, 0, 0},
      {w->b_gate, (size_t)L * 2 * R, false, 0, 0, 0},
      {w->b_res, (size_t)L * R, false, 0, 0, 0},
      {w->b_skip, (size_t)S, false, 0, 0, 0},
      {w->b_relu, (size_t)A, false, 0, 0, 0},
      {w->b_out, (size_t)A, false, 0, 0, 0},
  };
  size_t total = 0;
  for (Arr& a : arrs) {
    a.off = total;
    total = align_up(total + a.n * (a.matrix ? we : 4), 256);
    if (a.matrix && i8) {
      a.soff = total;
      total = align_up(total + a.n / a.cols * 4, 256);
    }
  }
  std::vector<unsigned char> host(total, 0);
  for (const Arr& a : arrs) {
    if (a.matrix && bf) {
      uint16_t* d = reinterpret_cast<uint16_t*>(host.data() + a.off);
      for (size_t i = 0; i < a.n; ++i) d[i] = wn_to_bf16(a.src[i]);
    } else if (a.matrix && i8) {
      quantize_rows_i8(a.src, a.n / a.cols, a.cols, reinterpret_cast<int8_t*>(host.data() + a.off),
                       reinterpret_cast<float*>(host.data() + a.soff));
    } else {
      std::memcpy(host.data() + a.off, a.src, a.n * 4);
    }
  }
  hipError_t e = hipMalloc(&h->dmem, total);
  if (e != hipSuccess) {
    delete h;
    return e == hipErrorOutOfMemory ? fail(WN_ENOMEM, "hipMalloc of weights") : hip_fail(e, "hipMalloc");
  }
  e = hipMemcpy(h->dmem, host.data(), total, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(h->dmem);
    delete h;
    return hip_fail(e, "hipMemcpy of weights");
  }
  // the abort request word (wn_abort), in host memory the kernels can read while they run
  e = hipHostMalloc(reinterpret_cast<void**>(&h->abort_host), 256, hipHostMallocCoherent | hipHostMallocMapped);
  if (e == hipSuccess) {
    *h->abort_host = 0;
    e = hipHostGetDevicePointer(reinterpret_cast<void**>(&h->abort_dev), h->abort_host, 0);
  }
  if (e != hipSuccess) {
    if (h->abort_host) (void)hipHostFree(h->abort_host);
    (void)hipFree(h->dmem);
    delete h;
    return e == hipErrorOutOfMemory ? fail(WN_ENOMEM, "pinned host allocation of the abort word")
                                    : hip_fail(e, "abort word");
  }
  char* d = static_cast<char*>(h->dmem);
  // [taps][A][R]: the last table embeds y_{t-1}, the first of two y_{t-2}
  h->w.embed = d + arrs[0].off + (size_t)(c->embed_taps - 1) * A * R * we;
  h->w.embed_prev = c->embed_taps == 2 ? d + arrs[0].off : nullptr;
  h->w.w_prev = d + arrs[1].off;
  h->w.w_cur = d + arrs[2].off;
  h->w.w_res = d + arrs[3].off;
  h->w.w_skip = d + arrs[4].off;
  h->w.w_relu = d + arrs[5].off;
  h->w.w_out = d + arrs[6].off;
  h->w.b_embed = reinterpret_cast<const float*>(d + arrs[7].off);
  h->w.b_gate = reinterpret_cast<const float*>(d + arrs[8].off);
  h->w.b_res = reinterpret_cast<const float*>(d + arrs[9].off);
  h->w.b_skip = reinterpret_cast<const float*>(d + arrs[10].off);
  h->w.b_relu = reinterpret_cast<const float*>(d + arrs[11].off);
  h->w.b_out = reinterpret_cast<const float*>(d + arrs[12].off);
  h->w.bf16 = bf ? 1 : 0;
  h->w.i8 = i8 ? 1 : 0;
  if (i8) {
    auto sc = [&](int k) { return reinterpret_cast<const float*>(d + arrs[k].soff); };
    h->w.s_embed = sc(0) + (size_t)(c->embed_taps - 1) * A;
    h->w.s_embed_prev = c->embed_taps == 2 ? sc(0) : nullptr;
    h->w.s_prev = sc(1);
    h->w.s_cur = sc(2);
    h->w.s_res = sc(3);
    h->w.s_skip = sc(4);
    h->w.s_relu = sc(5);
    h->w.s_out = sc(6);
  }
  h->w.approx_nl = c->nonlinearity == WN_NONLIN_PAPER ? 1 : 0;

  // The multi-CU kernels need one CU per block of their grid and a supported shape: the fp32 one runs
  // on fp32 weights (for bf16 and int8 models on an exact fp32 copy), the MFMA one on bf16 or int8
  // weights.
  if (const char* force = std::getenv("WN_KERNEL")) h->force = force;
  const bool want_chain = h->force != "stream";
  int cus = 0, coop = 0;
  (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, h->device);
  (void)hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, h->device);
  if (want_chain && wn_chain_supported(R, S, L) && cus >= WN_CHAIN_GRID && coop) h->chain_ok = true;
  if (want_chain && (bf || i8) && wn_mchain_supported(R, S, L) && cus >= WN_CHAIN_GRID && coop) h->mchain_ok = true;
  if (h->chain_ok || h->mchain_ok) h->xcd_map = wn_chain_xcd_map_ok();
  if (h->chain_ok && (i8 || bf)) {
    // fp32 copies of the matrices for the multi-CU kernel: each bf16 weight (exact in fp32), or each
    // int8 code * scale, rounded to fp32 once here (the per-stream kernel multiplies its row sums by
    // the scale instead)
    size_t ftotal = 0;
    std::vector<size_t> foff(7);
    for (int k = 0; k < 7; ++k) {
      foff[k] = ftotal;
      ftotal = align_up(ftotal + arrs[k].n * 4, 256);
    }
    std::vector<float> fh(ftotal / 4, 0.f);
    for (int k = 0; k < 7; ++k) {
      if (bf) {
        const uint16_t* bits = reinterpret_cast<const uint16_t*>(host.data() + arrs[k].off);
        for (size_t i = 0; i < arrs[k].n; ++i) {
          const uint32_t u = (uint32_t)bits[i] << 16;
          std::memcpy(&fh[foff[k] / 4 + i], &u, 4);
        }
      } else {
        const int8_t* codes = reinterpret_cast<const int8_t*>(host.data() + arrs[k].off);
        const float* scale = reinterpret_cast<const float*>(host.data() + arrs[k].soff);
        for (size_t i = 0; i < arrs[k].n; ++i) fh[foff[k] / 4 + i] = (float)codes[i] * scale[i / arrs[k].cols];
      }
    }
    e = hipMalloc(&h->dmem_f32, ftotal);
    if (e == hipSuccess) e = hipMemcpy(h->dmem_f32, fh.data(), ftotal, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      if (h->dmem_f32) (void)hipFree(h->dmem_f32);
      (void)hipFree(h->dmem);
      (void)hipHostFree(h->abort_host);
      delete h;
      return e == hipErrorOutOfMemory ? fail(WN_ENOMEM, "hipMalloc of fp32 weights") : hip_fail(e, "fp32 weights upload");
    }
    char* f = static_cast<char*>(h->dmem_f32);
    h->w_chain = h->w;
    h->w_chain.embed = f + foff[0] + (size_t)(c->embed_taps - 1) * A * R * 4;
    h->w_chain.embed_prev = c->embed_taps == 2 ? f + foff[0] : nullptr;
    h->w_chain.w_prev = f + foff[1];
    h->w_chain.w_cur = f + foff[2];
    h->w_chain.w_res = f + foff[3];
    h->w_chain.w_skip = f + foff[4];
    h->w_chain.w_relu = f + foff[5];
    h->w_chain.w_out = f + foff[6];
    h->w_chain.i8 = 0;
    h->w_chain.bf16 = 0;
  }
  // The batched MFMA kernel needs bf16 weights, r = 64 and its LDS footprint on one CU.
  int lds_max = 0;
  (void)hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, h->device);
  if (want_chain && bf && wn_group_supported(R, S, L) && wn_group_lds_bytes(L, S, c->embed_taps == 2) + 256 <= (size_t)lds_max) {
    const std::vector<uint16_t> tiles =
        wn_group_pack(L, R, S, w->w_prev, w->w_cur, w->w_res, w->w_skip, w->w_relu, w->w_out);
    e = hipMalloc(&h->dpack, tiles.size() * sizeof(uint16_t));
    if (e == hipSuccess) e = hipMemcpy(h->dpack, tiles.data(), tiles.size() * sizeof(uint16_t), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      if (h->dpack) (void)hipFree(h->dpack);
      (void)hipFree(h->dmem);
      (void)hipHostFree(h->abort_host);
      delete h;
      return e == hipErrorOutOfMemory ? fail(WN_ENOMEM, "hipMalloc of packed weights")
                                      : hip_fail(e, "packed weights upload");
    }
    h->group_ok = true;
  }
  *out = h;
  return WN_OK;
}

size_t wn_workspace_bytes(const wn_handle* h, int32_t B) {
  if (!h || B < 1) return 0;
  return ws_layout(h, B).total;
}

int wn_generate(wn_handle* h, int32_t B, int32_t T, const float* cond, const float* uniforms, int32_t* samples,
                void* workspace, size_t ws_bytes, int32_t reset, void* stream) {
  g_err.clear();
  int rc = check_call(h, B, T, cond, uniforms, samples, workspace, ws_bytes, reset);
  if (rc != WN_OK || T == 0) return rc;
  return launch(h, B, T, cond, uniforms, nullptr, samples, nullptr, workspace, reset, stream, false, kDirect);
}

int wn_generate_sampled(wn_handle* h, int32_t B, int32_t T, const float* cond, const float* uniforms,
                        int32_t* samples, void* workspace, size_t ws_bytes, int32_t reset,
                        const wn_sampler* sampler, void* stream) {
  g_err.clear();
  const wn_sampler sp = sampler ? *sampler : kDirect;
  int rc = check_sampler(sp);
  if (rc != WN_OK) return rc;
  rc = check_call(h, B, T, cond, uniforms, samples, workspace, ws_bytes, reset);
  if (rc != WN_OK || T == 0) return rc;
  return launch(h, B, T, cond, uniforms, nullptr, samples, nullptr, workspace, reset, stream, false, sp);
}

int wn_teacher_force(wn_handle* h, int32_t B, int32_t T, const float* cond, const int32_t* y, float* logits,
                     void* workspace, size_t ws_bytes, int32_t reset, void* stream) {
  g_err.clear();
  int rc = check_call(h, B, T, cond, y, logits, workspace, ws_bytes, reset);
  if (rc != WN_OK || T == 0) return rc;
  return launch(h, B, T, cond, nullptr, y, nullptr, logits, workspace, reset, stream, true, kDirect);
}

int wn_status(wn_handle* h, const void* workspace, void* stream) {
  g_err.clear();
  if (!h || !workspace) return fail(WN_EINVAL, "null argument");
  DeviceScope scope(h->device);
  if (!scope.ok()) return fail(WN_EHIP, "cannot select the handle's device");
  int32_t st = 0;
  hipError_t e = hipMemcpyAsync(&st, workspace, sizeof(st), hipMemcpyDeviceToHost, static_cast<hipStream_t>(stream));
  if (e == hipSuccess) e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "reading the status word");
  return st;
}

int wn_abort(wn_handle* h, int32_t on) {
  g_err.clear();
  if (!h) return fail(WN_EINVAL, "null handle");
  if (on != 0 && on != 1) return fail(WN_EINVAL, "on must be 0 or 1");
  __atomic_store_n(h->abort_host, on, __ATOMIC_SEQ_CST);
  return WN_OK;
}

const char* wn_kernel_variant(const wn_handle* h, int32_t B) {
  if (!h || B < 1) return "";
  switch (variant_for(h, B)) {
    case WN_VARIANT_CHAIN: return "multi_cu_chain";
    case WN_VARIANT_MCHAIN: return "multi_cu_mfma";
    case WN_VARIANT_GROUP: return "mfma_group";
    default: return "stream_l2";
  }
}

int wn_launch_info(const wn_handle* h, int32_t B, int32_t* workgroups, int32_t* replicas) {
  if (!h || B < 1 || !workgroups || !replicas) return WN_EINVAL;
  WnChainPlan p;
  const int v = variant_for(h, B);
  if ((v == WN_VARIANT_MCHAIN && mchain_plan_for(h, B, &p)) || (v == WN_VARIANT_CHAIN && chain_plan_for(h, B, &p))) {
    int used = 0;
    for (int b = 0; b < WN_CHAIN_GRID; ++b) used += p.role_of_block[b] != 0xffff;
    *workgroups = used;
    *replicas = p.nrep;
  } else if (v == WN_VARIANT_GROUP) {
    const int gs = wn_group_streams(B);
    *workgroups = (B + gs - 1) / gs;
    *replicas = *workgroups;
  } else {
    *workgroups = B;
    *replicas = B;
  }
  return WN_OK;
}

void wn_destroy(wn_handle* h) {
  if (!h) return;
  {
    DeviceScope scope(h->device);
    if (h->dmem) (void)hipFree(h->dmem);
    if (h->dpack) (void)hipFree(h->dpack);
    if (h->dmem_f32) (void)hipFree(h->dmem_f32);
    if (h->abort_host) (void)hipHostFree(h->abort_host);
  }
  delete h;
}

const char* wn_error_string(int code) {
  switch (code) {
    case WN_OK: return "success";
    case WN_EINVAL: return "invalid argument";
    case WN_EUNSUPPORTED: return "model not supported by any kernel";
    case WN_ENOMEM: return "out of memory";
    case WN_EHIP: return "HIP runtime error";
    case WN_ETIMEOUT: return "kernel wait timed out";
    case WN_EABORTED: return "kernel aborted";
    default: return "unknown error";
  }
}

const char* wn_last_error(void) { return g_err.c_str(); }

}  // extern "C"
