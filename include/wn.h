/*
 * wn.h -- C ABI of libwn, autoregressive WaveNet sample generation on an
 * AMD Instinct MI355X (gfx950).
 *
 * The model is the auto-regressive WaveNet of Deep Voice (arXiv 1702.07825),
 * Appendix A.1: an input embedding of the previous mu-law sample, l gated layers
 * of width-2 dilated causal convolutions with residual and skip 1x1
 * projections, a relu -> 1x1 -> relu -> 1x1 head over a = 256 classes, a softmax
 * and a draw from it ("direct sampling", Appendix A.4, "Sampling from Output
 * Distribution").  Generation runs one sample per step; the per-layer
 * conditioning is an input computed beforehand, as in the paper's inference
 * benchmark (Section 5), which excludes the conditioning network.
 *
 * Per stream b and step t (t = 0 .. T-1 within a call, tg = global step):
 *   x0      = E[y_{tg-1}] + B_embed        (two taps: + E_prev[y_{tg-2}], Section 5.1)
 *   a_j     = W_prev_j x_{j-1}[tg - d_j] + W_cur_j x_{j-1}[tg] + B_j + L[b,t,j,:]
 *   h_j     = tanh(a_j[0:r]) * sigmoid(a_j[r:2r])
 *   x_j     = x_{j-1} + W_res_j h_j + B_res_j
 *   q       = B_skip + sum_j W_skip_j h_j
 *   logits  = W_out relu(W_relu relu(q) + B_relu) + B_out
 *   y_tg    = #{k <= a-2 : C_k <= u[b,t]},  C_k = p_0 + .. + p_k,  p = softmax(logits)
 * Layer histories are zero before the first step, y_{-1} = initial_sample, and
 * y_{-2} contributes nothing.
 *
 * Conventions:
 *  - Every matrix is row-major [out][in], fp32 on the host.  wn_create copies
 *    (and for WN_BF16 / WN_I8 converts, see wn_dtype_t) them into device memory owned
 *    by the handle; the caller's host arrays may be freed afterwards.
 *  - cond, uniforms, samples, y, logits and workspace are DEVICE pointers owned
 *    by the caller.  Calls are asynchronous and ordered on `stream` (a
 *    hipStream_t, NULL = the default stream); the caller keeps every buffer alive
 *    until the stream has passed the call.
 *  - A handle is bound to the HIP device current at wn_create; the library makes
 *    that device current for the duration of each call and restores the
 *    caller's device before returning.
 *  - Return codes: WN_OK on success, a negative wn_status_t otherwise.  Nothing
 *    is launched when an argument check fails.  wn_last_error() gives a detail
 *    string for the calling thread's last failure.
 *  - Two calls that share one workspace must not overlap in time.
 *  - Environment variables (tuning and tests; read at wn_create or at each call):
 *      WN_KERNEL=name        wn_create: serve every call with one kernel family (a name that
 *                            wn_kernel_variant returns; calls it cannot serve use stream_l2)
 *      WN_SPIN_LIMIT=n       each call: polls before a multi-CU wait gives up (wn_status)
 *      WN_LOCAL_POSTS=0      each call: the multi-CU kernel writes every message through to
 *                            memory instead of stopping same-XCD messages at the XCD's L2
 *      WN_GROUP_STREAMS=8|16 each call: streams per workgroup of the batched bf16 kernel
 *      WN_AUX_LAYERS=n       each call: layers per aux CU of the multi-CU kernels (fp32: 1 instead
 *                            of two; MFMA: 1..5 instead of the default runs); it changes the
 *                            launch layout and the workspace size
 *      WN_MFMA_COLUMNS=16    each call: the multi-CU MFMA kernel carries 16 streams per replica
 *                            (one per tile column) also where 8 in paired columns would do
 *    Apart from a small WN_SPIN_LIMIT, which can make a wait time out, none of them changes a
 *    result beyond rounding.
 */
#ifndef WN_H_
#define WN_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  WN_OK = 0,
  WN_EINVAL = -1,        /* a null pointer, a size out of range, a short workspace */
  WN_EUNSUPPORTED = -2,  /* a valid model that no kernel here implements (see wn_create) */
  WN_ENOMEM = -3,        /* device or host allocation failed */
  WN_EHIP = -4,          /* a HIP runtime call failed; wn_last_error() has its message */
  WN_ETIMEOUT = -5,      /* a kernel's bounded wait expired (reported by wn_status) */
  WN_EABORTED = -6       /* a call stopped early on a wn_abort request (reported by wn_status) */
} wn_status_t;

/*
 * Storage of the matrices and the embedding table (biases, activations and accumulation are always
 * fp32):
 *   WN_F32   as given
 *   WN_BF16  rounded to bfloat16, nearest even
 *   WN_I8    int8 codes with one fp32 scale per row (the paper runs int16 weights in its CPU
 *            kernels, Section 5.1, and names lower precision as further work): per row
 *            s = max|w| / 127 rounded to fp32, code = w / s (the quotient in double) rounded to
 *            nearest, ties to even, clamped to [-127, 127]; a zero row has s = 0.  The weight used
 *            is code * s.
 */
typedef enum { WN_F32 = 0, WN_BF16 = 1, WN_I8 = 2 } wn_dtype_t;

/*
 * How a step's output distribution P = softmax(logits) becomes its sample: the ways the paper
 * lists (Appendix A.4, "Sampling from Output Distribution").  C_k is the CDF of the distribution
 * sampled and u the step's uniform.
 *   WN_SAMPLE_DIRECT       y = #{k <= a-2 : C_k <= u} on P (what wn_generate does)
 *   WN_SAMPLE_TEMPERATURE  the same on P^(1/t) / Z = softmax(logits / t), t = temperature > 0
 *   WN_SAMPLE_TOPK         the same on P kept where its logit is at least the top_k-th largest
 *                          logit (ties at the top_k-th are kept) and renormalised, 1 <= top_k <= a
 *   WN_SAMPLE_MODE         argmax P, the smallest index among equal maxima (u unused)
 *   WN_SAMPLE_MEAN         E_P[y] = sum_k k P(k) to the nearest index, halves up (u unused; the
 *                          paper does not say how the mean becomes an index)
 */
typedef enum {
  WN_SAMPLE_DIRECT = 0,
  WN_SAMPLE_TEMPERATURE = 1,
  WN_SAMPLE_TOPK = 2,
  WN_SAMPLE_MODE = 3,
  WN_SAMPLE_MEAN = 4
} wn_sample_mode_t;

typedef struct {
  int32_t mode;       /* wn_sample_mode_t */
  float temperature;  /* WN_SAMPLE_TEMPERATURE: t > 0 (finite); ignored otherwise */
  int32_t top_k;      /* WN_SAMPLE_TOPK: 1 .. a; ignored otherwise */
} wn_sampler;

/* Nonlinearities: exact (hardware exp2 and reciprocal, the default), or the approximations of
 * Appendix C ("Nonlinearity Approximation Details"): tanh and sigmoid through
 * e~(x) = 1 + |x| + 0.5658 x^2 + 0.143 x^4, e^x through the fp32 bit pattern of 2^(x / ln 2) with
 * the appendix's rational fit of 2^z - z.  Their largest errors against the exact functions are
 * 1.5e-3 (tanh), 2.6e-3 (sigmoid) and 4.8e-5 (e^x on x <= 0). */
typedef enum { WN_NONLIN_EXACT = 0, WN_NONLIN_PAPER = 1 } wn_nonlin_t;

typedef struct {
  int32_t n_layers;          /* l, 1 .. 64 */
  int32_t r;                 /* residual channels: 16, 32, 64 or 128 */
  int32_t s;                 /* skip channels: 32, 64, 128 or 256 */
  int32_t a;                 /* output classes: must be 256 (8-bit mu-law) */
  const int32_t* dilations;  /* host [n_layers], each 1 .. 65536; copied by wn_create */
  int32_t embed_taps;        /* 1: x0 = E[y_{t-1}] + B_embed;
                                2: x0 = E_prev[y_{t-2}] + E_cur[y_{t-1}] + B_embed, the width-2
                                input convolution of Section 5.1 (y_{t-2} before the first step
                                contributes nothing) */
  int32_t initial_sample;    /* y_{-1}, 0 .. a-1; 128 is the mu-law code of silence */
  int32_t weight_dtype;      /* wn_dtype_t: storage of the matrices and the embedding;
                                biases, activations and accumulation are always fp32 */
  int32_t nonlinearity;      /* wn_nonlin_t: the gate's tanh and sigmoid and the softmax's exp */
} wn_config;

typedef struct {             /* host fp32, row-major, shapes below */
  const float* embed;        /* [taps][a][r] embedding tables: the last embeds y_{t-1},
                                            with two taps the first embeds y_{t-2}      */
  const float* b_embed;      /* [r]                                                 */
  const float* w_prev;       /* [l][2r][r]   conv tap on x_{t-d} (rows 0..r-1 tanh)  */
  const float* w_cur;        /* [l][2r][r]   conv tap on x_t                         */
  const float* b_gate;       /* [l][2r]      B = B_h || B_g                          */
  const float* w_res;        /* [l][r][r]                                           */
  const float* b_res;        /* [l][r]                                              */
  const float* w_skip;       /* [l][s][r]    column block j of the skip projection  */
  const float* b_skip;       /* [s]                                                 */
  const float* w_relu;       /* [a][s]                                              */
  const float* b_relu;       /* [a]                                                 */
  const float* w_out;        /* [a][a]                                              */
  const float* b_out;        /* [a]                                                 */
} wn_weights;

typedef struct wn_handle wn_handle;

/*
 * Validate a model, copy its weights to the current device and return a handle.
 * Model: Appendix A.1 (layer equations) and Section 5 (the W_prev/W_cur split
 * of each dilated convolution into two matrix-vector products per step).
 * Errors: WN_EINVAL for null pointers or values out of the ranges above;
 * WN_EUNSUPPORTED for a != 256, or an (r, s) pair outside
 * {(16,32), (32,128), (64,128), (64,256), (128,256)}; WN_ENOMEM; WN_EHIP.
 * *out is set only on success.
 */
int wn_create(const wn_config* config, const wn_weights* weights, wn_handle** out);

/*
 * Bytes of device workspace one call with B streams needs: the generator state
 * of every stream (each layer's dilation history of r fp32 values per step of
 * its dilation, the step counter and the last two samples) plus a status word.
 * The layout is private.  Returns 0 for a null handle or B < 1.
 */
size_t wn_workspace_bytes(const wn_handle* h, int32_t B);

/*
 * Generate T samples for each of B independent streams (one utterance each).
 *   cond      device fp32 [B][T][l][2r]  per-layer conditioning L (Appendix A.1):
 *             columns 0..r-1 are added to the tanh half, r..2r-1 to the sigmoid half
 *   uniforms  device fp32 [B][T], each in [0, 1): the draw of step t uses uniforms[b][t]
 *   samples   device int32 [B][T] out, values 0 .. a-1
 *   workspace device, >= wn_workspace_bytes(h, B) bytes, 256-byte aligned
 *   reset     1: start every stream from zero histories and y_{-1} = initial_sample;
 *             0: continue from the state the previous call on this workspace left
 *             (same B), so T1 steps then T2 steps equal T1 + T2 steps in one call.
 * T = 0 is a no-op (returns WN_OK).  Errors: WN_EINVAL (B < 1, T < 0, null
 * pointers when T > 0, misaligned or short workspace, reset not 0/1); WN_EHIP.
 */
int wn_generate(wn_handle* h, int32_t B, int32_t T, const float* cond, const float* uniforms,
                int32_t* samples, void* workspace, size_t ws_bytes, int32_t reset, void* stream);

/*
 * wn_generate with another way of turning each step's distribution into its sample (see
 * wn_sampler; Appendix A.4).  sampler = NULL is direct sampling.  uniforms are required for
 * every mode (MODE and MEAN read none of them).  Errors: those of wn_generate, and WN_EINVAL for
 * an unknown mode, a temperature that is not finite and > 0, or top_k outside 1 .. a.
 */
int wn_generate_sampled(wn_handle* h, int32_t B, int32_t T, const float* cond, const float* uniforms,
                        int32_t* samples, void* workspace, size_t ws_bytes, int32_t reset,
                        const wn_sampler* sampler, void* stream);

/*
 * Teacher forcing: step t consumes y[b][t-1] (for t = 0: y_{-1} = initial_sample
 * after a reset, else the last sample of the previous call) instead of its own
 * draw, and writes the pre-softmax logits of every step.
 *   y       device int32 [B][T], values 0 .. a-1 (values outside are clamped)
 *   logits  device fp32 [B][T][a] out
 * Other arguments and errors as wn_generate.
 */
int wn_teacher_force(wn_handle* h, int32_t B, int32_t T, const float* cond, const int32_t* y,
                     float* logits, void* workspace, size_t ws_bytes, int32_t reset, void* stream);

/*
 * Wait for `stream` and return the status word the kernels left in `workspace`:
 * WN_OK, WN_ETIMEOUT or WN_EABORTED; WN_EINVAL for null arguments; WN_EHIP if
 * the stream reports an error.  Blocks the calling thread.  The multi-CU kernel's
 * waits for other CUs give up after a bounded number of polls (a few seconds);
 * the environment variable WN_SPIN_LIMIT, read at each call, sets that number
 * (tests force the timeout path with it).  After WN_ETIMEOUT or WN_EABORTED the
 * workspace state is stale: the next call must pass reset = 1.
 */
int wn_status(wn_handle* h, const void* workspace, void* stream);

/*
 * Request (on = 1) or withdraw (on = 0) an early stop of this handle's calls, from any host
 * thread, also while a call runs.  The request is a word in pinned host memory that the handle
 * owns; every kernel of a wn_generate, wn_generate_sampled or wn_teacher_force call of this
 * handle reads it at the call's first step and every 64 steps after, and once it reads 1 the
 * whole grid leaves at a step boundary (its outputs from that step on are not written) and the
 * call's status word becomes WN_EABORTED (wn_status).  While the request stands, calls still
 * launch and stop at their first step; withdraw it before the next call, which must pass
 * reset = 1.  A call that has passed its last check finishes normally (status WN_OK).
 * Errors: WN_EINVAL (null handle, on not 0 or 1).  Nothing is launched.
 */
int wn_abort(wn_handle* h, int32_t on);

/* Name of the kernel family that calls with B streams use (for reports):
 *   multi_cu_chain  fp32 (and int8) weights, resident across many CUs, VALU products
 *   multi_cu_mfma   bf16 and int8 weights (r = 64, s = 256), resident across many CUs, up to 16
 *                   streams per replica as the columns of MFMA tiles
 *   mfma_group      bf16 weights (r = 64), every layer of a group of streams on one CU
 *   stream_l2       any model, one workgroup per stream */
const char* wn_kernel_variant(const wn_handle* h, int32_t B);

/* For reports: the workgroups (one per CU) a call with B streams launches, and how many
 * independent copies of the model they form (multi-CU kernel: replicas; the others: one per
 * workgroup).  WN_EINVAL for a null handle or pointer or B < 1. */
int wn_launch_info(const wn_handle* h, int32_t B, int32_t* workgroups, int32_t* replicas);

/* Free the handle's device weights.  Null is allowed.  No call may be in flight. */
void wn_destroy(wn_handle* h);

/* Static description of a return code. */
const char* wn_error_string(int code);

/* Detail of the calling thread's last failure ("" if none). */
const char* wn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* WN_H_ */
