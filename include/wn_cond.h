/*
 * wn_cond.h -- C ABI of libwn's conditioning network on an AMD Instinct MI355X
 * (gfx950): the per-layer conditioning L of every audio step, computed from
 * linguistic features at the frame rate (Deep Voice, arXiv 1702.07825,
 * Appendix A.2, "Conditioning Network").
 *
 * Two bidirectional QRNN layers with fo-pooling and width-2 convolutions; a
 * unidirectional layer computes, over the frames in its own order,
 *   h~_t = tanh(W_h * x + B_h), o_t = sigmoid(W_o * x + B_o), f_t = sigmoid(W_f * x + B_f)
 *   h_t  = f_t h_{t-1} + (1 - f_t) h~_t   (h before the first frame is 0),  z_t = o_t h_t
 * where W * x is the width-2 convolution over the frame before t in that order
 * (zero before the first) and frame t.  The backward direction runs on the
 * reversed frames (its previous frame is t + 1); a layer's output stacks the
 * forward channels, then the backward ones.  After the second layer, output
 * channel 2k + d is channel k of direction d, so that the tanh and the sigmoid
 * half of every WaveNet layer get channels of both directions; the second layer
 * has h2 = n_layers * r channels per direction, and the 2 h2 channels of an
 * audio step are the WaveNet's L, layer j in block j of 2r.  Audio step tau
 * repeats frame floor(tau * frame_rate / audio_rate) (upsampling by repetition).
 *
 * Conventions as in wn.h: host fp32 weights copied by wn_cond_create; features,
 * cond and workspace are caller-owned device pointers; calls are asynchronous
 * on `stream`; negative wn_status_t codes on failure, wn_last_error() for detail.
 */
#ifndef WN_COND_H_
#define WN_COND_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t n_features;   /* F, 1 .. 4096 (227 in the paper) */
  int32_t h1;           /* channels per direction of the first QRNN layer, 1 .. 4096 */
  int32_t n_layers, r;  /* the WaveNet conditioned: h2 = n_layers * r, 1 .. 8192 */
  int32_t frame_rate;   /* Hz of the features (256 in the paper) */
  int32_t audio_rate;   /* Hz of the audio steps */
} wn_cond_config;

typedef struct {        /* host fp32; gate rows in blocks h~, o, f; tap 0 = previous frame, 1 = current */
  const float* w1;      /* [2][3 h1][2][F]   direction, gate row, tap, input */
  const float* b1;      /* [2][3 h1] */
  const float* w2;      /* [2][3 h2][2][2 h1] */
  const float* b2;      /* [2][3 h2] */
} wn_cond_weights;

typedef struct wn_cond wn_cond;

/* Validate a configuration and copy the weights to the current device.  Errors: WN_EINVAL
 * (null pointers, sizes out of range), WN_ENOMEM, WN_EHIP.  *out is set only on success. */
int wn_cond_create(const wn_cond_config* config, const wn_cond_weights* weights, wn_cond** out);

/* Device workspace bytes one call with B streams of n_frames frames needs (0 if invalid). */
size_t wn_cond_workspace_bytes(const wn_cond* c, int32_t B, int32_t n_frames);

/*
 * Conditioning of T audio steps for each of B streams.
 *   features  device fp32 [B][n_frames][F]
 *   cond      device fp32 [B][T][n_layers][2r] out (the layout wn_generate reads)
 *   workspace device, >= wn_cond_workspace_bytes(c, B, n_frames) bytes, 256-byte aligned
 * T = 0 is a no-op.  Errors: WN_EINVAL (B < 1, n_frames < 1, T < 0, null pointers, a short or
 * misaligned workspace, or floor((T - 1) * frame_rate / audio_rate) >= n_frames); WN_EHIP.
 */
int wn_condition(wn_cond* c, int32_t B, int32_t n_frames, const float* features, int32_t T, float* cond,
                 void* workspace, size_t ws_bytes, void* stream);

/*
 * Bytes of the static scratch array wn_condition_static uses on each device: a call with B streams
 * of n_frames frames is accepted while wn_cond_workspace_bytes(c, B, n_frames) is at most this
 * (64 MiB: about 5.8 s of audio at 256 frames per second for l = 20, r = 64, h1 = 256).
 */
#define WN_COND_SCRATCH_BYTES ((size_t)64 << 20)

/*
 * wn_condition without a workspace argument, for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).  The scratch the
 * three kernels use (gate pre-activations, the first layer's output, the frame-rate output) lives
 * in one static device array per device, WN_COND_SCRATCH_BYTES long, which the library holds
 * from its first use on a device until the process ends; wn_cond_create looks up that device's
 * address of it.  This call allocates nothing and calls no allocating routine.
 * Every call on one device shares that device's array: two calls that overlap in time on one
 * device (on different streams, or from different threads or handles) race and give undefined
 * results; calls ordered on one stream do not.  The array keeps the last call's contents; no
 * result depends on them (every word a call reads it has written first).
 * Arguments, results and errors as wn_condition, plus WN_EINVAL when
 * wn_cond_workspace_bytes(c, B, n_frames) > WN_COND_SCRATCH_BYTES (nothing is launched).
 */
int wn_condition_static(wn_cond* c, int32_t B, int32_t n_frames, const float* features, int32_t T, float* cond,
                        void* stream);

/* Free the device weights.  Null is allowed.  No call may be in flight. */
void wn_cond_destroy(wn_cond* c);

#ifdef __cplusplus
}
#endif

#endif /* WN_COND_H_ */
