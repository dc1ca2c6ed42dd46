// Internal interface between the libwn host code and its HIP kernels (gfx950).
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>
#include <vector>

#define WN_MAX_LAYERS 64
#define WN_A 256
// Per-stream generator state in the workspace, int64 words: steps taken, y_{t-1}, y_{t-2}
// (-1 before the first input), one spare.
#define WN_STATE_WORDS 4

// Model sizes and the per-stream history layout: layer j keeps d_j slots of r
// floats starting at hoff[j] (in floats) inside a stream's history block of
// hist_len floats.
struct WnDims {
  int L, R, S;
  int hist_len;
  int dil[WN_MAX_LAYERS];
  int hoff[WN_MAX_LAYERS];
};

// Device copies of the weights.  Matrices are row-major [out][in] and either
// fp32, bf16 (uint16 bit patterns) or int8 codes with one fp32 scale per row; biases are fp32.
struct WnDevWeights {
  const void* embed;       // [A][R] embedding of y_{t-1}
  const void* embed_prev;  // [A][R] embedding of y_{t-2} (two-tap input convolution), or null
  const void* w_prev;  // [L][2R][R]
  const void* w_cur;   // [L][2R][R]
  const void* w_res;   // [L][R][R]
  const void* w_skip;  // [L][S][R]
  const void* w_relu;  // [A][S]
  const void* w_out;   // [A][A]
  const float* b_embed;
  const float* b_gate;
  const float* b_res;
  const float* b_skip;
  const float* b_relu;
  const float* b_out;
  int bf16;
  int i8;  // 1: int8 codes; the weight of row i is code * s_<matrix>[i]
  const float* s_embed;       // [A] scales of the y_{t-1} table
  const float* s_embed_prev;  // [A] scales of the y_{t-2} table (two taps)
  const float* s_prev;        // [L][2R]
  const float* s_cur;         // [L][2R]
  const float* s_res;         // [L][R]
  const float* s_skip;        // [L][S]
  const float* s_relu;        // [A]
  const float* s_out;         // [A]
  int approx_nl;  // 1: the approximate tanh, sigmoid and softmax exp of the paper's Appendix C
};

// One call's inputs and outputs (device pointers, caller-owned).
struct WnIO {
  const float* cond;    // [B][T][L][2R]
  const float* u;       // [B][T]            (generation)
  const int32_t* y_in;  // [B][T]            (teacher forcing)
  int32_t* y_out;       // [B][T]            (generation)
  float* logits;        // [B][T][A]         (teacher forcing)
  int B, T, reset, init_sample;
  // how a step's distribution becomes its sample (generation): wn_sample_mode_t, 1 / temperature,
  // k of top-k sampling
  int smode;
  float inv_t;
  int top_k;
  // host-requested abort (wn_abort): a word in coherent pinned host memory, read with system-scope
  // loads every WN_ABORT_CHECK steps of a call; nonzero = stop
  const int* abort_flag;
};
// Steps between two reads of the abort word (a read crosses PCIe: ~1-2 us)
#define WN_ABORT_CHECK 64

// Caller-owned workspace, carved by the host code.
struct WnWorkspace {
  int32_t* status;      // one word
  int64_t* state;       // [B][WN_STATE_WORDS]
  float* hist;          // [B][hist_len]
};

struct WnStreamArgs {
  WnDims d;
  WnDevWeights w;
  WnIO io;
  WnWorkspace ws;
};

#define WN_MAX_CHAIN 32   // chain CUs of one replica of the multi-CU kernel
#define WN_CHAIN_GRID 256 // blocks of the multi-CU kernel (one per CU)
#define WN_CHAIN_MAX_G 16 // streams one replica interleaves
#define WN_CHAIN_MAP_WORDS (WN_CHAIN_GRID + 2)  // launch-time block -> XCD map and grid-barrier words

// Multi-CU kernel: tagged 64-bit words (value | step + 1 << 32).  The roles (chain, head and aux
// CUs) form a replica; nrep replicas run side by side, replica k serving streams
// [k G, min(B, (k + 1) G)), each interleaving its streams step by step.
struct WnChainArgs {
  WnDims d;
  WnDevWeights w;
  WnIO io;
  int32_t* status;
  int64_t* state;                // [B][WN_STATE_WORDS]
  unsigned long long* ring;      // [B][hist_len] tagged dilation histories
  unsigned long long* mb;        // [B][mb_words] mailboxes, placed after the histories
  long long mb_words;            // words of one stream's mailbox block
  // after the mailboxes: the XCD each block of this launch runs on ([WN_CHAIN_GRID] words), then a
  // grid barrier's arrival count and generation (2 words); cleared with the histories on a reset
  unsigned long long* xmap;
  int n_active;                  // blocks with a role (they meet at the grid barrier)
  // word offsets inside a stream's block: pre-activations [L][2][2R] (aux -> chain) at 0,
  // hidden states [L][2][R] (chain -> aux), skip partials [naux][2][S] (aux -> head),
  // layer-run outputs [nch][2][R] (chain -> next chain), partial logits [4][2][A]
  // (head -> chain CU 0), last layer's skip projection [2][S] (last chain CU -> head)
  int off_h, off_q, off_x, off_logit, off_qtail;
  int nch;                       // chain CUs per replica
  int layer_begin[WN_MAX_CHAIN + 1];
  int spin_limit;                // polls before a wait gives up with WN_ETIMEOUT
  int nrep, G;                   // replicas, streams per replica
  int ub;                        // steps of uniforms / samples staged in LDS per stream
  int tail_on_chain;             // 1: the last chain CU computes the last layer's skip projection
  int nla, naux, naux_q;         // layers per aux CU, aux CUs per replica, aux CUs posting a skip partial
  int local_posts;               // 1: posts to a reader on the same XCD stop at its L2
  int pair;                      // MFMA kernel: 1 = paired columns (8 streams per replica), 0 = 16 streams
  int aux_begin[WN_MAX_LAYERS + 1];  // MFMA kernel: first layer of each aux CU (then L)
  uint16_t role_of_block[WN_CHAIN_GRID];  // replica * per_replica + role; 0xffff = idle block
};

// How the multi-CU kernel lays out a model and a batch over the chip.
struct WnChainPlan {
  int nch, nrep, G, ub, tail_on_chain, pair;
  int nla, naux, naux_q;
  int layer_begin[WN_MAX_CHAIN + 1];
  int aux_begin[WN_MAX_LAYERS + 1];
  uint16_t role_of_block[WN_CHAIN_GRID];
  long long mb_words;
  int off_h, off_q, off_x, off_logit, off_qtail;
};

// Kernel families.  Each returns hipSuccess or the launch error.
bool wn_stream_supported(int R, int S);
hipError_t wn_stream_launch(const WnStreamArgs& args, bool teacher, hipStream_t stream);

bool wn_chain_supported(int R, int S, int L);
// Fills *p for B streams; false if the kernel cannot serve them (too many streams per replica,
// or a layout that does not fit).
bool wn_chain_plan(int L, int R, int S, int B, bool two_taps, WnChainPlan* p);
hipError_t wn_chain_reset(unsigned long long* words, size_t n, int* status, hipStream_t stream);
// Zeroes the status word before a run from zero of the per-stream or batched kernel (a kernel, not
// a memset: a caller may capture the call in a graph).
hipError_t wn_status_clear(int* status, hipStream_t stream);
// True when block b of a cooperative launch of the kernel's grid runs on XCD b mod 8 on the
// current device (checked with a probe launch), the layout the placement assumes.
bool wn_chain_xcd_map_ok();
hipError_t wn_chain_launch(const WnChainArgs& g, bool teacher, hipStream_t stream);

// Multi-CU kernel for bf16 and int8 models (r = 64): the chain kernel's roles on MFMA, 8 streams
// per replica in paired columns (hi and lo parts of a stream in two columns of a 16 x 16 tile) or 16
// streams, one per column.  Same argument block and workspace words as the chain kernel (mailbox
// offsets from wn_mchain_plan; the histories hold hist_len * wn_mchain_columns(plan) words per
// replica).
bool wn_mchain_supported(int R, int S, int L);
bool wn_mchain_plan(int L, int R, int S, int B, WnChainPlan* p);
int wn_mchain_columns(const WnChainPlan& p);
hipError_t wn_mchain_launch(const WnChainArgs& g, bool teacher, hipStream_t stream);

// Batched kernel for bf16 weights: one workgroup per group of 8 or 16 streams, MFMA for every
// product, weights pre-packed into MFMA operand tiles (wn_group_pack) and streamed from L2.
struct WnGroupArgs {
  WnDims d;
  WnDevWeights w;     // biases and the embedding (bf16) are read from here
  const void* packed; // tiles from wn_group_pack, device copy
  WnIO io;
  WnWorkspace ws;     // same layout as the per-stream kernel's
  int gs;             // streams per workgroup: 8 or 16 (wn_group_streams)
};
#define WN_GROUP_MAX_LAYERS 40
// Streams per workgroup for a call with B streams: 8 while that keeps one workgroup per CU, else
// 16; the environment variable WN_GROUP_STREAMS (8 or 16) overrides it.
int wn_group_streams(int B);
bool wn_group_supported(int R, int S, int L);
size_t wn_group_lds_bytes(int L, int S, bool two_taps);
// Packs W_prev/W_cur/W_res/W_skip of every layer and the two head matrices (fp32 host arrays
// in the wn_weights layout) into bf16 tiles, the order the kernel streams them in.
std::vector<uint16_t> wn_group_pack(int L, int R, int S, const float* w_prev, const float* w_cur,
                                    const float* w_res, const float* w_skip, const float* w_relu,
                                    const float* w_out);
hipError_t wn_group_launch(const WnGroupArgs& g, bool teacher, hipStream_t stream);

// The calling thread's last-error detail (wn_last_error): set it and return `code`, or clear it.
int wn_set_last_error(int code, const char* msg);
void wn_clear_last_error();

// fp32 -> bf16 bit pattern, round to nearest even (NaN stays NaN).
uint16_t wn_to_bf16(float f);
