/*
 * spectrain.h - C ABI of one SpecTrain pipeline stage on an MI355X (gfx950).
 *
 * SpecTrain (Chen, Yang, Cheng: "Efficient and Robust Parallel DNN Training
 * through Model Parallelism on Multi-GPU Platform") runs each pipeline stage's
 * forward and backward pass against weights predicted for the moment the
 * mini-batch completes its round trip (Section 3.2):
 *
 *   Eq. 1  v_t = gamma * v_{t-1} + (1 - gamma) * g_t          smoothed gradient
 *          W_{t+1} = W_t - eta * v_t                          momentum update
 *   Eq. 4  What_{t+s} = W_t - s * eta * v_{t-1}               s-step prediction
 *   Eq. 5  s = floor(k/2) + N - k - 1                          forward pass, stage k of N
 *   Eq. 6  s = floor(k/2)                                      backward pass
 *
 * A stage owns its master weights W, smoothed gradient v and gradient g (all
 * float32, one flat arena each), two predicted-weight buffers in the compute
 * dtype (slot 0 for the next forward, slot 1 for the next backward) and a ring
 * of activation stashes, one per mini-batch in flight (at most N - k in the
 * one-forward-one-backward order of Section 3.1).
 *
 * Conventions for every function below:
 *  - The return value is a status code (SPECTRAIN_OK = 0). No function throws
 *    or aborts; on failure spectrain_last_error() describes the cause.
 *  - Device work is enqueued asynchronously on the HIP stream given to
 *    spectrain_stage_create, in call order. Only the functions documented as
 *    synchronising wait for it.
 *  - "device pointer" arguments point to GPU memory owned by the caller; the
 *    library never frees them. Host pointers are only read during the call.
 *  - A stage handle may be used from one host thread at a time.
 *
 * Parameter order (the flat float32 array that crosses this boundary), per
 * kind, repeated per layer l = 0 .. num_layers-1:
 *   FC          weight [out, in] row-major, bias [out]
 *   CONV3X3     filter [C_out, 3, 3, C_in]                  (no bias)
 *   BOTTLENECK  conv1 [C_mid,1,1,C], conv2 [C_mid,3,3,C_mid], conv3 [C,1,1,C_mid]
 *               (both: then, with a CE head, head.weight [classes, channels of the
 *               stage output], head.bias [classes])
 *   TRANSFORMER qkv.weight [3d, d], qkv.bias [3d], out.weight [d, d], out.bias [d],
 *               ln1.weight [d], ln1.bias [d], ffn1.weight [F, d], ffn1.bias [F],
 *               ffn2.weight [d, F], ffn2.bias [d], ln2.weight [d], ln2.bias [d];
 *               then, with a CE head, vocab.weight [V, d], vocab.bias [V]
 *   RESLSTM     weight_x [4H, I], weight_h [4H, H], bias [4H], gate blocks (i, f, g, o);
 *               then, with a CE head, vocab.weight [V, H], vocab.bias [V]
 *
 * Activation layouts (compute dtype; bf16 is stored as raw 16-bit bf16):
 *   FC [B, features]; CONV3X3 and BOTTLENECK NHWC [B, H, W, C];
 *   TRANSFORMER [B, S, d]; RESLSTM time-major [T, B, H]; labels int32
 *   [B] (FC, CONV3X3, BOTTLENECK), [B, S] (TRANSFORMER, one target per token)
 *   or [T, B] (RESLSTM)
 *   with values in [0, classes); a label outside that range makes the
 *   reported loss NaN.
 */
#ifndef SPECTRAIN_H
#define SPECTRAIN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPECTRAIN_ABI_VERSION 3u

/* Status codes. */
enum {
  SPECTRAIN_OK = 0,
  SPECTRAIN_EINVAL = 1,     /* bad argument or descriptor */
  SPECTRAIN_ENOMEM = 2,     /* device allocation failed */
  SPECTRAIN_EHIP = 3,       /* a HIP runtime call failed; message carries its error string */
  SPECTRAIN_ESTATE = 4,     /* call out of order for the stage's current state */
  SPECTRAIN_ENONFINITE = 5  /* the last update produced a non-finite W or v */
};

typedef struct spectrain_stage* spectrain_stage_t;   /* opaque, owned by the library */

typedef enum { SPECTRAIN_FP32 = 0, SPECTRAIN_BF16 = 1 } spectrain_dtype;

typedef enum {
  SPECTRAIN_KIND_FC = 0,           /* dims: in, out, hidden; widths in, hidden x (L-1), out */
  SPECTRAIN_KIND_CONV3X3 = 1,      /* dims: C_in, C_out, H, W[, classes]; 3x3 stride 1 pad 1, ReLU */
  SPECTRAIN_KIND_BOTTLENECK = 2,   /* dims: C, C_mid, H, W[, classes]; 1x1-3x3-1x1, identity skip, ReLU */
  SPECTRAIN_KIND_TRANSFORMER = 3,  /* dims: d_model, heads, ffn, seq[, vocab with a CE head]; post-LN encoder layer */
  SPECTRAIN_KIND_RESLSTM = 4       /* dims: input, hidden, T, vocab; residual LSTM layers */
} spectrain_kind;

typedef enum {
  SPECTRAIN_HEAD_NONE = 0,  /* the caller passes dL/dY to backward */
  SPECTRAIN_HEAD_CE = 1     /* mean softmax cross-entropy over rows; caller passes int32 labels.
                               CONV3X3 and BOTTLENECK score the global average over H x W of the
                               stage output with a linear classifier (an even number of classes) */
} spectrain_head;

/* Which weights the backward pass of a mini-batch uses (Section 4.2 compares
 * the three ways a pipeline stage can treat weight staleness):
 *   PREDICT - the backward-predicted slot 1 (SpecTrain, s from Eq. 6; with
 *             s = 0 for both passes this is the unmitigated pipeline, the
 *             paper's Vanilla model parallelism);
 *   STASH   - the weights its own forward pass used (weight stashing, as in
 *             PipeDream, Section 3.2): every forward copies slot 0 into a ring
 *             of N - k weight versions, one per mini-batch in flight, and the
 *             matching backward reads that copy. The caller passes s = 0 to
 *             the update so that each forward sees the latest weights. */
typedef enum { SPECTRAIN_POLICY_PREDICT = 0, SPECTRAIN_POLICY_STASH = 1 } spectrain_weight_policy;

typedef struct {
  uint32_t abi_version;     /* SPECTRAIN_ABI_VERSION */
  int32_t kind;             /* spectrain_kind */
  int32_t dtype;            /* spectrain_dtype: operand/activation format; W, v, g are float32 */
  int32_t head;             /* spectrain_head */
  int32_t stage_index;      /* k, 0-based, 0 <= k < num_stages */
  int32_t num_stages;       /* N >= 1 */
  int32_t batch;            /* mini-batch size B >= 1 */
  int32_t num_layers;       /* L >= 1 (layers, blocks or LSTM layers) */
  int32_t dims[8];          /* kind-specific, see spectrain_kind; unused entries 0 */
  float lr;                 /* eta > 0 */
  float momentum;           /* gamma, 0 < gamma <= 1 */
  int32_t weight_policy;    /* spectrain_weight_policy */
} spectrain_stage_desc;

/* Eq. 5 (is_forward != 0) or Eq. 6: version difference s for stage k of N.
 * Returns s >= 0, or -1 when k < 0, k >= N or N < 1. */
int32_t spectrain_version_difference(int32_t k, int32_t N, int32_t is_forward);

/* Create a stage. W0_host: n_params float32 values in the parameter order
 * above (n_params must equal the kind's count, else EINVAL). hip_stream: a
 * hipStream_t (NULL = the null stream) on the current device; all of the
 * stage's device work runs on it. v starts at 0, so both predicted slots start
 * equal to W0 (Eq. 4 with v = 0). Device dims that the kernels need to be
 * multiples of 8 (bf16 channel/feature counts) are checked here (EINVAL).
 * Every device buffer the stage uses is allocated here: the arenas, the
 * stash ring, the workspace and a second workspace copy (for the forward of
 * spectrain_stage_forward_backward), and two streams of the stage's own
 * (default priority: weight gradients, and that forward). Synchronises the
 * stream before returning. */
int spectrain_stage_create(const spectrain_stage_desc* desc, const float* W0_host, size_t n_params,
                           void* hip_stream, spectrain_stage_t* out);

/* Number of parameters of the stage (the length of the flat arrays). */
int spectrain_stage_num_params(spectrain_stage_t st, size_t* n);

/* Eq. 4 for one slot: What_slot = W - s * eta * v, rounded to the compute
 * dtype. slot 0 feeds the next forward, slot 1 the next backward. EINVAL for
 * s < 0 or a bad slot. */
int spectrain_stage_predict(spectrain_stage_t st, int32_t s, int32_t slot);

/* Forward pass of mini-batch mb_id against slot 0, the weights predicted with
 * the forward version difference (Section 3.2: a pass runs on the weights
 * predicted for the time its mini-batch completes its round trip, Eq. 4 with
 * Eq. 5); with STASH, slot 0 is also copied into the mini-batch's weight
 * stash. The activations the backward pass needs are kept in the stage's
 * stash until then (Section 3.1: up to N - k mini-batches are in flight at
 * stage k). x_dev: input activations.
 * y_dev: output activations (HEAD_NONE; NULL with a CE head). labels_dev and
 * loss_dev (one float32, the mean CE) are used with a CE head only. The stage
 * keeps references to x_dev and y_dev until the matching backward returns:
 * the caller must keep them alive and unmodified until then. ESTATE when
 * N - k mini-batches are already in flight or mb_id is already in flight. */
int spectrain_stage_forward(spectrain_stage_t st, int64_t mb_id, const void* x_dev, void* y_dev,
                            const int32_t* labels_dev, float* loss_dev);

/* Backward pass of mini-batch mb_id against slot 1 (PREDICT: the weights
 * predicted with the backward version difference, Eq. 4 with Eq. 6, Section
 * 3.2) or the weights its forward used (STASH) for dX, and the stashed
 * activations for g (one gradient per backward, which the next update
 * applies, Section 3.1). dy_dev: dL/dY (HEAD_NONE; ignored with a CE head).
 * dx_dev: dL/dX output, or NULL to skip it (e.g. at k = 0). Overwrites g with
 * this mini-batch's gradient and frees its stash slot. ESTATE when mb_id is
 * not in flight or a previous gradient is still waiting for its update. */
int spectrain_stage_backward(spectrain_stage_t st, int64_t mb_id, const void* dy_dev, void* dx_dev);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * backward pass above, identical in arguments, state rules and results
 * (bitwise), whose split-K partial planes live in the library's per-device
 * scratch array instead of the stage's workspace (one half for the stage's
 * stream, one for the stream its weight gradients run on). The call
 * allocates and frees nothing; the array (128 MiB,
 * SPECTRAIN_NOALLOC_SCRATCH_BYTES) is held
 * by every GPU the library runs on until the process ends, and its address
 * is looked up on the first such call on a device. EINVAL when the stage's
 * split-K workspaces exceed the array. Every call on one GPU shares that
 * GPU's array, and the array keeps the last call's contents (every partial
 * a call reads it first writes, so nothing needs clearing): calls that
 * overlap on one GPU, on different streams, race. */
#define SPECTRAIN_NOALLOC_SCRATCH_BYTES (128u << 20)
int spectrain_stage_backward_noalloc(spectrain_stage_t st, int64_t mb_id, const void* dy_dev, void* dx_dev);

/* The forward of mb_fwd followed by the backward of mb_bwd, with the effect
 * of spectrain_stage_forward then spectrain_stage_backward (same arguments,
 * state rules and results, bitwise), the two passes running concurrently on
 * the GPU. In the one-forward-one-backward order of Section 3.1 a stage's
 * forward is followed by a backward with no update between them, so both
 * passes read weights of the same version (slot 0 and slot 1 as refreshed by
 * the last update, or the mini-batch's weight stash) and neither writes what
 * the other reads. The forward runs on a stream of the stage's own (default
 * priority) against a second copy of the stage's workspace, both made by
 * spectrain_stage_create, so the call allocates nothing and can be captured
 * in a HIP graph; the backward runs as spectrain_stage_backward does, and
 * work enqueued later on the stage's stream waits for both.
 * ESTATE, with nothing enqueued, when mb_fwd == mb_bwd, mb_fwd is in flight,
 * no stash slot is free (always so at the last stage, k = N - 1, whose
 * forward is the one its backward needs), mb_bwd is not in flight or a
 * gradient still waits for its update; EINVAL for a NULL x_dev, for a NULL
 * y_dev or dy_dev without a CE head, or a CE head without labels_dev and
 * loss_dev. */
int spectrain_stage_forward_backward(spectrain_stage_t st, int64_t mb_fwd, const void* x_dev, void* y_dev,
                                     const int32_t* labels_dev, float* loss_dev, int64_t mb_bwd, const void* dy_dev,
                                     void* dx_dev);

/* One fused pass over the arenas: Eq. 1, W <- W - eta v, then Eq. 4 for both
 * slots (slot 0 with s_next_fwd, slot 1 with s_next_bwd; a negative s leaves
 * that slot unchanged). ESTATE unless a backward produced g since the last
 * update. A non-finite W or v element raises a flag that makes the next call
 * on the stage return ENONFINITE. */
int spectrain_stage_update(spectrain_stage_t st, int32_t s_next_fwd, int32_t s_next_bwd);

/* Copy W and v (float32, parameter order) to host buffers of n_params values.
 * Either pointer may be NULL. Synchronises the stream. */
int spectrain_stage_get_state(spectrain_stage_t st, float* W_host, float* v_host);

/* Replace W and v (host float32, parameter order; v may be NULL for zero) and
 * re-predict both slots with s = 0. ESTATE while any mini-batch is in flight.
 * Synchronises the stream. */
int spectrain_stage_set_state(spectrain_stage_t st, const float* W_host, const float* v_host);

/* Copy a predicted slot (0 or 1), converted to float32, to the host.
 * Synchronises the stream. */
int spectrain_stage_get_predicted(spectrain_stage_t st, int32_t slot, float* What_host);

/* Per-kernel launch statistics of a stage, collected between
 * spectrain_stage_profile(st, 1 or 2) and a read. Durations come from HIP
 * events recorded around every launch on the stream it runs on (use a
 * separate pass, not the timed one). With enable == 2 every launch of the
 * stage, including the weight gradients and the forward of
 * spectrain_stage_forward_backward, is issued on the stage's stream, one at
 * a time, with the kernels and launch shapes of the concurrent call: each
 * duration is then the launch's own, not shared with launches of the other
 * streams. flops and bytes are the
 * algorithmic work of the launches: 2*M*N*K per GEMM (3x3 convolutions count
 * all 9 taps); for a GEMM each operand tensor read once (a convolution's
 * feature map once, not once per tap), each output written once and each
 * epilogue operand (bias, residual, ReLU mask) read once; for the fused
 * update 12 bytes read plus 8 + 2*sizeof(operand) written per parameter
 * (24 bytes for bf16 stages); one read of each input and one write of each
 * output for the elementwise and row passes. extra_bytes_total counts what a
 * launch moves beyond that by construction: the float32 K-slice partials of
 * a split GEMM, and the partial planes the update reads in place of g. */
typedef struct {
  char name[48];        /* kernel family: the kernel's name with its template arguments as a profiler
                           lists it (e.g. "gemm_bf16_kernel<0, 3, false, 128, 1>"), or a pass name
                           such as "fused_update", "layernorm_bwd", "lstm_step" */
  int64_t launches;
  double ms_total;      /* summed event-to-event duration */
  double flops_total;   /* algorithmic floating-point operations (0 if not a contraction) */
  double bytes_total;   /* algorithmic HBM bytes (0 if not counted) */
  double extra_bytes_total;   /* bytes beyond the algorithmic ones (split-K partial planes) */
} spectrain_kernel_stat;

/* enable 1 or 2: clear the statistics and time every following launch (2:
 * with every launch issued on the stage's stream, see above); enable == 0:
 * stop timing (statistics are kept for reading). EINVAL for other values. */
int spectrain_stage_profile(spectrain_stage_t st, int32_t enable);

/* Copy up to capacity kernel families into out (in first-launch order) and
 * store the number of families in *count. Synchronises the stream. */
int spectrain_stage_profile_read(spectrain_stage_t st, spectrain_kernel_stat* out, int32_t capacity,
                                 int32_t* count);

/* Copy activation buffer `index` that the forward pass of mini-batch mb_id
 * stored for its backward pass (the stash of Section 3.1, one per mini-batch
 * in flight) to host_out, for inspection and testing. *size receives the
 * buffer's size in bytes (0: the index is unused by this stage); with
 * host_out NULL nothing is copied. EINVAL for an index outside the kind's
 * list or a capacity below the size; ESTATE when mb_id is not in flight.
 * Synchronises the stream. Buffers are row-major in the activation layouts
 * above, in the compute dtype unless marked f32; P = B*H*W pixels, T = B*S
 * tokens (transformer) or T*B steps x rows (LSTM):
 *   FC          l-1: output of layer l-1 [B, hidden] (l = 1 .. L-1);
 *               L-1 with a CE head: dlogits [B, classes]
 *   CONV3X3     l-1: output of layer l-1 [P, C_out] (l = 1 .. L-1); with a CE head
 *               L-1: last output, L: pooled [B, C_out] (bf16), L+1: dlogits [B, classes] (bf16)
 *   BOTTLENECK  3l: t1 [P, C_mid], 3l+1: t2 [P, C_mid], 3l+2: block output [P, C]
 *               (l < L-1, or every block with a CE head); 3L: pooled [B, C], 3L+1: dlogits
 *   TRANSFORMER 13l+j: 0 qkv [T, 3d], 1 softmax row statistics (max, 1/sum) f32 [B*heads*S, 2]
 *               (sequence 128, head dimension 64) or probabilities f32 [B*heads, S, S],
 *               2 probabilities bf16 (the second form only), 3 ctx [T, d], 4 r1 = x + attention
 *               output [T, d], 5 mean of r1 f32 [T], 6 1/std of r1 f32 [T], 7 h = LN1(r1) [T, d],
 *               8 ReLU(FFN1) [T, F], 9 r2 = h + FFN2 [T, d], 10 mean of r2 f32, 11 1/std of r2 f32,
 *               12 layer output [T, d] (l < L-1, or every layer with a CE head);
 *               13L with a CE head: dlogits [T, V]
 *   RESLSTM     4l+j: 0 activated gates (i, f, g, o) f32 [T, B, 4H], 1 cell state c f32 [T, B, H],
 *               2 h [T, B, H], 3 layer output [T, B, H] (l < L-1, or every layer with a CE head);
 *               4L with a CE head: dlogits [T*B, V] */
int spectrain_stage_read_stash(spectrain_stage_t st, int64_t mb_id, int32_t index, void* host_out, size_t capacity,
                               size_t* size);

/* Release every device buffer of the stage. Synchronises the stream.
 * Passing NULL returns EINVAL. */
int spectrain_stage_destroy(spectrain_stage_t st);

/* Message of the last failed call on this host thread ("" if none). */
const char* spectrain_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SPECTRAIN_H */
