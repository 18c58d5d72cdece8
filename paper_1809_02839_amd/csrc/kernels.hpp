// Kernel launchers of the SpecTrain stage library. Every launcher enqueues
// on the given stream and returns hipSuccess or the launch error.
#pragma once

#include "common.hpp"

namespace spx {

// ---------------------------------------------------------------- GEMM ----
// C[m, n] = sum_k A(m, k) * B(n, k), float32 accumulation, M x N x K, with an
// optional batch over blockIdx.z. Operands are described by an access mode:
//   K-modes deliver 8 consecutive k of one row (16-byte loads),
//   R-modes deliver 8 consecutive rows of one k (16-byte loads, transposed on
//   the way into LDS).
enum OperandMode : int {
  OP_K_PLAIN = 0,      // X[r * ld + k]
  OP_K_CONV_FWD = 1,   // im2col of an NHWC map: k = tap * C + c, source pixel p + (kh-1, kw-1)
  OP_K_CONV_DGRAD = 2, // im2col for the data gradient: k = tap * C + c, source pixel p - (kh-1, kw-1)
  OP_R_PLAIN = 3,      // X[k * ld + r]
  OP_R_CONV_WGRAD = 4, // rows r = tap * C + c, k = pixel: X[pixel + (kh-1, kw-1)][c]
  OP_R_FILTER_T = 5,   // filter [C2][3][3][C] read as rows r = c, k = tap * C2 + c2
};

struct ConvGeom {
  int B = 0, H = 0, W = 0;
  int C = 0;    // channels of the gathered tensor (for FILTER_T: C_in, the row count)
  int C2 = 0;   // FILTER_T only: C_out
};

struct Operand {
  const void* ptr = nullptr;   // bf16 (or float32 for the float32 GEMM)
  long ld = 0;
  long extent = 0;             // elements addressable from ptr (batch 0); reads beyond it return 0
  long bs1 = 0, bs2 = 0;       // batch strides (elements) for z / zdiv and z % zdiv
  int mode = OP_K_PLAIN;
  ConvGeom g;
};

struct Epilogue {
  float* out_f32 = nullptr;        // value stored (or added, if accumulate) as float32
  bf16_t* out_bf16 = nullptr;      // value rounded to bf16 and stored
  long ldc = 0;
  long bs1 = 0, bs2 = 0;           // batch strides of every [M, N] tensor below
  const float* bias = nullptr;     // [N], added
  const bf16_t* bias_bf16 = nullptr;  // [N], added (bf16 GEMM only)
  const float* res_f32 = nullptr;  // [M, N] with ldc, added
  const bf16_t* res_bf16 = nullptr;// [M, N] with ldc, added
  const void* mask = nullptr;      // [M, N] with ldc: value zeroed where mask <= 0 (bf16 or f32 per GEMM dtype)
  float alpha = 1.0f;              // scales the accumulator before everything else
  int relu = 0;
  int accumulate = 0;              // out_f32 += value
};

struct GemmDesc {
  int M = 0, N = 0, K = 0;
  int batch = 1, zdiv = 1;
  float* workspace = nullptr;      // split-K partials (bf16 GEMM); NULL disables splitting
  size_t workspace_bytes = 0;
  bool concurrent = false;         // launched beside another pass's launches (selects the tile rule)
  Operand A, B;
  Epilogue epi;
};

// bf16 GEMM in up to two launches: the tiled MFMA kernel (GEMM_MAIN) and,
// when K is split across blocks, the ordered reduction of the float32
// partials through the epilogue (GEMM_REDUCE).
enum { GEMM_MAIN = 1, GEMM_REDUCE = 2, GEMM_ALL = 3 };
hipError_t gemm_bf16(const GemmDesc& d, hipStream_t s, int phases = GEMM_ALL);
int gemm_bf16_splits(const GemmDesc& d);   // K splits the launch will use (1 = none)
// The same count from the shape alone, for a workspace of workspace_bytes.
int gemm_bf16_split_rule(int M, int N, int K, int batch, size_t workspace_bytes, bool concurrent);
hipError_t gemm_f32(const GemmDesc& d, hipStream_t s);
// Names of the kernels a launch runs, as a profiler lists the instantiations
// (e.g. "gemm_bf16_kernel<0, 3, false, 128, 1>"); the returned buffer is
// thread-local and valid until the next call on the thread.
const char* gemm_bf16_kernel_name(const GemmDesc& d);
const char* gemm_bf16_reduce_name(const GemmDesc& d);
const char* gemm_f32_kernel_name(const GemmDesc& d);

// Global average pool of an NHWC bf16 tensor [B, HW, C] -> [B, C] (bf16 of the
// float32 mean), and its backward through the ReLU of the pooled tensor y:
// dx = y > 0 ? bf16(dpool / HW) : 0 (C % 8 == 0, 16-byte aligned tensors).
hipError_t avgpool_fwd(const bf16_t* x, int B, int HW, int C, bf16_t* out, hipStream_t s);
hipError_t avgpool_bwd_mask(const bf16_t* dpool, const bf16_t* y, int B, int HW, int C, bf16_t* dx, hipStream_t s);

// ------------------------------------------------------- update/predict ----
// Fused Eq. 1 + momentum update + Eq. 4 for two slots over n float32 values.
// what_dtype: 0 float32, 1 bf16. s < 0 skips a slot. flag is set to 1 when a
// non-finite W or v is produced.
hipError_t fused_update(float* W, float* v, const float* g, void* what_f, void* what_b, int what_dtype,
                        long n, float lr, float gamma, int s_f, int s_b, int* flag, hipStream_t s);
hipError_t predict_slot(const float* W, const float* v, void* what, int what_dtype, long n, float lr, int s_pred,
                        hipStream_t s);

// The same update with the gradient of some tensors still in split-K form:
// segment i covers arena elements [off, off + n) whose gradient is the sum,
// in split order, of `splits` float32 planes part[s * n + j] (the K-slice
// partials of the filter-gradient GEMM, row-major like the tensor). Elements
// outside every segment read g. Offsets and lengths are multiples of 8;
// segments are sorted and disjoint. The sum is the one the split-K reduction
// forms, so W, v and both slots are bitwise those of reduce-then-update.
constexpr int UPDATE_MAX_SEGMENTS = 24;
struct UpdateSegment {
  long off = 0, n = 0;
  const float* part = nullptr;
  int splits = 0;
};
hipError_t fused_update_partials(float* W, float* v, const float* g, const UpdateSegment* segs, int nsegs,
                                 void* what_f, void* what_b, int what_dtype, long n, float lr, float gamma, int s_f,
                                 int s_b, int* flag, hipStream_t s);

// Fused residual-LSTM recurrence steps (supported for B <= 64 and H a
// multiple of 32): forward z_t = zx_t + h_{t-1} W_h^T and the cell in one
// launch; backward dh_t = dh_out_t + dz_{t+1} W_h (W_h^T given) and the cell
// backward in one launch. Null h_prev / dz_next / c_prev mark the first step.
bool lstm_step_supported(int B, int H);
hipError_t lstm_step_fwd(const float* zx_t, const bf16_t* h_prev, const bf16_t* Wh, const float* c_prev, int B, int H,
                         float* gates_t, float* c_t, bf16_t* h_t, hipStream_t s);
hipError_t lstm_step_bwd(const bf16_t* dz_next, const bf16_t* WhT, const bf16_t* dh_out, const float* gates_t,
                         const float* c_t, const float* c_prev, int B, int H, float* dc, bf16_t* dz_t, hipStream_t s);
hipError_t transpose_bf16(const bf16_t* X, int R, int C, bf16_t* Y, hipStream_t s);   // R, C multiples of 32

// Fused attention core for sequence length 128 and head dimension 64 (one
// block per batch x head), on the packed qkv [B*S][3d] of a layer. Forward
// writes ctx [B*S][d] and the softmax row statistics (max, 1/sum) as float32
// [B*heads*S][2]; backward recomputes P from them and writes dQ, dK, dV into
// dqkv [B*S][3d]. Other shapes use the batched GEMM path.
bool attention_fused_supported(int seq, int head_dim, int d);
hipError_t attention_fwd(const bf16_t* qkv, int batch, int heads, int d, float scale, float* stats, bf16_t* ctx,
                         hipStream_t s);
hipError_t attention_bwd(const bf16_t* qkv, const bf16_t* dctx, const float* stats, int batch, int heads, int d,
                         float scale, bf16_t* dqkv, hipStream_t s);

// Row chunking of the two-pass column reductions (column sums, layer-norm
// parameter gradients) and the float32 workspace each pass needs.
constexpr int COLSUM_ROWS = 64;   // rows summed per block in the first pass
constexpr int LNB_ROWS = 16;      // rows per block of the layer-norm backward
inline long column_sum_ws_floats(long rows, long cols) { return ((rows + COLSUM_ROWS - 1) / COLSUM_ROWS) * cols; }
inline long layernorm_bwd_ws_floats(long rows, long d) { return 3 * ((rows + LNB_ROWS - 1) / LNB_ROWS) * d; }

// ------------------------------------------------------------ elementwise ----
// dst[i] = src[i] * (mask[i] > 0), bf16 (dtype 1) or float32 (dtype 0).
hipError_t mask_relu_grad(const void* src, const void* mask, void* dst, long n, int dtype, hipStream_t s);
// Wt [Ci][9][Co] from each 3x3 filter W [Co][9][Ci] of up to MAX layers, one
// launch (bf16; Co and every Ci multiples of 8).
struct FilterBatch {
  static constexpr int MAX = 16;
  const bf16_t* W[MAX];
  bf16_t* Wt[MAX];
  int Ci[MAX];
  int n, Co;
};
hipError_t filter_transpose_bf16(const FilterBatch& fb, hipStream_t s);
// out[c] (=|+=) sum over rows r of X[r * ld + c], X bf16 or float32; deterministic.
hipError_t column_sum(const void* X, int dtype, long rows, int cols, long ld, float* out, int accumulate,
                      float* partial_ws, hipStream_t s);
// Mean softmax cross-entropy over rows of float32 logits [R, C]; writes the
// mean loss to loss (one float) and dlogits = (softmax - onehot) / R in dtype.
hipError_t softmax_ce(const float* logits, const int32_t* labels, int R, int C, void* dlogits, int dtype,
                      float* loss, float* row_loss_ws, hipStream_t s);
// Layer norm over rows of bf16 r [R, D]: y = bf16(gamma * xhat + beta) with
// bf16 gamma/beta; stats mean and rstd (float32) are written per row.
hipError_t layernorm_fwd(const bf16_t* r, const bf16_t* gamma, const bf16_t* beta, int R, int D, float eps,
                         bf16_t* y, float* mean, float* rstd, hipStream_t s);
// Layer-norm backward for bf16 dy: dr = bf16(...); dgamma/dbeta (float32,
// overwritten) reduced over rows deterministically. dsum (may be null): the
// column sums of the stored dr as well (the bias gradient of the linear layer
// that produced the normalised sum); when dsum, dgamma, dbeta are adjacent
// D-float ranges one final reduction writes all three.
hipError_t layernorm_bwd(const bf16_t* dy, const bf16_t* r, const float* mean, const float* rstd,
                         const bf16_t* gamma, int R, int D, bf16_t* dr, float* dgamma, float* dbeta, float* dsum,
                         float* partial_ws, hipStream_t s);
// The same in two launches: the rows (dr and the per-block partials in
// partial_ws), then the reduction of the partials into dgamma, dbeta and dsum
// (which may be on another stream once the first has completed).
hipError_t layernorm_bwd_rows(const bf16_t* dy, const bf16_t* r, const float* mean, const float* rstd,
                              const bf16_t* gamma, int R, int D, bf16_t* dr, float* partial_ws, hipStream_t s);
hipError_t layernorm_bwd_params(const float* partial_ws, int R, int D, float* dgamma, float* dbeta, float* dsum,
                                hipStream_t s);
// Row softmax of float32 scores [R, C] -> P float32 and bf16(P).
hipError_t softmax_rows(const float* S, int R, int C, float* P, bf16_t* Pb, hipStream_t s);
// Softmax backward: dS = bf16(P * (dP - sum_j P dP)) per row.
hipError_t softmax_bwd(const float* P, const float* dP, int R, int C, bf16_t* dS, hipStream_t s);
// LSTM cell for one time step: z [B, 4H] float32 pre-activations (i, f, g, o)
// -> gates (activated, float32), c_t, h_t = bf16(o * tanh(c_t)).
hipError_t lstm_cell_fwd(const float* z, const float* c_prev, int B, int H, float* gates, float* c,
                         bf16_t* h, hipStream_t s);
// LSTM cell backward for one step: dh = dh_out + dh_rec; writes dz (bf16) and
// carries dc (in/out, float32).
hipError_t lstm_cell_bwd(const bf16_t* dh_out, const float* dh_rec, const float* gates, const float* c,
                         const float* c_prev, int B, int H, float* dc, bf16_t* dz, hipStream_t s);
// out = bf16(a + b) elementwise (bf16 inputs).
hipError_t add_bf16(const bf16_t* a, const bf16_t* b, bf16_t* out, long n, hipStream_t s);
// float32 <-> bf16 conversions.
hipError_t cast_f32_to_bf16(const float* x, bf16_t* y, long n, hipStream_t s);
hipError_t cast_bf16_to_f32(const bf16_t* x, float* y, long n, hipStream_t s);
hipError_t fill_f32(float* x, float v, long n, hipStream_t s);

}  // namespace spx
