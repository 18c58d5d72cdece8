// Memory-bound kernels of the stage step: ReLU-gradient masks, deterministic
// column sums (bias and layer-norm gradients), softmax cross-entropy,
// layer norm, attention softmax forward/backward and the LSTM cell.
// Every reduction runs in a fixed order, so results are bitwise reproducible.
#include <algorithm>
#include <atomic>

#include "kernels.hpp"

namespace spx {
namespace {

constexpr int NT = 256;

int blocks_for(long n, int per_thread) {
  long b = (n + static_cast<long>(NT) * per_thread - 1) / (static_cast<long>(NT) * per_thread);
  if (b < 1) b = 1;
  if (b > 65535L * 4) b = 65535L * 4;
  return static_cast<int>(b);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Block-wide reductions in a fixed order (256 threads = 4 waves).
__device__ float block_sum(float v, float* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  return (sh[0] + sh[1]) + (sh[2] + sh[3]);
}
__device__ float block_max(float v, float* sh) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  return fmaxf(fmaxf(sh[0], sh[1]), fmaxf(sh[2], sh[3]));
}

// ---------------------------------------------------------------- masks ----
__global__ void mask_bf16_kernel(const bf16_t* src, const bf16_t* mask, bf16_t* dst, long n) {
  for (long i = static_cast<long>(blockIdx.x) * NT + threadIdx.x; i < n; i += static_cast<long>(gridDim.x) * NT)
    dst[i] = bf16_to_f32(mask[i]) > 0.0f ? src[i] : static_cast<bf16_t>(0);
}
// 8 values per thread with 16-byte accesses (n % 8 == 0, 16-byte aligned).
__global__ void mask_bf16x8_kernel(const uint4* src, const uint4* mask, uint4* dst, long n8) {
  for (long i = static_cast<long>(blockIdx.x) * NT + threadIdx.x; i < n8; i += static_cast<long>(gridDim.x) * NT) {
    const uint4 a = src[i], m = mask[i];
    const uint32_t av[4] = {a.x, a.y, a.z, a.w}, mv[4] = {m.x, m.y, m.z, m.w};
    uint32_t o[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t lo = bf16_to_f32(static_cast<bf16_t>(mv[q] & 0xffff)) > 0.0f ? 0x0000ffffu : 0u;
      const uint32_t hi = bf16_to_f32(static_cast<bf16_t>(mv[q] >> 16)) > 0.0f ? 0xffff0000u : 0u;
      o[q] = av[q] & (lo | hi);
    }
    dst[i] = make_uint4(o[0], o[1], o[2], o[3]);
  }
}
__global__ void mask_f32_kernel(const float* src, const float* mask, float* dst, long n) {
  for (long i = static_cast<long>(blockIdx.x) * NT + threadIdx.x; i < n; i += static_cast<long>(gridDim.x) * NT)
    dst[i] = mask[i] > 0.0f ? src[i] : 0.0f;
}

// ------------------------------------------------- global average pool ----
// out[b][c] = bf16(sum over hw of x[b][hw][c] / HW) for an NHWC tensor; one
// thread per (b, c) sums its H x W values in order (columns of a block are
// consecutive channels, so every load of a wave is contiguous).
__global__ void avgpool_bf16_kernel(const bf16_t* x, int HW, int C, bf16_t* out) {
  const int c = blockIdx.x * NT + threadIdx.x, b = blockIdx.y;
  if (c >= C) return;
  const bf16_t* p = x + static_cast<long>(b) * HW * C + c;
  float s = 0.0f;
#pragma unroll 8
  for (int i = 0; i < HW; ++i) s += bf16_to_f32(p[static_cast<long>(i) * C]);
  out[static_cast<long>(b) * C + c] = f32_to_bf16(__fdiv_rn(s, static_cast<float>(HW)));
}

// Backward of the pool through the ReLU of the pooled activations:
// dx[b][hw][c] = y[b][hw][c] > 0 ? bf16(dpool[b][c] / HW) : 0, eight channels
// per thread (C % 8 == 0).
__global__ void avgpool_bwd_mask_kernel(const bf16_t* dpool, const bf16_t* y, long n8, int HW, int C,
                                        bf16_t* dx) {
  const int c8 = C / 8;
  const float hw_f = static_cast<float>(HW);
  for (long i = static_cast<long>(blockIdx.x) * NT + threadIdx.x; i < n8; i += static_cast<long>(gridDim.x) * NT) {
    const long pix = i / c8;
    const int cg = static_cast<int>(i - pix * c8);
    const long b = pix / HW;
    const uint4 g = *reinterpret_cast<const uint4*>(dpool + b * C + cg * 8);
    const uint4 m = reinterpret_cast<const uint4*>(y)[i];
    const uint32_t gv[4] = {g.x, g.y, g.z, g.w}, mv[4] = {m.x, m.y, m.z, m.w};
    uint32_t o[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t lo = f32_to_bf16(__fdiv_rn(bf16_to_f32(static_cast<bf16_t>(gv[q] & 0xffff)), hw_f));
      const uint32_t hi = f32_to_bf16(__fdiv_rn(bf16_to_f32(static_cast<bf16_t>(gv[q] >> 16)), hw_f));
      const bool plo = bf16_to_f32(static_cast<bf16_t>(mv[q] & 0xffff)) > 0.0f;
      const bool phi = bf16_to_f32(static_cast<bf16_t>(mv[q] >> 16)) > 0.0f;
      o[q] = (plo ? lo : 0u) | (phi ? hi << 16 : 0u);
    }
    reinterpret_cast<uint4*>(dx)[i] = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// --------------------------------------------------------- column sums ----
// Pass 1: block (cb, rb) sums rows [rb*RCH, (rb+1)*RCH) of its columns into
// partial[rb][col]. bf16 inputs with cols % 8 == 0 use 16-byte loads: 32
// column groups of 8 x 8 row lanes; otherwise 64 columns x 4 row lanes.
constexpr int RCH = COLSUM_ROWS;
__global__ void colsum_partial_bf16x8_kernel(const bf16_t* X, long rows, int cols, long ld, float* partial) {
  __shared__ float sh[8][256];
  const int cg = threadIdx.x & 31, rl = threadIdx.x >> 5;
  const int col = blockIdx.x * 256 + cg * 8;
  const long r0 = static_cast<long>(blockIdx.y) * RCH;
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  if (col < cols) {
#pragma unroll 8
    for (long r = r0 + rl; r < r0 + RCH && r < rows; r += 8) {
      const uint4 v = *reinterpret_cast<const uint4*>(X + r * ld + col);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        acc[2 * q] += __uint_as_float(w[q] << 16);
        acc[2 * q + 1] += __uint_as_float(w[q] & 0xffff0000u);
      }
    }
  }
#pragma unroll
  for (int q = 0; q < 8; ++q) sh[rl][cg * 8 + q] = acc[q];
  __syncthreads();
  const int c = threadIdx.x;   // 256 columns of this block
  if (blockIdx.x * 256 + c < cols) {
    float t = 0.0f;
#pragma unroll
    for (int q = 0; q < 8; ++q) t += sh[q][c];
    partial[static_cast<long>(blockIdx.y) * cols + blockIdx.x * 256 + c] = t;
  }
}
template <typename T>
__global__ void colsum_partial_kernel(const T* X, long rows, int cols, long ld, float* partial) {
  __shared__ float sh[4][64];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int col = blockIdx.x * 64 + tx;
  const long r0 = static_cast<long>(blockIdx.y) * RCH;
  float s = 0.0f;
  if (col < cols) {
#pragma unroll 8
    for (long r = r0 + ty; r < r0 + RCH && r < rows; r += 4) {
      if constexpr (sizeof(T) == 2) s += bf16_to_f32(X[r * ld + col]);
      else s += X[r * ld + col];
    }
  }
  sh[ty][tx] = s;
  __syncthreads();
  if (ty == 0 && col < cols) partial[static_cast<long>(blockIdx.y) * cols + col] = (sh[0][tx] + sh[1][tx]) + (sh[2][tx] + sh[3][tx]);
}
// Pass 2: 16 columns per block of 256 threads; thread t sums chunks
// c = t / 16 (mod 16) of column t % 16, and the 16 sums of a column are added
// in a fixed order.
__global__ __launch_bounds__(256) void colsum_final_kernel(const float* partial, int nchunks, int cols, float* out,
                                                           int accumulate) {
  __shared__ float sh[16][16];
  const int cx = threadIdx.x & 15, cy = threadIdx.x >> 4;
  const int col = blockIdx.x * 16 + cx;
  float s = 0.0f;
  if (col < cols) {
    // eight loads in flight per thread; the sum keeps its sequential order
#pragma unroll 8
    for (int c = cy; c < nchunks; c += 16) s += partial[static_cast<long>(c) * cols + col];
  }
  sh[cy][cx] = s;
  __syncthreads();
  if (cy == 0 && col < cols) {
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < 16; ++w) v += sh[w][cx];
    out[col] = accumulate ? out[col] + v : v;
  }
}

// colsum_final_kernel over partial rows of `stride` floats (columns [0, cols)
// of each row), the same order of additions.
__global__ __launch_bounds__(256) void colsum_strided_final_kernel(const float* partial, int nchunks, int cols,
                                                                   int stride, float* out) {
  __shared__ float sh[16][16];
  const int cx = threadIdx.x & 15, cy = threadIdx.x >> 4;
  const int col = blockIdx.x * 16 + cx;
  float s = 0.0f;
  if (col < cols) {
#pragma unroll 8
    for (int c = cy; c < nchunks; c += 16) s += partial[static_cast<long>(c) * stride + col];
  }
  sh[cy][cx] = s;
  __syncthreads();
  if (cy == 0 && col < cols) {
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < 16; ++w) v += sh[w][cx];
    out[col] = v;
  }
}

// ---------------------------------------------------- cross-entropy ----
constexpr int CE_ROW_MAX = 32768, CE_ROW_MIN = 4096, CE_ROW_NT = 1024;

// Long rows held in registers (CE_ROW_MIN <= C <= CE_ROW_MAX, C % 4 == 0, bf16
// gradients): one persistent 1024-thread block per CU walks the rows r =
// blockIdx.x, + gridDim.x, ...; thread t owns the 16-byte chunks c = t + 1024 i
// (i < 8) of every row, so the row needs no LDS, and its share of the next row
// is loaded into a second register set while the current row's exponentials,
// sums and gradients are formed and stored (each row is read from memory
// once). Exponentials use the hardware exp2-based __expf (relative error near
// 1e-7, far below the bf16 rounding of the gradient); the target's score is
// read back from memory.
constexpr int CE_ROW_CHUNKS = CE_ROW_MAX / 4 / CE_ROW_NT;   // 16-byte chunks per thread
__global__ __launch_bounds__(CE_ROW_NT) void softmax_ce_rows_kernel(const float* logits, const int32_t* labels, int R,
                                                                    int C, bf16_t* dlogits, float* row_loss) {
  __shared__ float sh[CE_ROW_NT / 64];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int C4 = C / 4;
  auto reduce = [&](float v, bool is_max) {
    v = is_max ? wave_max(v) : wave_sum(v);
    __syncthreads();   // sh may still be read by the previous reduction
    if (lane == 0) sh[wv] = v;
    __syncthreads();
    float t = sh[0];
#pragma unroll
    for (int w = 1; w < CE_ROW_NT / 64; ++w) t = is_max ? fmaxf(t, sh[w]) : t + sh[w];
    return t;
  };
  auto load = [&](int r, float4 (&v)[CE_ROW_CHUNKS]) {
    const float4* z = reinterpret_cast<const float4*>(logits + static_cast<long>(r) * C);
#pragma unroll
    for (int i = 0; i < CE_ROW_CHUNKS; ++i) {
      const int c = tid + CE_ROW_NT * i;
      if (c < C4) v[i] = z[c];
    }
  };
  const float inv_r = 1.0f / static_cast<float>(R);
  float4 cur[CE_ROW_CHUNKS], nxt[CE_ROW_CHUNKS];
  int r = blockIdx.x;
  if (r < R) load(r, nxt);
  for (; r < R; r += gridDim.x) {
#pragma unroll
    for (int i = 0; i < CE_ROW_CHUNKS; ++i) cur[i] = nxt[i];
    if (r + static_cast<int>(gridDim.x) < R) load(r + gridDim.x, nxt);   // in flight during this row
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < CE_ROW_CHUNKS; ++i)
      if (tid + CE_ROW_NT * i < C4) m = fmaxf(m, fmaxf(fmaxf(cur[i].x, cur[i].y), fmaxf(cur[i].z, cur[i].w)));
    m = reduce(m, true);
    const int lab = labels[r];
    const bool lab_ok = lab >= 0 && lab < C;
    const float zl = (tid == 0 && lab_ok) ? logits[static_cast<long>(r) * C + lab] : 0.0f;
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < CE_ROW_CHUNKS; ++i)
      if (tid + CE_ROW_NT * i < C4) {
        const float4 v = cur[i];
        cur[i] = make_float4(__expf(v.x - m), __expf(v.y - m), __expf(v.z - m), __expf(v.w - m));
        s += (cur[i].x + cur[i].y) + (cur[i].z + cur[i].w);
      }
    s = reduce(s, false);
    if (tid == 0) row_loss[r] = lab_ok ? (m + logf(s)) - zl : NAN;
    const float inv_s = 1.0f / s;
    uint2* out = reinterpret_cast<uint2*>(dlogits + static_cast<long>(r) * C);
#pragma unroll
    for (int i = 0; i < CE_ROW_CHUNKS; ++i) {
      const int c = tid + CE_ROW_NT * i;
      if (c >= C4) continue;
      const float4 e = cur[i];
      float p[4] = {e.x * inv_s, e.y * inv_s, e.z * inv_s, e.w * inv_s};
#pragma unroll
      for (int q = 0; q < 4; ++q) p[q] = ((4 * c + q == lab) ? p[q] - 1.0f : p[q]) * inv_r;
      out[c] = make_uint2(f32_to_bf16(p[0]) | (static_cast<uint32_t>(f32_to_bf16(p[1])) << 16),
                          f32_to_bf16(p[2]) | (static_cast<uint32_t>(f32_to_bf16(p[3])) << 16));
    }
  }
}

// Rows of C % 4 == 0 float32 scores with bf16 gradients: 16-byte loads, four
// chunks in flight per thread in each of the three passes over the row (max,
// sum of exponentials, gradient), 8-byte gradient stores.
__global__ __launch_bounds__(NT) void softmax_ce_bf16x4_kernel(const float* logits, const int32_t* labels, int R,
                                                               int C, bf16_t* dlogits, float* row_loss) {
  __shared__ float sh[4];
  const int r = blockIdx.x;
  const float4* z = reinterpret_cast<const float4*>(logits + static_cast<long>(r) * C);
  const int C4 = C / 4;
  float m = -INFINITY;
#pragma unroll 4
  for (int c = threadIdx.x; c < C4; c += NT) {
    const float4 v = z[c];
    m = fmaxf(m, fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w)));
  }
  m = block_max(m, sh);
  float s = 0.0f;
#pragma unroll 4
  for (int c = threadIdx.x; c < C4; c += NT) {
    const float4 v = z[c];
    s += (expf(v.x - m) + expf(v.y - m)) + (expf(v.z - m) + expf(v.w - m));
  }
  s = block_sum(s, sh);
  const int lab = labels[r];
  const bool lab_ok = lab >= 0 && lab < C;
  if (threadIdx.x == 0) row_loss[r] = lab_ok ? (m + logf(s)) - logits[static_cast<long>(r) * C + lab] : NAN;
  const float inv_s = 1.0f / s, inv_r = 1.0f / static_cast<float>(R);
  uint2* out = reinterpret_cast<uint2*>(dlogits + static_cast<long>(r) * C);
#pragma unroll 4
  for (int c = threadIdx.x; c < C4; c += NT) {
    const float4 v = z[c];
    float p[4] = {expf(v.x - m) * inv_s, expf(v.y - m) * inv_s, expf(v.z - m) * inv_s, expf(v.w - m) * inv_s};
#pragma unroll
    for (int q = 0; q < 4; ++q) p[q] = ((4 * c + q == lab) ? p[q] - 1.0f : p[q]) * inv_r;
    out[c] = make_uint2(f32_to_bf16(p[0]) | (static_cast<uint32_t>(f32_to_bf16(p[1])) << 16),
                        f32_to_bf16(p[2]) | (static_cast<uint32_t>(f32_to_bf16(p[3])) << 16));
  }
}

template <int DT>
__global__ __launch_bounds__(NT) void softmax_ce_kernel(const float* logits, const int32_t* labels, int R, int C,
                                                        void* dlogits, float* row_loss) {
  __shared__ float sh[4];
  const int r = blockIdx.x;
  const float* z = logits + static_cast<long>(r) * C;
  float m = -INFINITY;
  for (int c = threadIdx.x; c < C; c += NT) m = fmaxf(m, z[c]);
  m = block_max(m, sh);
  float s = 0.0f;
  for (int c = threadIdx.x; c < C; c += NT) s += expf(z[c] - m);
  s = block_sum(s, sh);
  // a label outside [0, C) yields a NaN loss for its row and no target term
  const int lab = labels[r];
  const bool lab_ok = lab >= 0 && lab < C;
  if (threadIdx.x == 0) row_loss[r] = lab_ok ? (m + logf(s)) - z[lab] : NAN;
  const float inv_s = 1.0f / s, inv_r = 1.0f / static_cast<float>(R);
  for (int c = threadIdx.x; c < C; c += NT) {
    float p = expf(z[c] - m) * inv_s;
    float d = ((c == lab) ? p - 1.0f : p) * inv_r;
    if (DT == 1) static_cast<bf16_t*>(dlogits)[static_cast<long>(r) * C + c] = f32_to_bf16(d);
    else static_cast<float*>(dlogits)[static_cast<long>(r) * C + c] = d;
  }
}
__global__ __launch_bounds__(NT) void mean_kernel(const float* x, int n, float* out) {
  __shared__ float sh[4];
  float s = 0.0f;
  for (int i = threadIdx.x; i < n; i += NT) s += x[i];
  s = block_sum(s, sh);
  if (threadIdx.x == 0) out[0] = s / static_cast<float>(n);
}

// ---------------------------------------------------------- layer norm ----
// One wave per row; lane l owns the VPL = D/64 consecutive columns
// [l*VPL, (l+1)*VPL), read and written with the widest aligned accesses.
template <int VPL>
__device__ __forceinline__ void ld_row(const bf16_t* p, float (&v)[VPL]) {
  if constexpr (VPL % 8 == 0) {
#pragma unroll
    for (int q = 0; q < VPL / 8; ++q) {
      const uint4 u = reinterpret_cast<const uint4*>(p)[q];
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        v[q * 8 + 2 * t] = __uint_as_float(w[t] << 16);
        v[q * 8 + 2 * t + 1] = __uint_as_float(w[t] & 0xffff0000u);
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < VPL; ++j) v[j] = bf16_to_f32(p[j]);
  }
}
template <int VPL>
__device__ __forceinline__ void st_row(bf16_t* p, const float (&v)[VPL]) {
  if constexpr (VPL % 8 == 0) {
#pragma unroll
    for (int q = 0; q < VPL / 8; ++q) {
      uint4 u;
      u.x = f32_to_bf16(v[q * 8 + 0]) | (static_cast<uint32_t>(f32_to_bf16(v[q * 8 + 1])) << 16);
      u.y = f32_to_bf16(v[q * 8 + 2]) | (static_cast<uint32_t>(f32_to_bf16(v[q * 8 + 3])) << 16);
      u.z = f32_to_bf16(v[q * 8 + 4]) | (static_cast<uint32_t>(f32_to_bf16(v[q * 8 + 5])) << 16);
      u.w = f32_to_bf16(v[q * 8 + 6]) | (static_cast<uint32_t>(f32_to_bf16(v[q * 8 + 7])) << 16);
      reinterpret_cast<uint4*>(p)[q] = u;
    }
  } else {
#pragma unroll
    for (int j = 0; j < VPL; ++j) p[j] = f32_to_bf16(v[j]);
  }
}

template <int VPL>
__global__ __launch_bounds__(NT) void layernorm_fwd_kernel(const bf16_t* r, const bf16_t* gamma, const bf16_t* beta,
                                                           int R, int D, float eps, bf16_t* y, float* mean,
                                                           float* rstd) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= R) return;
  const long base = static_cast<long>(row) * D + lane * VPL;
  float v[VPL], g[VPL], b[VPL];
  ld_row<VPL>(r + base, v);
  ld_row<VPL>(gamma + lane * VPL, g);
  ld_row<VPL>(beta + lane * VPL, b);
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < VPL; ++j) s += v[j];
  const float mu = wave_sum(s) / static_cast<float>(D);
  float q = 0.0f;
#pragma unroll
  for (int j = 0; j < VPL; ++j) q += (v[j] - mu) * (v[j] - mu);
  const float rs = rsqrtf(wave_sum(q) / static_cast<float>(D) + eps);
#pragma unroll
  for (int j = 0; j < VPL; ++j) v[j] = g[j] * ((v[j] - mu) * rs) + b[j];
  st_row<VPL>(y + base, v);
  if (lane == 0) {
    mean[row] = mu;
    rstd[row] = rs;
  }
}

// Rows per block in the backward; per-block partial dgamma/dbeta.
// Partials are [block][3 D]: the column sums of dr, then of dy * x_hat
// (dgamma), then of dy (dbeta).
template <int VPL>
__global__ __launch_bounds__(NT) void layernorm_bwd_kernel(const bf16_t* dy, const bf16_t* r, const float* mean,
                                                           const float* rstd, const bf16_t* gamma, int R, int D,
                                                           bf16_t* dr, float* part) {
  __shared__ float shg[4][64 * VPL];
  __shared__ float shb[4][64 * VPL];
  __shared__ float shd[4][64 * VPL];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  float gm[VPL], pg[VPL], pb[VPL], pd[VPL];
  ld_row<VPL>(gamma + lane * VPL, gm);
#pragma unroll
  for (int j = 0; j < VPL; ++j) pg[j] = pb[j] = pd[j] = 0.0f;
  // wave w takes rows w, w + 4, ...: all of its rows are loaded before any
  // is reduced, so the loads overlap the cross-lane sums
  constexpr int RPW = LNB_ROWS / 4;
  float dq[RPW][VPL], xq[RPW][VPL], muq[RPW], rsq[RPW];
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    const int row = blockIdx.x * LNB_ROWS + w + 4 * q;
    if (row < R) {
      const long base = static_cast<long>(row) * D + lane * VPL;
      ld_row<VPL>(dy + base, dq[q]);
      ld_row<VPL>(r + base, xq[q]);
      muq[q] = mean[row];
      rsq[q] = rstd[row];
    }
  }
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    const int row = blockIdx.x * LNB_ROWS + w + 4 * q;
    if (row >= R) break;
    const long base = static_cast<long>(row) * D + lane * VPL;
    const float mu = muq[q], rs = rsq[q];
    float(&d)[VPL] = dq[q];
    float(&xh)[VPL] = xq[q];
    float s1 = 0.0f, s2 = 0.0f;
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      xh[j] = (xh[j] - mu) * rs;
      pg[j] += d[j] * xh[j];
      pb[j] += d[j];
      d[j] *= gm[j];          // dy * gamma
      s1 += d[j];
      s2 += d[j] * xh[j];
    }
    const float m1 = wave_sum(s1) / static_cast<float>(D), m2 = wave_sum(s2) / static_cast<float>(D);
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      d[j] = rs * (d[j] - m1 - xh[j] * m2);
      pd[j] += bf16_to_f32(f32_to_bf16(d[j]));   // the value stored below
    }
    st_row<VPL>(dr + base, d);
  }
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    shg[w][lane * VPL + j] = pg[j];
    shb[w][lane * VPL + j] = pb[j];
    shd[w][lane * VPL + j] = pd[j];
  }
  __syncthreads();
  float* prow = part + static_cast<long>(blockIdx.x) * 3 * D;
  for (int c = threadIdx.x; c < D; c += NT) {
    prow[c] = (shd[0][c] + shd[1][c]) + (shd[2][c] + shd[3][c]);
    prow[D + c] = (shg[0][c] + shg[1][c]) + (shg[2][c] + shg[3][c]);
    prow[2 * D + c] = (shb[0][c] + shb[1][c]) + (shb[2][c] + shb[3][c]);
  }
}

// ------------------------------------------------------ softmax (rows) ----
__global__ __launch_bounds__(NT) void softmax_rows_kernel(const float* S, int R, int C, float* P, bf16_t* Pb) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= R) return;
  const float* s = S + static_cast<long>(row) * C;
  float m = -INFINITY;
  for (int c = lane; c < C; c += 64) m = fmaxf(m, s[c]);
  m = wave_max(m);
  float sum = 0.0f;
  for (int c = lane; c < C; c += 64) sum += expf(s[c] - m);
  sum = wave_sum(sum);
  const float inv = 1.0f / sum;
  for (int c = lane; c < C; c += 64) {
    const float p = expf(s[c] - m) * inv;
    P[static_cast<long>(row) * C + c] = p;
    Pb[static_cast<long>(row) * C + c] = f32_to_bf16(p);
  }
}

__global__ __launch_bounds__(NT) void softmax_bwd_kernel(const float* P, const float* dP, int R, int C, bf16_t* dS) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= R) return;
  const long base = static_cast<long>(row) * C;
  float dot = 0.0f;
  for (int c = lane; c < C; c += 64) dot += P[base + c] * dP[base + c];
  dot = wave_sum(dot);
  for (int c = lane; c < C; c += 64) dS[base + c] = f32_to_bf16(P[base + c] * (dP[base + c] - dot));
}

// ------------------------------------------------------------ LSTM cell ----

__global__ void lstm_cell_fwd_kernel(const float* z, const float* c_prev, int B, int H, float* gates, float* c,
                                     bf16_t* h) {
  const long n = static_cast<long>(B) * H;
  for (long t = static_cast<long>(blockIdx.x) * NT + threadIdx.x; t < n; t += static_cast<long>(gridDim.x) * NT) {
    const int b = static_cast<int>(t / H), j = static_cast<int>(t - static_cast<long>(b) * H);
    const long zb = static_cast<long>(b) * 4 * H;
    const float i = sigmoidf(z[zb + j]);
    const float f = sigmoidf(z[zb + H + j]);
    const float g = tanhf(z[zb + 2 * H + j]);
    const float o = sigmoidf(z[zb + 3 * H + j]);
    const float cp = c_prev ? c_prev[t] : 0.0f;
    const float cn = fmaf(f, cp, i * g);
    gates[zb + j] = i;
    gates[zb + H + j] = f;
    gates[zb + 2 * H + j] = g;
    gates[zb + 3 * H + j] = o;
    c[t] = cn;
    h[t] = f32_to_bf16(o * tanhf(cn));
  }
}

__global__ void lstm_cell_bwd_kernel(const bf16_t* dh_out, const float* dh_rec, const float* gates, const float* c,
                                     const float* c_prev, int B, int H, float* dc, bf16_t* dz) {
  const long n = static_cast<long>(B) * H;
  for (long t = static_cast<long>(blockIdx.x) * NT + threadIdx.x; t < n; t += static_cast<long>(gridDim.x) * NT) {
    const int b = static_cast<int>(t / H), j = static_cast<int>(t - static_cast<long>(b) * H);
    const long zb = static_cast<long>(b) * 4 * H;
    const float i = gates[zb + j], f = gates[zb + H + j], g = gates[zb + 2 * H + j], o = gates[zb + 3 * H + j];
    const float dh = bf16_to_f32(dh_out[t]) + (dh_rec ? dh_rec[t] : 0.0f);
    const float tc = tanhf(c[t]);
    const float d_o = dh * tc;
    const float dct = dc[t] + dh * o * (1.0f - tc * tc);
    const float di = dct * g, dg = dct * i, df = dct * (c_prev ? c_prev[t] : 0.0f);
    dc[t] = dct * f;
    dz[zb + j] = f32_to_bf16(di * i * (1.0f - i));
    dz[zb + H + j] = f32_to_bf16(df * f * (1.0f - f));
    dz[zb + 2 * H + j] = f32_to_bf16(dg * (1.0f - g * g));
    dz[zb + 3 * H + j] = f32_to_bf16(d_o * o * (1.0f - o));
  }
}

// ---------------------------------------------------------------- misc ----
__global__ void add_bf16_kernel(const bf16_t* a, const bf16_t* b, bf16_t* out, long n) {
  for (long i = static_cast<long>(blockIdx.x) * NT + threadIdx.x; i < n; i += static_cast<long>(gridDim.x) * NT)
    out[i] = f32_to_bf16(bf16_to_f32(a[i]) + bf16_to_f32(b[i]));
}
__global__ void cast_f2b_kernel(const float* x, bf16_t* y, long n) {
  for (long i = static_cast<long>(blockIdx.x) * NT + threadIdx.x; i < n; i += static_cast<long>(gridDim.x) * NT)
    y[i] = f32_to_bf16(x[i]);
}
__global__ void cast_b2f_kernel(const bf16_t* x, float* y, long n) {
  for (long i = static_cast<long>(blockIdx.x) * NT + threadIdx.x; i < n; i += static_cast<long>(gridDim.x) * NT)
    y[i] = bf16_to_f32(x[i]);
}
__global__ void fill_kernel(float* x, float v, long n) {
  for (long i = static_cast<long>(blockIdx.x) * NT + threadIdx.x; i < n; i += static_cast<long>(gridDim.x) * NT)
    x[i] = v;
}

// Wt[c][t][o] = W[o][t][c] for each 3x3 filter W [Co][9][Ci] of a batch of
// layers: the convolution data gradient then reads its weight operand with
// k = t Co + o contiguous, as the forward reads W. One 64 x 64 (o, c) tile of
// one tap of one layer per block (blockIdx.z = 9 layer + tap) through LDS,
// 16-byte loads along c and stores along o (Co, Ci multiples of 8).
__global__ __launch_bounds__(256) void filter_transpose_kernel(FilterBatch fb) {
  __shared__ bf16_t tile[64][66];   // [o][c]
  const int layer = blockIdx.z / 9, t = blockIdx.z - 9 * layer;
  const bf16_t* const W = fb.W[layer];
  bf16_t* const Wt = fb.Wt[layer];
  const int Co = fb.Co, Ci = fb.Ci[layer];
  const int c0 = blockIdx.x * 64, o0 = blockIdx.y * 64, tid = threadIdx.x;
  if (c0 >= Ci) return;   // the grid covers the widest layer
#pragma unroll
  for (int v = tid; v < 512; v += 256) {
    const int r = v >> 3, q = (v & 7) * 8, o = o0 + r, c = c0 + q;
    uint4 val = make_uint4(0, 0, 0, 0);
    if (o < Co && c < Ci) val = *reinterpret_cast<const uint4*>(W + (static_cast<long>(o) * 9 + t) * Ci + c);
    const uint32_t w[4] = {val.x, val.y, val.z, val.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      tile[r][q + 2 * j] = static_cast<bf16_t>(w[j] & 0xffff);
      tile[r][q + 2 * j + 1] = static_cast<bf16_t>(w[j] >> 16);
    }
  }
  __syncthreads();
#pragma unroll
  for (int v = tid; v < 512; v += 256) {
    const int r = v >> 3, q = (v & 7) * 8, c = c0 + r, o = o0 + q;
    if (c < Ci && o < Co) {
      uint32_t w[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        w[j] = static_cast<uint32_t>(tile[q + 2 * j][r]) | (static_cast<uint32_t>(tile[q + 2 * j + 1][r]) << 16);
      *reinterpret_cast<uint4*>(Wt + (static_cast<long>(c) * 9 + t) * Co + o) = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

}  // namespace

hipError_t filter_transpose_bf16(const FilterBatch& fb, hipStream_t s) {
  if (fb.n <= 0) return hipSuccess;
  if (fb.n > FilterBatch::MAX || fb.Co <= 0 || fb.Co % 8) return hipErrorInvalidValue;
  int cmax = 0;
  for (int l = 0; l < fb.n; ++l) {
    if (fb.Ci[l] <= 0 || fb.Ci[l] % 8 || !fb.W[l] || !fb.Wt[l]) return hipErrorInvalidValue;
    cmax = std::max(cmax, fb.Ci[l]);
  }
  hipLaunchKernelGGL(filter_transpose_kernel, dim3((cmax + 63) / 64, (fb.Co + 63) / 64, 9 * fb.n), dim3(256), 0, s, fb);
  return hipGetLastError();
}

hipError_t mask_relu_grad(const void* src, const void* mask, void* dst, long n, int dtype, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  auto al16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
  if (dtype == 1 && n % 8 == 0 && al16(src) && al16(mask) && al16(dst))
    hipLaunchKernelGGL(mask_bf16x8_kernel, dim3(blocks_for(n / 8, 1)), dim3(NT), 0, s, static_cast<const uint4*>(src),
                       static_cast<const uint4*>(mask), static_cast<uint4*>(dst), n / 8);
  else if (dtype == 1)
    hipLaunchKernelGGL(mask_bf16_kernel, dim3(blocks_for(n, 4)), dim3(NT), 0, s, static_cast<const bf16_t*>(src),
                       static_cast<const bf16_t*>(mask), static_cast<bf16_t*>(dst), n);
  else
    hipLaunchKernelGGL(mask_f32_kernel, dim3(blocks_for(n, 4)), dim3(NT), 0, s, static_cast<const float*>(src),
                       static_cast<const float*>(mask), static_cast<float*>(dst), n);
  return hipGetLastError();
}

hipError_t avgpool_fwd(const bf16_t* x, int B, int HW, int C, bf16_t* out, hipStream_t s) {
  if (B <= 0 || C <= 0) return hipSuccess;
  if (HW <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(avgpool_bf16_kernel, dim3((C + NT - 1) / NT, B), dim3(NT), 0, s, x, HW, C, out);
  return hipGetLastError();
}

hipError_t avgpool_bwd_mask(const bf16_t* dpool, const bf16_t* y, int B, int HW, int C, bf16_t* dx, hipStream_t s) {
  if (C % 8 || HW <= 0) return hipErrorInvalidValue;
  const long n8 = static_cast<long>(B) * HW * (C / 8);
  if (n8 <= 0) return hipSuccess;
  hipLaunchKernelGGL(avgpool_bwd_mask_kernel, dim3(blocks_for(n8, 1)), dim3(NT), 0, s, dpool, y, n8, HW, C, dx);
  return hipGetLastError();
}

hipError_t column_sum(const void* X, int dtype, long rows, int cols, long ld, float* out, int accumulate,
                      float* partial_ws, hipStream_t s) {
  if (cols <= 0) return hipSuccess;
  const int nchunks = rows > 0 ? static_cast<int>((rows + RCH - 1) / RCH) : 0;
  if (nchunks > 0) {
    if (dtype == 1 && cols % 8 == 0 && ld % 8 == 0 && (reinterpret_cast<uintptr_t>(X) & 15) == 0) {
      hipLaunchKernelGGL(colsum_partial_bf16x8_kernel, dim3((cols + 255) / 256, nchunks), dim3(NT), 0, s,
                         static_cast<const bf16_t*>(X), rows, cols, ld, partial_ws);
    } else if (dtype == 1) {
      hipLaunchKernelGGL(colsum_partial_kernel<bf16_t>, dim3((cols + 63) / 64, nchunks), dim3(NT), 0, s,
                         static_cast<const bf16_t*>(X), rows, cols, ld, partial_ws);
    } else {
      hipLaunchKernelGGL(colsum_partial_kernel<float>, dim3((cols + 63) / 64, nchunks), dim3(NT), 0, s,
                         static_cast<const float*>(X), rows, cols, ld, partial_ws);
    }
  }
  hipLaunchKernelGGL(colsum_final_kernel, dim3((cols + 15) / 16), dim3(256), 0, s, partial_ws, nchunks,
                     cols, out, accumulate);
  return hipGetLastError();
}

hipError_t softmax_ce(const float* logits, const int32_t* labels, int R, int C, void* dlogits, int dtype, float* loss,
                      float* row_loss_ws, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  const bool vec = C % 4 == 0 && (reinterpret_cast<uintptr_t>(logits) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(dlogits) & 7) == 0;
  if (dtype == 1 && vec && C >= CE_ROW_MIN && C <= CE_ROW_MAX) {
    // one persistent block per CU; the count is read once per device
    static std::atomic<int> cu_count[64];
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < 64) {
      cus = cu_count[dev].load(std::memory_order_relaxed);
      if (cus <= 0) {
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
        cu_count[dev].store(cus, std::memory_order_relaxed);
      }
    }
    hipLaunchKernelGGL(softmax_ce_rows_kernel, dim3(std::min(R, std::max(cus, 1))), dim3(CE_ROW_NT), 0, s, logits,
                       labels, R, C, static_cast<bf16_t*>(dlogits), row_loss_ws);
  }
  else if (dtype == 1 && vec)
    hipLaunchKernelGGL(softmax_ce_bf16x4_kernel, dim3(R), dim3(NT), 0, s, logits, labels, R, C,
                       static_cast<bf16_t*>(dlogits), row_loss_ws);
  else if (dtype == 1)
    hipLaunchKernelGGL(softmax_ce_kernel<1>, dim3(R), dim3(NT), 0, s, logits, labels, R, C, dlogits, row_loss_ws);
  else
    hipLaunchKernelGGL(softmax_ce_kernel<0>, dim3(R), dim3(NT), 0, s, logits, labels, R, C, dlogits, row_loss_ws);
  hipLaunchKernelGGL(mean_kernel, dim3(1), dim3(NT), 0, s, row_loss_ws, R, loss);
  return hipGetLastError();
}

hipError_t layernorm_fwd(const bf16_t* r, const bf16_t* gamma, const bf16_t* beta, int R, int D, float eps, bf16_t* y,
                         float* mean, float* rstd, hipStream_t s) {
  if (D % 64 || D > 64 * 32) return hipErrorInvalidValue;
  const dim3 grid((R + 3) / 4), block(NT);
  switch (D / 64) {
    case 1: hipLaunchKernelGGL(layernorm_fwd_kernel<1>, grid, block, 0, s, r, gamma, beta, R, D, eps, y, mean, rstd); break;
    case 2: hipLaunchKernelGGL(layernorm_fwd_kernel<2>, grid, block, 0, s, r, gamma, beta, R, D, eps, y, mean, rstd); break;
    case 4: hipLaunchKernelGGL(layernorm_fwd_kernel<4>, grid, block, 0, s, r, gamma, beta, R, D, eps, y, mean, rstd); break;
    case 8: hipLaunchKernelGGL(layernorm_fwd_kernel<8>, grid, block, 0, s, r, gamma, beta, R, D, eps, y, mean, rstd); break;
    case 16: hipLaunchKernelGGL(layernorm_fwd_kernel<16>, grid, block, 0, s, r, gamma, beta, R, D, eps, y, mean, rstd); break;
    case 32: hipLaunchKernelGGL(layernorm_fwd_kernel<32>, grid, block, 0, s, r, gamma, beta, R, D, eps, y, mean, rstd); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t layernorm_bwd_rows(const bf16_t* dy, const bf16_t* r, const float* mean, const float* rstd,
                              const bf16_t* gamma, int R, int D, bf16_t* dr, float* partial_ws, hipStream_t s) {
  if (D % 64 || D > 64 * 32) return hipErrorInvalidValue;
  const int nb = (R + LNB_ROWS - 1) / LNB_ROWS;
  const dim3 grid(nb), block(NT);
  float* p = partial_ws;
  switch (D / 64) {
    case 1: hipLaunchKernelGGL(layernorm_bwd_kernel<1>, grid, block, 0, s, dy, r, mean, rstd, gamma, R, D, dr, p); break;
    case 2: hipLaunchKernelGGL(layernorm_bwd_kernel<2>, grid, block, 0, s, dy, r, mean, rstd, gamma, R, D, dr, p); break;
    case 4: hipLaunchKernelGGL(layernorm_bwd_kernel<4>, grid, block, 0, s, dy, r, mean, rstd, gamma, R, D, dr, p); break;
    case 8: hipLaunchKernelGGL(layernorm_bwd_kernel<8>, grid, block, 0, s, dy, r, mean, rstd, gamma, R, D, dr, p); break;
    case 16: hipLaunchKernelGGL(layernorm_bwd_kernel<16>, grid, block, 0, s, dy, r, mean, rstd, gamma, R, D, dr, p); break;
    case 32: hipLaunchKernelGGL(layernorm_bwd_kernel<32>, grid, block, 0, s, dy, r, mean, rstd, gamma, R, D, dr, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t layernorm_bwd_params(const float* partial_ws, int R, int D, float* dgamma, float* dbeta, float* dsum,
                                hipStream_t s) {
  const int nb = (R + LNB_ROWS - 1) / LNB_ROWS;
  const float* p = partial_ws;
  // partial columns [0, D) sum dr, [D, 2D) dgamma, [2D, 3D) dbeta
  if (dsum && dsum + D == dgamma && dgamma + D == dbeta) {
    hipLaunchKernelGGL(colsum_final_kernel, dim3((3 * D + 15) / 16), dim3(256), 0, s, p, nb, 3 * D, dsum, 0);
    return hipGetLastError();
  }
  float* out[3] = {dsum, dgamma, dbeta};
  for (int i = 0; i < 3; ++i)
    if (out[i])
      hipLaunchKernelGGL(colsum_strided_final_kernel, dim3((D + 15) / 16), dim3(256), 0, s, p + i * D, nb, D, 3 * D,
                         out[i]);
  return hipGetLastError();
}

hipError_t layernorm_bwd(const bf16_t* dy, const bf16_t* r, const float* mean, const float* rstd, const bf16_t* gamma,
                         int R, int D, bf16_t* dr, float* dgamma, float* dbeta, float* dsum, float* partial_ws,
                         hipStream_t s) {
  const hipError_t e = layernorm_bwd_rows(dy, r, mean, rstd, gamma, R, D, dr, partial_ws, s);
  if (e != hipSuccess) return e;
  return layernorm_bwd_params(partial_ws, R, D, dgamma, dbeta, dsum, s);
}

hipError_t softmax_rows(const float* S, int R, int C, float* P, bf16_t* Pb, hipStream_t s) {
  hipLaunchKernelGGL(softmax_rows_kernel, dim3((R + 3) / 4), dim3(NT), 0, s, S, R, C, P, Pb);
  return hipGetLastError();
}

hipError_t softmax_bwd(const float* P, const float* dP, int R, int C, bf16_t* dS, hipStream_t s) {
  hipLaunchKernelGGL(softmax_bwd_kernel, dim3((R + 3) / 4), dim3(NT), 0, s, P, dP, R, C, dS);
  return hipGetLastError();
}

hipError_t lstm_cell_fwd(const float* z, const float* c_prev, int B, int H, float* gates, float* c, bf16_t* h,
                         hipStream_t s) {
  const long n = static_cast<long>(B) * H;
  hipLaunchKernelGGL(lstm_cell_fwd_kernel, dim3(blocks_for(n, 1)), dim3(NT), 0, s, z, c_prev, B, H, gates, c, h);
  return hipGetLastError();
}

hipError_t lstm_cell_bwd(const bf16_t* dh_out, const float* dh_rec, const float* gates, const float* c,
                         const float* c_prev, int B, int H, float* dc, bf16_t* dz, hipStream_t s) {
  const long n = static_cast<long>(B) * H;
  hipLaunchKernelGGL(lstm_cell_bwd_kernel, dim3(blocks_for(n, 1)), dim3(NT), 0, s, dh_out, dh_rec, gates, c, c_prev,
                     B, H, dc, dz);
  return hipGetLastError();
}

hipError_t add_bf16(const bf16_t* a, const bf16_t* b, bf16_t* out, long n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(add_bf16_kernel, dim3(blocks_for(n, 4)), dim3(NT), 0, s, a, b, out, n);
  return hipGetLastError();
}
hipError_t cast_f32_to_bf16(const float* x, bf16_t* y, long n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(cast_f2b_kernel, dim3(blocks_for(n, 4)), dim3(NT), 0, s, x, y, n);
  return hipGetLastError();
}
hipError_t cast_bf16_to_f32(const bf16_t* x, float* y, long n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(cast_b2f_kernel, dim3(blocks_for(n, 4)), dim3(NT), 0, s, x, y, n);
  return hipGetLastError();
}
hipError_t fill_f32(float* x, float v, long n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_kernel, dim3(blocks_for(n, 4)), dim3(NT), 0, s, x, v, n);
  return hipGetLastError();
}

}  // namespace spx
