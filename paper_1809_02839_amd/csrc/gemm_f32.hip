// float32 GEMM for float32 stages (the small fully-connected workload) on
// the matrix cores: 64 x 64 block tile, K step 16 staged in LDS as [k][row],
// 4 waves each owning a 32 x 32 sub-tile of v_mfma_f32_32x32x2_f32 (eight
// per K step; float32 operands, float32 accumulation). Any M, N, K and
// leading dimension; plain operand modes only.
// These stages are a few MFLOP per layer, so latency rather than matrix-core
// throughput bounds them: when the tiles are few and K is long, K is split
// over blocks (each block's K loop stays short) and a second pass sums the
// partials in split order and applies the epilogue.
#include <algorithm>
#include <cstdio>

#include "kernels.hpp"

namespace spx {
namespace {

constexpr int TB = 64, TK = 16, NT = 256;
constexpr int TARGET_BLOCKS = 128;   // split K until about this many blocks run
constexpr int MIN_SPLIT_STEPS = 4;   // K steps per split at least
constexpr int MAX_SPLITS = 64;

struct F32Args {
  int M, N, K;
  int splits, k_per_split;   // splits > 1: raw partials [split][M][N] to `partial`
  float* partial;
  const float* A;
  long lda;
  const float* B;
  long ldb;
  float* out;
  long ldc;
  const float* bias;
  const float* res;
  const float* mask;
  float alpha;
  int relu, accumulate;
};

template <int MODE>
__device__ __forceinline__ void load_tile(const float* X, long ld, int rows, int K, int row0, int k0, int tid,
                                          float (*S)[TB + 4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int r, k;
    if (MODE == OP_K_PLAIN) {
      k = tid & 15;
      r = (tid >> 4) + 16 * i;
    } else {
      r = tid & 63;
      k = (tid >> 6) + 4 * i;
    }
    int gr = row0 + r, gk = k0 + k;
    float v = 0.0f;
    if (gr < rows && gk < K) v = (MODE == OP_K_PLAIN) ? X[static_cast<long>(gr) * ld + gk] : X[static_cast<long>(gk) * ld + gr];
    S[k][r] = v;
  }
}

// value = acc * alpha + bias + residual, ReLU, mask, then stored or added.
__device__ __forceinline__ void epilogue_f32(const F32Args& a, int row, int col, float acc) {
  const long idx = static_cast<long>(row) * a.ldc + col;
  float v = acc * a.alpha;
  if (a.bias) v += a.bias[col];
  if (a.res) v += a.res[idx];
  if (a.relu) v = fmaxf(v, 0.0f);
  if (a.mask && !(a.mask[idx] > 0.0f)) v = 0.0f;
  if (a.accumulate) a.out[idx] += v;
  else a.out[idx] = v;
}

// Wave w owns rows 32 (w / 2) .. and columns 32 (w % 2) .. of the block
// tile. Each MFMA takes two k: lane l supplies k = l / 32 of row l % 32 of
// each operand (B first, so the output's register layout is indexed by B's
// columns): lane l then holds output row l % 32 of columns
// 8 (r / 4) + 4 (l / 32) + r % 4 in register r.
template <int MA, int MB>
__global__ __launch_bounds__(NT) void gemm_f32_kernel(F32Args a) {
  __shared__ float As[TK][TB + 4];
  __shared__ float Bs[TK][TB + 4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row0 = blockIdx.y * TB, col0 = blockIdx.x * TB;
  const int wm = wave >> 1, wn = wave & 1;
  f32x16_t acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.0f;
  const int kbeg = blockIdx.z * a.k_per_split, kend = min(a.K, kbeg + a.k_per_split);
  const int ra = wm * 32 + (lane & 31), rb = wn * 32 + (lane & 31), kh = lane >> 5;
  for (int k0 = kbeg; k0 < kend; k0 += TK) {
    load_tile<MA>(a.A, a.lda, a.M, kend, row0, k0, tid, As);
    load_tile<MB>(a.B, a.ldb, a.N, kend, col0, k0, tid, Bs);
    __syncthreads();
#pragma unroll
    for (int k = 0; k < TK; k += 2)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(Bs[k + kh][rb], As[k + kh][ra], acc, 0, 0, 0);
    __syncthreads();
  }
  const int row = row0 + ra;
  if (row >= a.M) return;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int col = col0 + wn * 32 + 8 * (r >> 2) + 4 * kh + (r & 3);
    if (col >= a.N) continue;
    if (a.splits > 1)
      a.partial[(static_cast<long>(blockIdx.z) * a.M + row) * a.N + col] = acc[r];
    else
      epilogue_f32(a, row, col, acc[r]);
  }
}

// Sums the split partials of each output in split order, then the epilogue.
__global__ __launch_bounds__(256) void gemm_f32_reduce_kernel(F32Args a) {
  const long mn = static_cast<long>(a.M) * a.N;
  for (long t = static_cast<long>(blockIdx.x) * 256 + threadIdx.x; t < mn; t += static_cast<long>(gridDim.x) * 256) {
    float s = a.partial[t];
    for (int sp = 1; sp < a.splits; ++sp) s += a.partial[sp * mn + t];
    const int row = static_cast<int>(t / a.N), col = static_cast<int>(t - static_cast<long>(row) * a.N);
    epilogue_f32(a, row, col, s);
  }
}

template <int MA, int MB>
hipError_t launch(const F32Args& a, hipStream_t s) {
  dim3 grid((a.N + TB - 1) / TB, (a.M + TB - 1) / TB, a.splits);
  hipLaunchKernelGGL((gemm_f32_kernel<MA, MB>), grid, dim3(NT), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits == 1) return e;
  const long mn = static_cast<long>(a.M) * a.N;
  const long blocks = std::min<long>((mn + 255) / 256, 4096);
  hipLaunchKernelGGL(gemm_f32_reduce_kernel, dim3(static_cast<int>(blocks)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

const char* gemm_f32_kernel_name(const GemmDesc& d) {
  static thread_local char buf[48];
  std::snprintf(buf, sizeof(buf), "gemm_f32_kernel<%d, %d>", d.A.mode, d.B.mode);
  return buf;
}

hipError_t gemm_f32(const GemmDesc& d, hipStream_t s) {
  if (d.M <= 0 || d.N <= 0) return hipSuccess;
  if (d.batch != 1 || !d.epi.out_f32 || d.epi.out_bf16 || d.epi.res_bf16) return hipErrorInvalidValue;
  F32Args a{};
  a.M = d.M;
  a.N = d.N;
  a.K = d.K;
  a.A = static_cast<const float*>(d.A.ptr);
  a.lda = d.A.ld;
  a.B = static_cast<const float*>(d.B.ptr);
  a.ldb = d.B.ld;
  a.out = d.epi.out_f32;
  a.ldc = d.epi.ldc;
  a.bias = d.epi.bias;
  a.res = d.epi.res_f32;
  a.mask = static_cast<const float*>(d.epi.mask);
  a.alpha = d.epi.alpha;
  a.relu = d.epi.relu;
  a.accumulate = d.epi.accumulate;
  // K split: enough blocks to hide the K loop's latency, each split at least
  // MIN_SPLIT_STEPS steps long, partials within the workspace.
  const long tiles = static_cast<long>((a.N + TB - 1) / TB) * ((a.M + TB - 1) / TB);
  const int ksteps = (a.K + TK - 1) / TK;
  int splits = 1;
  if (d.workspace && tiles < TARGET_BLOCKS && ksteps >= 2 * MIN_SPLIT_STEPS) {
    splits = static_cast<int>(std::min<long>(TARGET_BLOCKS / tiles, ksteps / MIN_SPLIT_STEPS));
    splits = std::min(splits, MAX_SPLITS);
    while (splits > 1 && static_cast<size_t>(splits) * a.M * a.N * 4 > d.workspace_bytes) --splits;
  }
  const int steps_per = std::max(1, (ksteps + splits - 1) / splits);
  a.splits = std::max(1, (ksteps + steps_per - 1) / steps_per);   // no empty split
  a.k_per_split = steps_per * TK;
  a.partial = d.workspace;
  const int ma = d.A.mode, mb = d.B.mode;
  if (ma == OP_K_PLAIN && mb == OP_K_PLAIN) return launch<OP_K_PLAIN, OP_K_PLAIN>(a, s);
  if (ma == OP_K_PLAIN && mb == OP_R_PLAIN) return launch<OP_K_PLAIN, OP_R_PLAIN>(a, s);
  if (ma == OP_R_PLAIN && mb == OP_R_PLAIN) return launch<OP_R_PLAIN, OP_R_PLAIN>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace spx
