// float32 GEMM for float32 stages (the small fully-connected workload):
// 64 x 64 block tile, K step 16, 256 threads each computing a 4 x 4 patch
// with FMAs. Any M, N, K and leading dimension; plain operand modes only.
// These stages are a few MFLOP per layer, so latency rather than matrix-core
// throughput bounds them.
#include "kernels.hpp"

namespace spx {
namespace {

constexpr int TB = 64, TK = 16, NT = 256;

struct F32Args {
  int M, N, K;
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

template <int MA, int MB>
__global__ __launch_bounds__(NT) void gemm_f32_kernel(F32Args a) {
  __shared__ float As[TK][TB + 4];
  __shared__ float Bs[TK][TB + 4];
  const int tid = threadIdx.x;
  const int row0 = blockIdx.y * TB, col0 = blockIdx.x * TB;
  const int tx = tid & 15, ty = tid >> 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < a.K; k0 += TK) {
    load_tile<MA>(a.A, a.lda, a.M, a.K, row0, k0, tid, As);
    load_tile<MB>(a.B, a.ldb, a.N, a.K, col0, k0, tid, Bs);
    __syncthreads();
#pragma unroll
    for (int k = 0; k < TK; ++k) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[k][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[k][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = row0 + ty * 4 + i;
    if (row >= a.M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = col0 + tx * 4 + j;
      if (col >= a.N) continue;
      const long idx = static_cast<long>(row) * a.ldc + col;
      float v = acc[i][j] * a.alpha;
      if (a.bias) v += a.bias[col];
      if (a.res) v += a.res[idx];
      if (a.relu) v = fmaxf(v, 0.0f);
      if (a.mask && !(a.mask[idx] > 0.0f)) v = 0.0f;
      if (a.accumulate) a.out[idx] += v;
      else a.out[idx] = v;
    }
  }
}

template <int MA, int MB>
hipError_t launch(const F32Args& a, hipStream_t s) {
  dim3 grid((a.N + TB - 1) / TB, (a.M + TB - 1) / TB);
  hipLaunchKernelGGL((gemm_f32_kernel<MA, MB>), grid, dim3(NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace

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
  const int ma = d.A.mode, mb = d.B.mode;
  if (ma == OP_K_PLAIN && mb == OP_K_PLAIN) return launch<OP_K_PLAIN, OP_K_PLAIN>(a, s);
  if (ma == OP_K_PLAIN && mb == OP_R_PLAIN) return launch<OP_K_PLAIN, OP_R_PLAIN>(a, s);
  if (ma == OP_R_PLAIN && mb == OP_R_PLAIN) return launch<OP_R_PLAIN, OP_R_PLAIN>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace spx
