// Fused momentum update and weight prediction (Section 3.2): one pass over
// the stage's flat float32 arenas that reads W, v, g once and writes
//   v' = gamma v + (1 - gamma) g                    (Eq. 1)
//   W' = W - eta v'                                  (momentum update)
//   What_f = W' - s_f eta v',  What_b = W' - s_b eta v'   (Eq. 4, both slots)
// The predicted slots are stored in the operand dtype (bf16 or float32).
// HBM traffic per parameter: 12 bytes read, 8 + 2 * sizeof(operand) written.
#include "kernels.hpp"

namespace spx {
namespace {

constexpr int NT = 256;
constexpr int VEC = 8;   // parameters per thread per iteration: two 16-byte float loads per array

struct f8 {
  float4 a, b;
};

__device__ __forceinline__ f8 ld8(const float* p) {
  f8 r;
  r.a = *reinterpret_cast<const float4*>(p);
  r.b = *reinterpret_cast<const float4*>(p + 4);
  return r;
}
__device__ __forceinline__ void st8(float* p, const f8& v) {
  *reinterpret_cast<float4*>(p) = v.a;
  *reinterpret_cast<float4*>(p + 4) = v.b;
}

__device__ __forceinline__ void store_pred(void* dst, int dtype, long i, const float (&x)[VEC]) {
  if (dtype == 1) {
    uint4 o;
    o.x = f32_to_bf16(x[0]) | (static_cast<uint32_t>(f32_to_bf16(x[1])) << 16);
    o.y = f32_to_bf16(x[2]) | (static_cast<uint32_t>(f32_to_bf16(x[3])) << 16);
    o.z = f32_to_bf16(x[4]) | (static_cast<uint32_t>(f32_to_bf16(x[5])) << 16);
    o.w = f32_to_bf16(x[6]) | (static_cast<uint32_t>(f32_to_bf16(x[7])) << 16);
    *reinterpret_cast<uint4*>(static_cast<bf16_t*>(dst) + i) = o;
  } else {
    float* d = static_cast<float*>(dst) + i;
    *reinterpret_cast<float4*>(d) = make_float4(x[0], x[1], x[2], x[3]);
    *reinterpret_cast<float4*>(d + 4) = make_float4(x[4], x[5], x[6], x[7]);
  }
}

__global__ __launch_bounds__(NT) void fused_update_kernel(float* __restrict__ W, float* __restrict__ v,
                                                          const float* __restrict__ g, void* wf, void* wb,
                                                          int dtype, long nvec, float lr, float gamma,
                                                          float one_minus_gamma, float sf_lr, float sb_lr,
                                                          int do_f, int do_b, int* flag) {
  const long stride = static_cast<long>(gridDim.x) * NT;
  bool bad = false;
  for (long t = static_cast<long>(blockIdx.x) * NT + threadIdx.x; t < nvec; t += stride) {
    const long i = t * VEC;
    f8 w = ld8(W + i), m = ld8(v + i), gr = ld8(g + i);
    float wv[VEC] = {w.a.x, w.a.y, w.a.z, w.a.w, w.b.x, w.b.y, w.b.z, w.b.w};
    float mv[VEC] = {m.a.x, m.a.y, m.a.z, m.a.w, m.b.x, m.b.y, m.b.z, m.b.w};
    const float gv[VEC] = {gr.a.x, gr.a.y, gr.a.z, gr.a.w, gr.b.x, gr.b.y, gr.b.z, gr.b.w};
    float pf[VEC], pb[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
      mv[j] = fmaf(gamma, mv[j], one_minus_gamma * gv[j]);
      wv[j] = fmaf(-lr, mv[j], wv[j]);
      pf[j] = fmaf(-sf_lr, mv[j], wv[j]);
      pb[j] = fmaf(-sb_lr, mv[j], wv[j]);
      bad |= !isfinite(wv[j]) || !isfinite(mv[j]);
    }
    st8(W + i, f8{make_float4(wv[0], wv[1], wv[2], wv[3]), make_float4(wv[4], wv[5], wv[6], wv[7])});
    st8(v + i, f8{make_float4(mv[0], mv[1], mv[2], mv[3]), make_float4(mv[4], mv[5], mv[6], mv[7])});
    if (do_f) store_pred(wf, dtype, i, pf);
    if (do_b) store_pred(wb, dtype, i, pb);
  }
  if (bad) *reinterpret_cast<volatile int*>(flag) = 1;
}

__global__ __launch_bounds__(NT) void predict_kernel(const float* __restrict__ W, const float* __restrict__ v,
                                                     void* out, int dtype, long nvec, float s_lr) {
  const long stride = static_cast<long>(gridDim.x) * NT;
  for (long t = static_cast<long>(blockIdx.x) * NT + threadIdx.x; t < nvec; t += stride) {
    const long i = t * VEC;
    f8 w = ld8(W + i), m = ld8(v + i);
    const float wv[VEC] = {w.a.x, w.a.y, w.a.z, w.a.w, w.b.x, w.b.y, w.b.z, w.b.w};
    const float mv[VEC] = {m.a.x, m.a.y, m.a.z, m.a.w, m.b.x, m.b.y, m.b.z, m.b.w};
    float p[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) p[j] = fmaf(-s_lr, mv[j], wv[j]);
    store_pred(out, dtype, i, p);
  }
}

int grid_for(long nvec) {
  long blocks = (nvec + NT - 1) / NT;
  const long cap = 256 * 16;  // 16 blocks per CU, grid-stride beyond
  return static_cast<int>(blocks < 1 ? 1 : (blocks > cap ? cap : blocks));
}

}  // namespace

// n must be a multiple of 8 (arenas are padded to 64-element tensor slots).
hipError_t fused_update(float* W, float* v, const float* g, void* what_f, void* what_b, int what_dtype, long n,
                        float lr, float gamma, int s_f, int s_b, int* flag, hipStream_t s) {
  if (n % VEC) return hipErrorInvalidValue;
  const long nvec = n / VEC;
  if (nvec == 0) return hipSuccess;
  const float sf_lr = s_f >= 0 ? static_cast<float>(s_f) * lr : 0.0f;
  const float sb_lr = s_b >= 0 ? static_cast<float>(s_b) * lr : 0.0f;
  hipLaunchKernelGGL(fused_update_kernel, dim3(grid_for(nvec)), dim3(NT), 0, s, W, v, g, what_f, what_b,
                     what_dtype, nvec, lr, gamma, 1.0f - gamma, sf_lr, sb_lr, s_f >= 0 ? 1 : 0, s_b >= 0 ? 1 : 0,
                     flag);
  return hipGetLastError();
}

hipError_t predict_slot(const float* W, const float* v, void* what, int what_dtype, long n, float lr, int s_pred,
                        hipStream_t s) {
  if (n % VEC || s_pred < 0) return hipErrorInvalidValue;
  const long nvec = n / VEC;
  if (nvec == 0) return hipSuccess;
  hipLaunchKernelGGL(predict_kernel, dim3(grid_for(nvec)), dim3(NT), 0, s, W, v, what, what_dtype, nvec,
                     static_cast<float>(s_pred) * lr);
  return hipGetLastError();
}

}  // namespace spx
