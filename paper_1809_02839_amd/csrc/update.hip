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

// Partial-aware update: the arena is cut into jobs, alternately plain ranges
// (gradient read from g) and split-K segments (gradient summed from the
// K-slice planes); every block takes CHUNK consecutive elements of one job.
constexpr int ITER = 4;
constexpr long CHUNK = static_cast<long>(NT) * VEC * ITER;
constexpr int MAX_JOBS = 2 * UPDATE_MAX_SEGMENTS + 1;

struct Job {
  long off, n;         // arena elements [off, off + n)
  const float* part;   // split-K planes of this range (plane stride n), or null: read g
  int splits;
  int block0;          // first block of this job
};
struct JobTable {
  Job job[MAX_JOBS];
  int njobs;
};

__global__ __launch_bounds__(NT) void fused_update_partials_kernel(float* __restrict__ W, float* __restrict__ v,
                                                                   const float* __restrict__ g, JobTable jt,
                                                                   void* wf, void* wb, int dtype, float lr,
                                                                   float gamma, float one_minus_gamma, float sf_lr,
                                                                   float sb_lr, int do_f, int do_b, int* flag) {
  int j = 0;
  while (j + 1 < jt.njobs && static_cast<int>(blockIdx.x) >= jt.job[j + 1].block0) ++j;
  const Job jb = jt.job[j];
  const long c0 = static_cast<long>(static_cast<int>(blockIdx.x) - jb.block0) * CHUNK;
  bool bad = false;
#pragma unroll 1
  for (int it = 0; it < ITER; ++it) {
    const long r = c0 + static_cast<long>(it) * NT * VEC + threadIdx.x * VEC;   // offset inside the job
    if (r >= jb.n) break;
    const long i = jb.off + r;
    f8 w = ld8(W + i), m = ld8(v + i);
    float gv[VEC];
    if (jb.part) {
      // the split-K reduction's sum: plane 0, then planes 1, 2, ... added in order
      const f8 p0 = ld8(jb.part + r);
      gv[0] = p0.a.x; gv[1] = p0.a.y; gv[2] = p0.a.z; gv[3] = p0.a.w;
      gv[4] = p0.b.x; gv[5] = p0.b.y; gv[6] = p0.b.z; gv[7] = p0.b.w;
      for (int s0 = 1; s0 < jb.splits; s0 += 4) {
        f8 t[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (s0 + q < jb.splits) t[q] = ld8(jb.part + (s0 + q) * jb.n + r);
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (s0 + q < jb.splits) {
            gv[0] += t[q].a.x; gv[1] += t[q].a.y; gv[2] += t[q].a.z; gv[3] += t[q].a.w;
            gv[4] += t[q].b.x; gv[5] += t[q].b.y; gv[6] += t[q].b.z; gv[7] += t[q].b.w;
          }
      }
    } else {
      const f8 gr = ld8(g + i);
      gv[0] = gr.a.x; gv[1] = gr.a.y; gv[2] = gr.a.z; gv[3] = gr.a.w;
      gv[4] = gr.b.x; gv[5] = gr.b.y; gv[6] = gr.b.z; gv[7] = gr.b.w;
    }
    float wv[VEC] = {w.a.x, w.a.y, w.a.z, w.a.w, w.b.x, w.b.y, w.b.z, w.b.w};
    float mv[VEC] = {m.a.x, m.a.y, m.a.z, m.a.w, m.b.x, m.b.y, m.b.z, m.b.w};
    float pf[VEC], pb[VEC];
#pragma unroll
    for (int q = 0; q < VEC; ++q) {
      mv[q] = fmaf(gamma, mv[q], one_minus_gamma * gv[q]);
      wv[q] = fmaf(-lr, mv[q], wv[q]);
      pf[q] = fmaf(-sf_lr, mv[q], wv[q]);
      pb[q] = fmaf(-sb_lr, mv[q], wv[q]);
      bad |= !isfinite(wv[q]) || !isfinite(mv[q]);
    }
    st8(W + i, f8{make_float4(wv[0], wv[1], wv[2], wv[3]), make_float4(wv[4], wv[5], wv[6], wv[7])});
    st8(v + i, f8{make_float4(mv[0], mv[1], mv[2], mv[3]), make_float4(mv[4], mv[5], mv[6], mv[7])});
    if (do_f) store_pred(wf, dtype, i, pf);
    if (do_b) store_pred(wb, dtype, i, pb);
  }
  if (bad) *reinterpret_cast<volatile int*>(flag) = 1;
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

hipError_t fused_update_partials(float* W, float* v, const float* g, const UpdateSegment* segs, int nsegs,
                                 void* what_f, void* what_b, int what_dtype, long n, float lr, float gamma, int s_f,
                                 int s_b, int* flag, hipStream_t s) {
  if (n % VEC || nsegs < 0 || nsegs > UPDATE_MAX_SEGMENTS) return hipErrorInvalidValue;
  JobTable jt{};
  long pos = 0, blocks = 0;
  auto add = [&](long off, long len, const float* part, int splits) {
    if (len <= 0) return;
    Job& jb = jt.job[jt.njobs++];
    jb.off = off;
    jb.n = len;
    jb.part = part;
    jb.splits = splits;
    jb.block0 = static_cast<int>(blocks);
    blocks += (len + CHUNK - 1) / CHUNK;
  };
  for (int i = 0; i < nsegs; ++i) {
    const UpdateSegment& sg = segs[i];
    if (sg.off < pos || sg.n <= 0 || sg.off % VEC || sg.n % VEC || sg.off + sg.n > n || !sg.part ||
        sg.splits < 1)
      return hipErrorInvalidValue;
    add(pos, sg.off - pos, nullptr, 0);
    add(sg.off, sg.n, sg.part, sg.splits);
    pos = sg.off + sg.n;
  }
  add(pos, n - pos, nullptr, 0);
  if (blocks == 0) return hipSuccess;
  if (blocks > (1L << 30)) return hipErrorInvalidValue;
  const float sf_lr = s_f >= 0 ? static_cast<float>(s_f) * lr : 0.0f;
  const float sb_lr = s_b >= 0 ? static_cast<float>(s_b) * lr : 0.0f;
  hipLaunchKernelGGL(fused_update_partials_kernel, dim3(static_cast<unsigned>(blocks)), dim3(NT), 0, s, W, v, g,
                     jt, what_f, what_b, what_dtype, lr, gamma, 1.0f - gamma, sf_lr, sb_lr, s_f >= 0 ? 1 : 0,
                     s_b >= 0 ? 1 : 0, flag);
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
