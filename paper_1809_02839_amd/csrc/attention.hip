// Fused multi-head attention core of the transformer encoder stage on gfx950
// (sequence length 128, head dimension 64): one block per (batch, head).
//
// Forward:  S = Q K^T * scale (float32), P = softmax(S) row-wise (float32),
//           ctx = bf16(P) V (float32 accumulation, bf16 result). Only the
//           row statistics (max, 1 / sum) are kept for the backward pass.
// Backward: P is recomputed from Q, K and the statistics with the same
//           instructions in the same order (so it is bit-identical to the
//           forward's), then dV = bf16(P)^T dO, dP = dO V^T,
//           dS = bf16(P * (dP - rowsum(P * dP))), dQ = dS K * scale,
//           dK = dS^T Q * scale (bf16 results).
//
// Four waves; wave w owns rows 32 w .. 32 w + 31 of every 128-row product.
// Products use v_mfma_f32_32x32x16_bf16 with the B fragment first, so a lane
// holds one row and groups of four consecutive columns of each 32 x 32 tile:
// a row's 128 scores live in lanes l and l ^ 32, and row reductions need one
// cross-lane exchange. Q rows (scores) and V rows (dP) come straight from
// global memory as rows of 8 consecutive k; K is staged in LDS once per block
// and read from there by all four waves; operands needed transposed (V for
// P V, P and dS for dV and dK, dO, K, Q) are staged in LDS as stored and read
// with ds_read_b64_tr_b16.
#include "kernels.hpp"

namespace spx {
namespace {

constexpr int S = 128, DH = 64, NT = 256;
constexpr int PP = S + 8;    // LDS pitch of 128-wide tiles (bf16 elements)
constexpr int PD = DH + 8;   // LDS pitch of 64-wide tiles

typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

__device__ __forceinline__ bf16x8_t gld8(const bf16_t* p) {
  return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u16x8_t*>(p));
}

// 8 consecutive k of row `row` from an LDS tile stored [row][k] with pitch P.
template <int P>
__device__ __forceinline__ bf16x8_t frag_rows(const bf16_t* s, int row, int k) {
  return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u16x8_t*>(s + row * P + k));
}

// The same operand for "row" m0 + lane % 32 and k = k0 + 8 (lane / 32) .. + 7
// from an LDS tile stored [k][row] with pitch P, by two transposing reads:
// within each 16-lane group, lane i receives element i % 4 of the 8-byte
// chunk addressed by lane 4 q + i / 4 (q < 4).
template <int P>
__device__ __forceinline__ bf16x8_t frag_cols(const bf16_t* s, int m0, int k0, int lane) {
  const int g = lane >> 4, i = lane & 15;
  const bf16_t* p = s + (k0 + 8 * (g >> 1) + (i >> 2)) * P + m0 + 16 * (g & 1) + 4 * (i & 3);
  const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(p));
  const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(p + 4 * P));
  const u16x8_t v = {static_cast<uint16_t>(lo[0]), static_cast<uint16_t>(lo[1]), static_cast<uint16_t>(lo[2]),
                     static_cast<uint16_t>(lo[3]), static_cast<uint16_t>(hi[0]), static_cast<uint16_t>(hi[1]),
                     static_cast<uint16_t>(hi[2]), static_cast<uint16_t>(hi[3])};
  return __builtin_bit_cast(bf16x8_t, v);
}

__device__ __forceinline__ f32x16_t mfma(bf16x8_t b, bf16x8_t a, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, a, c, 0, 0, 0);
}

// A thread's four 16-byte vectors of a 128 x 64 bf16 block (rows ld apart in
// global memory) and their copy into an LDS tile [128][PD]. Loading several
// blocks before storing any makes their copies cost one round trip to
// memory rather than one per vector.
struct Rows4 {
  uint4 v0, v1, v2, v3;
};
static_assert(S * (DH / 8) == 4 * NT, "four 16-byte vectors per thread");

__device__ __forceinline__ uint4 row_vec(const bf16_t* src, long ld, int e) {
  return *reinterpret_cast<const uint4*>(src + (e >> 3) * ld + (e & 7) * 8);
}

__device__ __forceinline__ Rows4 stage_load(const bf16_t* src, long ld, int tid) {
  return Rows4{row_vec(src, ld, tid), row_vec(src, ld, tid + NT), row_vec(src, ld, tid + 2 * NT),
               row_vec(src, ld, tid + 3 * NT)};
}

__device__ __forceinline__ void stage_store(bf16_t* dst, const Rows4& r, int tid) {
  auto at = [&](int e) { return reinterpret_cast<uint4*>(dst + (e >> 3) * PD + (e & 7) * 8); };
  *at(tid) = r.v0;
  *at(tid + NT) = r.v1;
  *at(tid + 2 * NT) = r.v2;
  *at(tid + 3 * NT) = r.v3;
}

// Scores of the wave's 32 query rows against all 128 keys: acc[j] holds keys
// 32 j .. 32 j + 31. Q rows come from global memory (row stride ld), K from
// its staged LDS tile [128][PD].
__device__ __forceinline__ void scores_lds_k(const bf16_t* Qg, long ld, const bf16_t* Ks, int wave, int lane,
                                             f32x16_t (&acc)[4]) {
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.0f;
  const int kq = 8 * (lane >> 5);
#pragma unroll
  for (int kk = 0; kk < DH; kk += 16) {
    const bf16x8_t fq = gld8(Qg + (32 * wave + (lane & 31)) * ld + kk + kq);
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = mfma(frag_rows<PD>(Ks, 32 * j + (lane & 31), kk + kq), fq, acc[j]);
  }
}

// Column of register r of tile j for lane l: 32 j + 8 (r / 4) + 4 (l / 32) + r % 4.
__device__ __forceinline__ int col_of(int j, int r, int lane) { return 32 * j + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// Store a wave's 32 x 64 bf16 result (acc[0..1], columns 32 jn ..) scaled by alpha.
__device__ __forceinline__ void store_rows(bf16_t* out, long ld, int row0, const f32x16_t (&acc)[2], float alpha,
                                           int lane) {
  const int row = row0 + (lane & 31);
#pragma unroll
  for (int jn = 0; jn < 2; ++jn)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint32_t h[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) h[q] = f32_to_bf16(acc[jn][4 * g + q] * alpha);
      *reinterpret_cast<uint2*>(out + row * ld + col_of(jn, 4 * g, lane)) =
          make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
    }
}

__global__ __launch_bounds__(NT) void attention_fwd_kernel(const bf16_t* qkv, int heads, int d, float scale,
                                                           float* stats, bf16_t* ctx) {
  __shared__ __attribute__((aligned(16))) bf16_t Ps[S * PP];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[S * PD];
  __shared__ __attribute__((aligned(16))) bf16_t Ks[S * PD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x / heads, h = blockIdx.x - b * heads;
  const long ld = 3L * d;
  const bf16_t* Qg = qkv + static_cast<long>(b) * S * ld + h * DH;
  const bf16_t* Kg = Qg + d;
  {
    const Rows4 v = stage_load(Qg + 2 * d, ld, tid), k = stage_load(Kg, ld, tid);
    stage_store(Vs, v, tid);
    stage_store(Ks, k, tid);
  }
  __syncthreads();   // K staged: the scores read it from LDS

  f32x16_t acc[4];
  scores_lds_k(Qg, ld, Ks, wave, lane, acc);
  // row softmax: the row's scores are in this lane and lane ^ 32
  // (every operation of P's recomputation is written the same way in the
  // backward pass, with no multiply-add contraction, so both give equal bits)
  float m = -INFINITY;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      acc[j][r] = __fmul_rn(acc[j][r], scale);
      m = fmaxf(m, acc[j][r]);
    }
  m = fmaxf(m, __shfl_xor(m, 32));
  float sum = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      acc[j][r] = expf(__fsub_rn(acc[j][r], m));
      sum += acc[j][r];
    }
  sum += __shfl_xor(sum, 32);
  const float inv = 1.0f / sum;
  const int row = 32 * wave + (lane & 31);
  if (lane < 32) {
    float* st = stats + (static_cast<long>(blockIdx.x) * S + row) * 2;
    st[0] = m;
    st[1] = inv;
  }
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint32_t hb[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) hb[q] = f32_to_bf16(__fmul_rn(acc[j][4 * g + q], inv));
      *reinterpret_cast<uint2*>(Ps + row * PP + col_of(j, 4 * g, lane)) =
          make_uint2(hb[0] | (hb[1] << 16), hb[2] | (hb[3] << 16));
    }
  __syncthreads();
  // ctx rows = bf16(P) V: k runs over the 128 keys
  f32x16_t o[2];
#pragma unroll
  for (int jn = 0; jn < 2; ++jn)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[jn][r] = 0.0f;
#pragma unroll
  for (int kk = 0; kk < S; kk += 16) {
    const bf16x8_t fp = frag_rows<PP>(Ps, row, kk + 8 * (lane >> 5));
#pragma unroll
    for (int jn = 0; jn < 2; ++jn) o[jn] = mfma(frag_cols<PD>(Vs, 32 * jn, kk, lane), fp, o[jn]);
  }
  store_rows(ctx + static_cast<long>(b) * S * d + h * DH, d, 32 * wave, o, 1.0f, lane);
}

// LDS: bf16(P) (later dS), dO (later Q) and K, 72 KB, so two blocks share a CU.
__global__ __launch_bounds__(NT, 2) void attention_bwd_kernel(const bf16_t* qkv, const bf16_t* dctx, const float* stats,
                                                           int heads, int d, float scale, bf16_t* dqkv) {
  __shared__ __attribute__((aligned(16))) bf16_t Ps[S * PP];    // bf16(P), later dS
  __shared__ __attribute__((aligned(16))) bf16_t dOs[S * PD];   // dO, then Q once dV is formed
  __shared__ __attribute__((aligned(16))) bf16_t Ks[S * PD];
  bf16_t* const Qs = dOs;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x / heads, h = blockIdx.x - b * heads;
  const long ld = 3L * d;
  const bf16_t* Qg = qkv + static_cast<long>(b) * S * ld + h * DH;
  const bf16_t* Kg = Qg + d;
  const bf16_t* Vg = Qg + 2 * d;
  const bf16_t* dOg = dctx + static_cast<long>(b) * S * d + h * DH;
  bf16_t* dQg = dqkv + static_cast<long>(b) * S * ld + h * DH;
  {
    const Rows4 o = stage_load(dOg, d, tid), k = stage_load(Kg, ld, tid);
    stage_store(dOs, o, tid);
    stage_store(Ks, k, tid);
  }
  __syncthreads();   // K staged: the scores read it from LDS

  // P recomputed exactly as in the forward pass
  f32x16_t p[4];
  scores_lds_k(Qg, ld, Ks, wave, lane, p);
  const int row = 32 * wave + (lane & 31);
  const float* st = stats + (static_cast<long>(blockIdx.x) * S + row) * 2;
  const float m = st[0], inv = st[1];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) p[j][r] = __fmul_rn(expf(__fsub_rn(__fmul_rn(p[j][r], scale), m)), inv);
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint32_t hb[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) hb[q] = f32_to_bf16(p[j][4 * g + q]);
      *reinterpret_cast<uint2*>(Ps + row * PP + col_of(j, 4 * g, lane)) =
          make_uint2(hb[0] | (hb[1] << 16), hb[2] | (hb[3] << 16));
    }
  __syncthreads();   // dO, K and bf16(P) staged

  // dP = dO V^T for the wave's rows (V rows from global memory), then
  // dS = P * (dP - rowsum(P * dP)) kept in registers until P is consumed
  f32x16_t dp[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) dp[j][r] = 0.0f;
#pragma unroll
  for (int kk = 0; kk < DH; kk += 16) {
    const bf16x8_t fo = frag_rows<PD>(dOs, row, kk + 8 * (lane >> 5));
#pragma unroll
    for (int j = 0; j < 4; ++j) dp[j] = mfma(gld8(Vg + (32 * j + (lane & 31)) * ld + kk + 8 * (lane >> 5)), fo, dp[j]);
  }
  float dot = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) dot += p[j][r] * dp[j][r];
  dot += __shfl_xor(dot, 32);
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) dp[j][r] = p[j][r] * (dp[j][r] - dot);

  // dV rows (keys 32 w ..) = bf16(P)^T dO
  f32x16_t o[2];
#pragma unroll
  for (int jn = 0; jn < 2; ++jn)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[jn][r] = 0.0f;
#pragma unroll
  for (int kk = 0; kk < S; kk += 16) {
    const bf16x8_t fa = frag_cols<PP>(Ps, 32 * wave, kk, lane);
#pragma unroll
    for (int jn = 0; jn < 2; ++jn) o[jn] = mfma(frag_cols<PD>(dOs, 32 * jn, kk, lane), fa, o[jn]);
  }
  store_rows(dQg + 2 * d, ld, 32 * wave, o, 1.0f, lane);
  const Rows4 q = stage_load(Qg, ld, tid);
  __syncthreads();   // every wave has read bf16(P) and dO
  stage_store(Qs, q, tid);

#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint32_t hb[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) hb[q] = f32_to_bf16(dp[j][4 * g + q]);
      *reinterpret_cast<uint2*>(Ps + row * PP + col_of(j, 4 * g, lane)) =
          make_uint2(hb[0] | (hb[1] << 16), hb[2] | (hb[3] << 16));
    }
  __syncthreads();   // dS and Q staged

  // dQ rows (queries 32 w ..) = dS K * scale
#pragma unroll
  for (int jn = 0; jn < 2; ++jn)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[jn][r] = 0.0f;
#pragma unroll
  for (int kk = 0; kk < S; kk += 16) {
    const bf16x8_t fa = frag_rows<PP>(Ps, row, kk + 8 * (lane >> 5));
#pragma unroll
    for (int jn = 0; jn < 2; ++jn) o[jn] = mfma(frag_cols<PD>(Ks, 32 * jn, kk, lane), fa, o[jn]);
  }
  store_rows(dQg, ld, 32 * wave, o, scale, lane);

  // dK rows (keys 32 w ..) = dS^T Q * scale
#pragma unroll
  for (int jn = 0; jn < 2; ++jn)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[jn][r] = 0.0f;
#pragma unroll
  for (int kk = 0; kk < S; kk += 16) {
    const bf16x8_t fa = frag_cols<PP>(Ps, 32 * wave, kk, lane);
#pragma unroll
    for (int jn = 0; jn < 2; ++jn) o[jn] = mfma(frag_cols<PD>(Qs, 32 * jn, kk, lane), fa, o[jn]);
  }
  store_rows(dQg + d, ld, 32 * wave, o, scale, lane);
}

}  // namespace

bool attention_fused_supported(int seq, int head_dim, int d) {
  return seq == S && head_dim == DH && d % 8 == 0;
}

hipError_t attention_fwd(const bf16_t* qkv, int batch, int heads, int d, float scale, float* stats, bf16_t* ctx,
                         hipStream_t s) {
  if (!attention_fused_supported(S, d / heads, d) || d != heads * DH) return hipErrorInvalidValue;
  hipLaunchKernelGGL(attention_fwd_kernel, dim3(batch * heads), dim3(NT), 0, s, qkv, heads, d, scale, stats, ctx);
  return hipGetLastError();
}

hipError_t attention_bwd(const bf16_t* qkv, const bf16_t* dctx, const float* stats, int batch, int heads, int d,
                         float scale, bf16_t* dqkv, hipStream_t s) {
  if (!attention_fused_supported(S, d / heads, d) || d != heads * DH) return hipErrorInvalidValue;
  hipLaunchKernelGGL(attention_bwd_kernel, dim3(batch * heads), dim3(NT), 0, s, qkv, dctx, stats, heads, d, scale,
                     dqkv);
  return hipGetLastError();
}

}  // namespace spx
