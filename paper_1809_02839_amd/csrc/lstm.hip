// Fused recurrent steps of the residual LSTM layer on gfx950.
//
// Forward step t: z_t = zx_t + h_{t-1} W_h^T (zx_t: the input projection plus
// bias, computed for all steps by one GEMM beforehand), then the cell
//   i = sigmoid(z_i), f = sigmoid(z_f), g = tanh(z_g), o = sigmoid(z_o),
//   c_t = f c_{t-1} + i g,  h_t = o tanh(c_t).
// Backward step t: dh_t = dh_out_t + dz_{t+1} W_h (the recurrent gradient of
// step t+1), then the cell backward producing dz_t and dc_t.
//
// One launch per step: every step needs all of h_{t-1} (or dz_{t+1}), which
// the previous launch completes. Block b owns a slice of hidden units and all
// four gates of each, so the contraction and the cell of a unit run in the
// same block: the z (or dh) tile goes through LDS from the MFMA layout to one
// (row, unit) per thread. The contraction uses v_mfma_f32_16x16x32_bf16 with
// operands loaded straight from global memory (h or dz rows are shared by all
// blocks and stay in L2; each block's weight rows are re-read every step from
// its XCD's L2). A forward block covers 32 batch rows and 8 units (the tile
// shape that loads the fewest operand bytes per CU at 64 rows and 1024 units:
// 64 KB of h and 64 KB of weights), a backward block 16 rows and 16 units;
// the waves of a block split K, issue all their loads at once and add their
// partial tiles in a fixed order in LDS, so a step costs about one round of
// load latency.
#include "kernels.hpp"

namespace spx {
namespace {

constexpr int FWD_UNITS = 8;    // forward: 8 units x 4 gates = 32 z columns per block
constexpr int FWD_ROWS = 32;    // forward: batch rows per block
constexpr int FWD_WAVES = 8;    // forward: K = H split over 8 waves
constexpr int FWD_CHUNK = 4;    // forward: fragments per operand tile a wave loads before its MFMAs
constexpr int BWD_UNITS = 16;   // backward: 16 units of dh per block
constexpr int BWD_WAVES = 16;   // backward: K = 4H split over 16 waves
constexpr int CHUNK = 8;        // fragments a wave loads before its MFMAs

__device__ __forceinline__ bf16x8_t ld8(const bf16_t* p) {
  return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u16x8_t*>(p));
}

// One wave's share of a 16 x 16 tile: acc[r] = sum_k A[row][k] * Bm[col][k]
// over the 32-wide k fragments f = CHUNK (wave + WAVES j) + q (q < CHUNK) of
// K (a multiple of 32), where lane l supplies row l % 16 of A (arow) and
// column l % 16 of Bm (brow), both already offset by the lane's k quarter.
// Every chunk's loads are issued before its MFMAs, so a wave waits for one
// round of loads per chunk. Lane l ends with rows 4 (l / 16) + r of column
// l % 16 of its partial sum.
template <int WAVES>
__device__ __forceinline__ f32x4_t contract16(const bf16_t* arow, const bf16_t* brow, int K, int wave) {
  const int nf = K / 32;
  f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int f0 = wave * CHUNK; f0 < nf; f0 += WAVES * CHUNK) {
    bf16x8_t a[CHUNK], b[CHUNK];
#pragma unroll
    for (int q = 0; q < CHUNK; ++q)
      if (f0 + q < nf) {
        a[q] = ld8(arow + 32 * (f0 + q));
        b[q] = ld8(brow + 32 * (f0 + q));
      }
#pragma unroll
    for (int q = 0; q < CHUNK; ++q)
      if (f0 + q < nf) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[q], b[q], acc, 0, 0, 0);
  }
  return acc;
}

// One wave's share of a 32 x 32 tile as 2 x 2 tiles of 16 x 16, like
// contract16: arow[i] / brow[j] supply rows 16 i + l % 16 of A and 16 j + l % 16
// of Bm (already offset by the lane's k quarter). Each A and Bm fragment is
// loaded once for the two tiles that use it. Lane l ends with rows
// 16 i + 4 (l / 16) + r of column 16 j + l % 16 in acc[i][j][r].
template <int WAVES>
__device__ __forceinline__ void contract32(const bf16_t* const (&arow)[2], const bf16_t* const (&brow)[2], int K,
                                           int wave, f32x4_t (&acc)[2][2]) {
  const int nf = K / 32;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  for (int f0 = wave * FWD_CHUNK; f0 < nf; f0 += WAVES * FWD_CHUNK) {
    bf16x8_t a[2][FWD_CHUNK], b[2][FWD_CHUNK];
#pragma unroll
    for (int q = 0; q < FWD_CHUNK; ++q)
      if (f0 + q < nf) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          a[i][q] = ld8(arow[i] + 32 * (f0 + q));
          b[i][q] = ld8(brow[i] + 32 * (f0 + q));
        }
      }
#pragma unroll
    for (int q = 0; q < FWD_CHUNK; ++q)
      if (f0 + q < nf) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i][q], b[j][q], acc[i][j], 0, 0, 0);
      }
  }
}

// Sum the WAVES partial tiles in wave order into tile[16][17] (LDS).
template <int WAVES>
__device__ __forceinline__ void reduce_tile(const f32x4_t& acc, float (*red)[16][17], float (*tile)[17], int wave,
                                            int lane, int tid) {
#pragma unroll
  for (int r = 0; r < 4; ++r) red[wave][4 * (lane >> 4) + r][lane & 15] = acc[r];
  __syncthreads();
  if (tid < 256) {
    const int i = tid >> 4, j = tid & 15;
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) v += red[w][i][j];
    tile[i][j] = v;
  }
  __syncthreads();
}

// Block (bx, by): batch rows FWD_ROWS by .., units FWD_UNITS bx ..
__global__ __launch_bounds__(64 * FWD_WAVES) void lstm_step_fwd_kernel(const float* zx_t, const bf16_t* h_prev,
                                                                       const bf16_t* Wh, const float* c_prev, int B,
                                                                       int H, float* gates_t, float* c_t,
                                                                       bf16_t* h_t) {
  __shared__ float red[FWD_WAVES][FWD_ROWS][FWD_ROWS + 1];
  __shared__ float zs[FWD_ROWS][FWD_ROWS + 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int u0 = blockIdx.x * FWD_UNITS, r0 = blockIdx.y * FWD_ROWS;
  const long H4 = 4L * H;
  // the cell's own operands are loaded first so their latency overlaps the contraction
  const int crow = r0 + tid / FWD_UNITS, cuu = tid % FWD_UNITS, cu = u0 + cuu;
  const bool cell = tid < FWD_ROWS * FWD_UNITS && crow < B;
  float zx[4] = {0.0f, 0.0f, 0.0f, 0.0f}, cp = 0.0f;
  if (cell) {
#pragma unroll
    for (int g = 0; g < 4; ++g) zx[g] = zx_t[crow * H4 + g * H + cu];
    if (c_prev) cp = c_prev[static_cast<long>(crow) * H + cu];
  }
  if (h_prev) {
    // block column c = 4 unit + gate is the weight row gate * H + u0 + unit;
    // rows past B read row 0 (valid memory) and are never read back
    const int kq = 8 * (lane >> 4);
    const bf16_t* arow[2];
    const bf16_t* brow[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int row = r0 + 16 * i + (lane & 15), col = 16 * i + (lane & 15);
      arow[i] = h_prev + static_cast<long>(row < B ? row : 0) * H + kq;
      brow[i] = Wh + static_cast<long>((col & 3) * H + u0 + (col >> 2)) * H + kq;
    }
    f32x4_t acc[2][2];
    contract32<FWD_WAVES>(arow, brow, H, wave, acc);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[wave][16 * i + 4 * (lane >> 4) + r][16 * j + (lane & 15)] = acc[i][j][r];
    __syncthreads();
    // the partial tiles summed in wave order, two entries per thread
#pragma unroll
    for (int e = tid; e < FWD_ROWS * FWD_ROWS; e += 64 * FWD_WAVES) {
      const int i = e / FWD_ROWS, j = e % FWD_ROWS;
      float v = 0.0f;
#pragma unroll
      for (int w = 0; w < FWD_WAVES; ++w) v += red[w][i][j];
      zs[i][j] = v;
    }
    __syncthreads();
  }
  if (cell) {
    float z[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) z[g] = zx[g] + (h_prev ? zs[crow - r0][4 * cuu + g] : 0.0f);
    const float i = sigmoidf(z[0]), f = sigmoidf(z[1]), gg = tanhf(z[2]), o = sigmoidf(z[3]);
    const float cn = fmaf(f, cp, i * gg);
    float* gr = gates_t + crow * H4 + cu;
    gr[0] = i;
    gr[H] = f;
    gr[2 * H] = gg;
    gr[3 * H] = o;
    c_t[static_cast<long>(crow) * H + cu] = cn;
    h_t[static_cast<long>(crow) * H + cu] = f32_to_bf16(o * tanhf(cn));
  }
}

// Block (bx, by): batch rows 16 by .. 16 by + 15, units BWD_UNITS bx ..
__global__ __launch_bounds__(64 * BWD_WAVES) void lstm_step_bwd_kernel(const bf16_t* dz_next, const bf16_t* WhT,
                                                                       const bf16_t* dh_out, const float* gates_t,
                                                                       const float* c_t, const float* c_prev, int B,
                                                                       int H, float* dc, bf16_t* dz_t) {
  __shared__ float red[BWD_WAVES][16][17];
  __shared__ float dhs[16][17];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int u0 = blockIdx.x * BWD_UNITS, r0 = blockIdx.y * 16;
  const long H4 = 4L * H;
  // the cell's own operands are loaded first so their latency overlaps the contraction
  const int crow = r0 + tid / BWD_UNITS, cuu = tid % BWD_UNITS, cu = u0 + cuu;
  const bool cell = tid < 16 * BWD_UNITS && crow < B;
  const long t1 = static_cast<long>(crow) * H + cu;
  float gi = 0.0f, gf = 0.0f, gg = 0.0f, go = 0.0f, ct = 0.0f, cpv = 0.0f, dcv = 0.0f, dho = 0.0f;
  if (cell) {
    const float* gr = gates_t + crow * H4 + cu;
    gi = gr[0];
    gf = gr[H];
    gg = gr[2 * H];
    go = gr[3 * H];
    ct = c_t[t1];
    if (c_prev) cpv = c_prev[t1];
    dcv = dc[t1];
    dho = bf16_to_f32(dh_out[t1]);
  }
  if (dz_next) {
    // dh_rec[row][u0 + n] = sum_k dz_{t+1}[row][k] W_h[k][u0 + n] = sum_k dz[row][k] W_h^T[u0 + n][k]
    const int kq = 8 * (lane >> 4), row = r0 + (lane & 15);
    const bf16_t* arow = dz_next + static_cast<long>(row < B ? row : 0) * H4 + kq;
    const bf16_t* brow = WhT + static_cast<long>(u0 + (lane & 15)) * H4 + kq;
    reduce_tile<BWD_WAVES>(contract16<BWD_WAVES>(arow, brow, static_cast<int>(H4), wave), red, dhs, wave, lane, tid);
  }
  if (cell) {
    const float dh = dho + (dz_next ? dhs[crow - r0][cuu] : 0.0f);
    const float tc = tanhf(ct);
    const float d_o = dh * tc;
    const float dct = dcv + dh * go * (1.0f - tc * tc);
    const float di = dct * gg, dg = dct * gi, df = dct * cpv;
    dc[t1] = dct * gf;
    bf16_t* dr = dz_t + crow * H4 + cu;
    dr[0] = f32_to_bf16(di * gi * (1.0f - gi));
    dr[H] = f32_to_bf16(df * gf * (1.0f - gf));
    dr[2 * H] = f32_to_bf16(dg * (1.0f - gg * gg));
    dr[3 * H] = f32_to_bf16(d_o * go * (1.0f - go));
  }
}

// Y[c][r] = X[r][c] for X [R][C] bf16, R and C multiples of 32; 32 x 32 tiles
// through LDS (padded rows), 4 elements per thread.
__global__ __launch_bounds__(256) void transpose_bf16_kernel(const bf16_t* X, int R, int C, bf16_t* Y) {
  __shared__ bf16_t tile[32][34];
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;   // 32 x 8
  const int r0 = blockIdx.y * 32, c0 = blockIdx.x * 32;
#pragma unroll
  for (int j = 0; j < 32; j += 8) tile[ty + j][tx] = X[static_cast<long>(r0 + ty + j) * C + c0 + tx];
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 32; j += 8) Y[static_cast<long>(c0 + ty + j) * R + r0 + tx] = tile[tx][ty + j];
}

}  // namespace

bool lstm_step_supported(int B, int H) { return B >= 1 && B <= 64 && H >= 32 && H % 32 == 0; }

hipError_t lstm_step_fwd(const float* zx_t, const bf16_t* h_prev, const bf16_t* Wh, const float* c_prev, int B,
                         int H, float* gates_t, float* c_t, bf16_t* h_t, hipStream_t s) {
  if (!lstm_step_supported(B, H)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(lstm_step_fwd_kernel, dim3(H / FWD_UNITS, (B + FWD_ROWS - 1) / FWD_ROWS), dim3(64 * FWD_WAVES), 0, s, zx_t,
                     h_prev, Wh, c_prev, B, H, gates_t, c_t, h_t);
  return hipGetLastError();
}

hipError_t lstm_step_bwd(const bf16_t* dz_next, const bf16_t* WhT, const bf16_t* dh_out, const float* gates_t,
                         const float* c_t, const float* c_prev, int B, int H, float* dc, bf16_t* dz_t,
                         hipStream_t s) {
  if (!lstm_step_supported(B, H)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(lstm_step_bwd_kernel, dim3(H / BWD_UNITS, (B + 15) / 16), dim3(64 * BWD_WAVES), 0, s, dz_next,
                     WhT, dh_out, gates_t, c_t, c_prev, B, H, dc, dz_t);
  return hipGetLastError();
}

hipError_t transpose_bf16(const bf16_t* X, int R, int C, bf16_t* Y, hipStream_t s) {
  if (R % 32 || C % 32 || R <= 0 || C <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(transpose_bf16_kernel, dim3(C / 32, R / 32), dim3(256), 0, s, X, R, C, Y);
  return hipGetLastError();
}

}  // namespace spx
