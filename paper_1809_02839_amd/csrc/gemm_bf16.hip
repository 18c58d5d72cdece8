// bf16 GEMM on gfx950 matrix cores (v_mfma_f32_32x32x16_bf16), float32
// accumulation, used for every dense contraction of a stage: linear and 1x1
// layers, 3x3 convolutions as implicit GEMM (forward, data gradient, filter
// gradient) and the batched products inside attention.
//
// Block tile 128 x 128, K step 32, 256 threads = 4 waves in a 2 x 2 grid, each
// wave owning a 64 x 64 sub-tile (2 x 2 MFMA tiles of 32 x 32). Both operand
// tiles are staged in LDS as [row][k] with k contiguous, which is the layout
// the MFMA operand fetch wants (8 consecutive k per lane, one 16-byte
// ds_read). Two LDS buffers: the next K step's global loads are issued before
// the current step's MFMAs and written to the other buffer afterwards.
#include "kernels.hpp"

namespace spx {
namespace {

constexpr int BM = 128, BN = 128, BK = 32, NT = 256;
constexpr int PITCH = BK + 8;  // bf16 per LDS row: 80 bytes keeps 16-byte rows on distinct banks
constexpr int TILE_ELEMS = 128 * PITCH;

// LDS index of (row, k) inside one operand tile. The 16-byte chunk index is
// XOR-swizzled with row/8 so that the transposed 4-byte writes of R-mode
// operands do not all fall on one bank.
__device__ __forceinline__ int lds_idx(int row, int k) {
  return row * PITCH + (((k >> 3) ^ (row >> 3)) & 3) * 8 + (k & 7);
}

struct OperandDev {
  const bf16_t* p;
  long ld;
  int rows;        // extent of the row dimension (M for A, N for B)
  int K;
  int H, W, C, C2;
  FastDiv fdC, fdC2, fdHW, fdW;
};

__device__ __forceinline__ uint4 zero4() { return make_uint4(0, 0, 0, 0); }

// ---- K-mode: 8 consecutive k of one row ----------------------------------
template <int MODE>
struct KLoader {
  // per-thread, per-vector constant row info
  int row_ok[2];
  long row_base[2];   // PLAIN: row * ld; CONV: pixel index
  int ph[2], pw[2];   // CONV: pixel coordinates
  int kq[2];

  __device__ void init(const OperandDev& o, int row0, int tid) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      int v = tid + NT * i;
      int r = row0 + (v >> 2);
      kq[i] = v & 3;
      row_ok[i] = r < o.rows;
      if (MODE == OP_K_PLAIN) {
        row_base[i] = static_cast<long>(r) * o.ld;
      } else {
        row_base[i] = r;
        uint32_t rr = row_ok[i] ? r : 0;
        uint32_t b = o.fdHW.div(rr);
        uint32_t rem = rr - b * static_cast<uint32_t>(o.H * o.W);
        uint32_t h = o.fdW.div(rem);
        ph[i] = h;
        pw[i] = rem - h * o.W;
      }
    }
  }

  __device__ __forceinline__ void load(const OperandDev& o, int k0, uint4 (&reg)[2]) const {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      int k = k0 + kq[i] * 8;
      uint4 val = zero4();
      if (row_ok[i] && k < o.K) {
        if (MODE == OP_K_PLAIN) {
          val = *reinterpret_cast<const uint4*>(o.p + row_base[i] + k);
        } else {
          uint32_t tap = o.fdC.div(k);
          int c = k - static_cast<int>(tap) * o.C;
          int kh = (tap * 11) >> 5;  // tap / 3 for tap < 9
          int kw = tap - 3 * kh;
          int dh = (MODE == OP_K_CONV_FWD) ? kh - 1 : 1 - kh;
          int dw = (MODE == OP_K_CONV_FWD) ? kw - 1 : 1 - kw;
          int hh = ph[i] + dh, ww = pw[i] + dw;
          if (hh >= 0 && hh < o.H && ww >= 0 && ww < o.W) {
            long pix = row_base[i] + static_cast<long>(dh) * o.W + dw;
            val = *reinterpret_cast<const uint4*>(o.p + pix * o.C + c);
          }
        }
      }
      reg[i] = val;
    }
  }

  __device__ __forceinline__ void store(bf16_t* lds, const uint4 (&reg)[2], int tid) const {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      int v = tid + NT * i;
      *reinterpret_cast<uint4*>(lds + lds_idx(v >> 2, kq[i] * 8)) = reg[i];
    }
  }
};

// ---- R-mode: 8 consecutive rows of one k ----------------------------------
template <int MODE>
struct RLoader {
  int kp;        // this thread loads k = 2*kp and 2*kp + 1 of each K step
  int rg;        // row group: tile rows rg*8 .. rg*8+7
  int rows_ok;
  long col;      // PLAIN: first row index; WGRAD: channel c; FILTER_T: first row (c)
  int tap;       // WGRAD: filter tap of this row group

  __device__ void init(const OperandDev& o, int row0, int tid) {
    kp = tid & 15;
    rg = tid >> 4;
    int r = row0 + rg * 8;
    rows_ok = r < o.rows;   // rows are a multiple of 8
    if (MODE == OP_R_CONV_WGRAD) {
      uint32_t rr = rows_ok ? r : 0;
      tap = o.fdC.div(rr);
      col = rr - tap * o.C;
    } else {
      tap = 0;
      col = r;
    }
  }

  __device__ __forceinline__ uint4 fetch(const OperandDev& o, int k) const {
    if (!rows_ok || k >= o.K) return zero4();
    if (MODE == OP_R_PLAIN) {
      return *reinterpret_cast<const uint4*>(o.p + static_cast<long>(k) * o.ld + col);
    } else if (MODE == OP_R_CONV_WGRAD) {
      uint32_t b = o.fdHW.div(k);
      uint32_t rem = k - b * static_cast<uint32_t>(o.H * o.W);
      int h = o.fdW.div(rem);
      int w = rem - h * o.W;
      int kh = (tap * 11) >> 5, kw = tap - 3 * kh;
      int hh = h + kh - 1, ww = w + kw - 1;
      if (hh < 0 || hh >= o.H || ww < 0 || ww >= o.W) return zero4();
      long pix = static_cast<long>(k) + static_cast<long>(kh - 1) * o.W + (kw - 1);
      return *reinterpret_cast<const uint4*>(o.p + pix * o.C + col);
    } else {  // OP_R_FILTER_T: filter [C2][9][C], k = tap * C2 + c2
      uint32_t t = o.fdC2.div(k);
      int c2 = k - static_cast<int>(t) * o.C2;
      return *reinterpret_cast<const uint4*>(o.p + (static_cast<long>(c2) * 9 + t) * o.C + col);
    }
  }

  __device__ __forceinline__ void load(const OperandDev& o, int k0, uint4 (&reg)[2]) const {
    reg[0] = fetch(o, k0 + 2 * kp);
    reg[1] = fetch(o, k0 + 2 * kp + 1);
  }

  __device__ __forceinline__ void store(bf16_t* lds, const uint4 (&reg)[2], int) const {
    const uint32_t* a = reinterpret_cast<const uint32_t*>(&reg[0]);
    const uint32_t* b = reinterpret_cast<const uint32_t*>(&reg[1]);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      uint32_t lo = (j & 1) ? (a[j >> 1] >> 16) : (a[j >> 1] & 0xffffu);
      uint32_t hi = (j & 1) ? (b[j >> 1] >> 16) : (b[j >> 1] & 0xffffu);
      *reinterpret_cast<uint32_t*>(lds + lds_idx(rg * 8 + j, 2 * kp)) = lo | (hi << 16);
    }
  }
};

template <int MODE>
struct LoaderFor {
  using type = typename std::conditional<(MODE <= OP_K_CONV_DGRAD), KLoader<MODE>, RLoader<MODE>>::type;
};

struct EpiDev {
  float* out_f32;
  bf16_t* out_bf16;
  long ldc;
  const float* bias;
  const bf16_t* bias_bf16;
  const float* res_f32;
  const bf16_t* res_bf16;
  const bf16_t* mask;
  float alpha;
  int relu, accumulate;
};

struct KArgs {
  int M, N, K, zdiv, tiles_n, tiles_total;
  OperandDev A, B;
  long a_bs1, a_bs2, b_bs1, b_bs2, c_bs1, c_bs2;
  EpiDev e;
};

template <int MA, int MB>
__global__ __launch_bounds__(NT, 2) void gemm_bf16_kernel(KArgs args) {
  __shared__ __attribute__((aligned(16))) bf16_t lds[2][2][TILE_ELEMS];  // [buffer][A|B]

  const int tid = threadIdx.x;
  // XCD-aware tile order: hardware places consecutive blocks on consecutive
  // XCDs; renumber so each XCD receives a contiguous run of tiles (rows of
  // tiles sharing A rows then stay within one L2).
  int bid = blockIdx.x;
  int tile = bid;
  if ((args.tiles_total & 7) == 0) tile = (bid & 7) * (args.tiles_total >> 3) + (bid >> 3);
  const int tm = tile / args.tiles_n, tn = tile - tm * args.tiles_n;
  const int row0 = tm * BM, col0 = tn * BN;

  const int z = blockIdx.y;
  const int z1 = z / args.zdiv, z2 = z - z1 * args.zdiv;
  OperandDev A = args.A, B = args.B;
  A.p += z1 * args.a_bs1 + z2 * args.a_bs2;
  B.p += z1 * args.b_bs1 + z2 * args.b_bs2;
  const long coff = z1 * args.c_bs1 + z2 * args.c_bs2;

  typename LoaderFor<MA>::type la;
  typename LoaderFor<MB>::type lb;
  la.init(A, row0, tid);
  lb.init(B, col0, tid);

  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  uint4 ra[2], rb[2];
  const int nk = (args.K + BK - 1) / BK;
  la.load(A, 0, ra);
  lb.load(B, 0, rb);
  la.store(lds[0][0], ra, tid);
  lb.store(lds[0][1], rb, tid);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      la.load(A, (kt + 1) * BK, ra);
      lb.load(B, (kt + 1) * BK, rb);
    }
    const bf16_t* sa = lds[cur][0];
    const bf16_t* sb = lds[cur][1];
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      bf16x8_t fa[2], fb[2];
      const int kl = kk + (lane >> 5) * 8;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        u16x8_t t = *reinterpret_cast<const u16x8_t*>(sa + lds_idx(wm * 64 + i * 32 + (lane & 31), kl));
        fa[i] = __builtin_bit_cast(bf16x8_t, t);
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        u16x8_t t = *reinterpret_cast<const u16x8_t*>(sb + lds_idx(wn * 64 + j * 32 + (lane & 31), kl));
        fb[j] = __builtin_bit_cast(bf16x8_t, t);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      la.store(lds[cur ^ 1][0], ra, tid);
      lb.store(lds[cur ^ 1][1], rb, tid);
    }
    __syncthreads();
  }

  // Epilogue: lane holds column (lane % 32) and rows 8*(r/4) + 4*(lane/32) + r%4.
  const EpiDev& e = args.e;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = col0 + wn * 64 + j * 32 + (lane & 31);
      if (col >= args.N) continue;
      const float bias = e.bias ? e.bias[col] : (e.bias_bf16 ? bf16_to_f32(e.bias_bf16[col]) : 0.0f);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = row0 + wm * 64 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        if (row >= args.M) continue;
        const long idx = coff + static_cast<long>(row) * e.ldc + col;
        float v = acc[i][j][r] * e.alpha + bias;
        if (e.res_f32) v += e.res_f32[idx];
        if (e.res_bf16) v += bf16_to_f32(e.res_bf16[idx]);
        if (e.relu) v = fmaxf(v, 0.0f);
        if (e.out_f32) {
          if (e.accumulate) e.out_f32[idx] += v;
          else e.out_f32[idx] = v;
        }
        if (e.out_bf16) {
          bf16_t h = f32_to_bf16(v);
          if (e.mask && !(bf16_to_f32(e.mask[idx]) > 0.0f)) h = 0;
          e.out_bf16[idx] = h;
        }
      }
    }
  }
}

OperandDev make_operand(const Operand& o, int rows, int K) {
  OperandDev d{};
  d.p = static_cast<const bf16_t*>(o.ptr);
  d.ld = o.ld;
  d.rows = rows;
  d.K = K;
  d.H = o.g.H;
  d.W = o.g.W;
  d.C = o.g.C;
  d.C2 = o.g.C2;
  d.fdC = FastDiv(o.g.C > 0 ? o.g.C : 1);
  d.fdC2 = FastDiv(o.g.C2 > 0 ? o.g.C2 : 1);
  d.fdHW = FastDiv(o.g.H * o.g.W > 0 ? o.g.H * o.g.W : 1);
  d.fdW = FastDiv(o.g.W > 0 ? o.g.W : 1);
  return d;
}

template <int MA, int MB>
hipError_t launch(const KArgs& a, int batch, hipStream_t s) {
  dim3 grid(a.tiles_total, batch);
  hipLaunchKernelGGL((gemm_bf16_kernel<MA, MB>), grid, dim3(NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t gemm_bf16(const GemmDesc& d, hipStream_t s) {
  if (d.M <= 0 || d.N <= 0 || d.batch <= 0) return hipSuccess;
  KArgs a{};
  a.M = d.M;
  a.N = d.N;
  a.K = d.K;
  a.zdiv = d.zdiv > 0 ? d.zdiv : 1;
  a.tiles_n = (d.N + BN - 1) / BN;
  a.tiles_total = a.tiles_n * ((d.M + BM - 1) / BM);
  a.A = make_operand(d.A, d.M, d.K);
  a.B = make_operand(d.B, d.N, d.K);
  a.a_bs1 = d.A.bs1;
  a.a_bs2 = d.A.bs2;
  a.b_bs1 = d.B.bs1;
  a.b_bs2 = d.B.bs2;
  a.c_bs1 = d.epi.bs1;
  a.c_bs2 = d.epi.bs2;
  a.e.out_f32 = d.epi.out_f32;
  a.e.out_bf16 = d.epi.out_bf16;
  a.e.ldc = d.epi.ldc;
  a.e.bias = d.epi.bias;
  a.e.bias_bf16 = d.epi.bias_bf16;
  a.e.res_f32 = d.epi.res_f32;
  a.e.res_bf16 = d.epi.res_bf16;
  a.e.mask = static_cast<const bf16_t*>(d.epi.mask);
  a.e.alpha = d.epi.alpha;
  a.e.relu = d.epi.relu;
  a.e.accumulate = d.epi.accumulate;
  const int ma = d.A.mode, mb = d.B.mode;
  if (ma == OP_K_PLAIN && mb == OP_K_PLAIN) return launch<OP_K_PLAIN, OP_K_PLAIN>(a, d.batch, s);
  if (ma == OP_K_PLAIN && mb == OP_R_PLAIN) return launch<OP_K_PLAIN, OP_R_PLAIN>(a, d.batch, s);
  if (ma == OP_R_PLAIN && mb == OP_R_PLAIN) return launch<OP_R_PLAIN, OP_R_PLAIN>(a, d.batch, s);
  if (ma == OP_K_CONV_FWD && mb == OP_K_PLAIN) return launch<OP_K_CONV_FWD, OP_K_PLAIN>(a, d.batch, s);
  if (ma == OP_K_CONV_DGRAD && mb == OP_R_FILTER_T) return launch<OP_K_CONV_DGRAD, OP_R_FILTER_T>(a, d.batch, s);
  if (ma == OP_R_PLAIN && mb == OP_R_CONV_WGRAD) return launch<OP_R_PLAIN, OP_R_CONV_WGRAD>(a, d.batch, s);
  return hipErrorInvalidValue;
}

}  // namespace spx
