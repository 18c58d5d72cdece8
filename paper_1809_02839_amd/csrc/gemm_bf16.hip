// bf16 GEMM on gfx950 matrix cores (v_mfma_f32_32x32x16_bf16), float32
// accumulation, used for every dense contraction of a stage: linear and 1x1
// layers, 3x3 convolutions as implicit GEMM (forward, data gradient, filter
// gradient) and the batched products inside attention.
//
// Block tile 128 x 128 (or 128 x 64, see shape_of), K step 64, 256 threads =
// 4 waves in a 2 x 2 grid, each wave owning a 64 x 64 (64 x 32) sub-tile of
// 2 x 2 (2 x 1) MFMA tiles of 32 x 32; some convolution gathers (forward, and
// data gradient against a transposed filter) use 512 threads, two waves per
// sub-tile that share each K step. K-mode operand
// tiles are staged in LDS as [row][k] (8 consecutive k per lane make one
// 16-byte MFMA operand read; the 144-byte row pitch puts eight consecutive
// rows on disjoint banks); R-mode tiles (rows contiguous in memory) are staged
// as [k][row] as loaded, with the 16-byte units of each 256-byte k row
// permuted by an XOR with 4 (k mod 4), and transposed by the LDS reads. In
// the register-staged kernel (the 128 x 64 tiles) global loads run two K
// steps ahead of the MFMAs (two register stages, two LDS buffers). All
// global reads are
// buffer loads whose resource spans exactly the operand tensor: an offset
// outside it (zero padding of convolutions, ragged tile edges) reads zero.
//
// Direct loads (every 128-wide block, 4 or 8 waves): the buffer loads carry the LDS
// flag, so each lane's 16 bytes go straight into a two-stage LDS ring at the
// position fixed by its lane number, with no register stage and no LDS store
// instruction (LDS stores contend with the MFMA operand reads; direct loads
// measured beside LDS reads do not). The lanes' source addresses are
// permuted instead of the destinations: K-mode tiles become rows of 64 k
// without padding whose 16-byte chunks are XOR-swizzled by row pairs, R-mode
// tiles keep the layout above.
//
// Epilogue: an unsplit launch whose output rows allow 16-byte accesses
// stages its float32 tile in LDS and then gives each thread eight
// consecutive columns of a row, so the residual and mask loads and the output
// stores of a wave cover whole row segments (an output line is never written
// piecemeal, which had tripled the HBM write traffic of the bottleneck's
// 1x1 data gradient). Whole tiles whose epilogue has only bf16 operands run
// straight-line rows compiled for that operand set (the generic rows test
// every feature per group and issue about one instruction per ten cycles);
// bf16 rounding uses the conversion instruction. Other launches write from
// the MFMA layout, with every epilogue load of a lane issued before its
// first store.
//
// Split-K: a 128 x 128 launch may divide K into `splits` ranges; each writes
// float32 partial tiles to a workspace and an elementwise pass sums the
// partials in a fixed order and applies the epilogue, so results do not
// depend on timing.
#include <algorithm>
#include <cstdio>

#include "kernels.hpp"

namespace spx {
namespace {

constexpr int BM = 128, BN = 128, BK = 64, NT = 256;
constexpr int PITCH = BK + 8;            // K-mode tile [row][k]: bf16 per row (144 bytes)
constexpr int RPITCH = 128;              // R-mode tile [k][row]: bf16 per k row (256 bytes, swizzled)
constexpr int TILE_ELEMS = 128 * PITCH;  // one operand tile (K-mode; the R-mode tile needs BK * RPITCH)
static_assert(TILE_ELEMS >= BK * RPITCH, "both tile layouts fit one operand buffer");

// Element offset, inside a k row of an R-mode tile, of row (column) c: the
// 16-byte unit c / 8 is XORed with 4 (k mod 4). A transposing read covers
// four consecutive k rows at the same columns in each 16-lane group; the
// XOR spreads them over disjoint 64-byte bank ranges, where a common pitch
// would put the two groups of a half-wave on the same banks.
__device__ __forceinline__ int rcol(int k, int c) { return (((c >> 3) ^ ((k & 3) << 2)) << 3) | (c & 7); }
constexpr int BUF_FLAGS = 0x00020000;    // gfx9 raw buffer resource word 3
constexpr int OOB = 0x7ffffff0;          // byte offset past every resource: the load returns 0
constexpr int MAX_SPLITS = 16;           // K slices of one split-K launch

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

// MFMA operand (8 consecutive k of one row) from a K-mode tile [row][PITCH].
__device__ __forceinline__ bf16x8_t frag_k(const bf16_t* s, int row, int k) {
  return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u16x8_t*>(s + row * PITCH + k));
}

// The same operand from a K-mode tile filled by direct loads: rows of 64 k
// without padding, the eight 16-byte chunks of row r permuted by an XOR with
// (r / 2) % 8. Sixteen lanes reading one chunk of sixteen consecutive rows
// then hit every bank once (rows 2j and 2j + 1 share a slot but lie in
// different halves of the 64 banks).
__device__ __forceinline__ bf16x8_t frag_kd(const bf16_t* s, int row, int k) {
  return __builtin_bit_cast(
      bf16x8_t, *reinterpret_cast<const u16x8_t*>(s + row * BK + ((((k >> 3) ^ ((row >> 1) & 7))) << 3)));
}

// The same operand from an R-mode tile [k][RPITCH] with two transposing LDS
// reads (ds_read_b64_tr_b16). Within each group of 16 lanes, lane i receives
// element i % 4 of the 8-byte chunk addressed by lane 4 q + i / 4, for q < 4.
// Lane (group g, index i) therefore addresses k row k0 + 8 (g / 2) + i / 4 at
// rows m0 + 16 (g % 2) + 4 (i % 4): it receives rows m0 + 16 (g % 2) + i and
// k0 + 8 (g / 2) + q, which is the MFMA operand layout (row lane % 32, k half
// lane / 32). The second read takes the next four k.
__device__ __forceinline__ bf16x8_t frag_r(const bf16_t* s, int m0, int k0, int lane) {
  const int g = lane >> 4, i = lane & 15;
  const int k = k0 + 8 * (g >> 1) + (i >> 2);   // k + 4 (the second read) has the same swizzle
  const bf16_t* p = s + k * RPITCH + rcol(k, m0 + 16 * (g & 1) + 4 * (i & 3));
  const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(p));
  const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(p + 4 * RPITCH));
  const u16x8_t v = {static_cast<uint16_t>(lo[0]), static_cast<uint16_t>(lo[1]), static_cast<uint16_t>(lo[2]),
                     static_cast<uint16_t>(lo[3]), static_cast<uint16_t>(hi[0]), static_cast<uint16_t>(hi[1]),
                     static_cast<uint16_t>(hi[2]), static_cast<uint16_t>(hi[3])};
  return __builtin_bit_cast(bf16x8_t, v);
}

struct OperandDev {
  const bf16_t* p;
  long ld;
  long extent;     // elements addressable from p (batch 0)
  int rows;        // extent of the row dimension (M for A, N for B)
  int K;
  int H, W, C, C2;
  int step_h, step_w;   // WGRAD gather: BK pixels expressed as (rows, columns) inside an image
  FastDiv fdC, fdC2, fdHW, fdW;
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
  int M, N, K, zdiv, tiles_n, tiles_total, batch, splits, k_per_split;
  OperandDev A, B;
  long a_bs1, a_bs2, b_bs1, b_bs2, c_bs1, c_bs2;
  float* partial;        // splits > 1: [split][batch][M][N] float32
  int vec_epi;           // output, bias, residual and mask allow the four-column epilogue
  int vec8;              // ... and the eight-column one (N, ldc multiples of 8, 16-byte aligned tensors)
  int bn;                // block tile width in N (host side: selects the kernel)
  int ksl;               // waves per output sub-tile (host side: selects the kernel)
  int dma;               // operand tiles loaded directly into LDS (host side: selects the kernel)
  EpiDev e;
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const bf16_t* p, long elems) {
  long bytes = elems * 2;
  if (bytes > 0x7fffffe0L) bytes = 0x7fffffe0L;
  if (bytes < 0) bytes = 0;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(p), static_cast<short>(0), static_cast<int>(bytes),
                                           BUF_FLAGS);
}

__device__ __forceinline__ uint4 bload(__amdgpu_buffer_rsrc_t r, int byte_off) {
  u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Direct load into LDS: the 16 bytes of lane l land at LDS byte address
// lds_base + 16 l (lds_base wave-uniform, passed in M0); an offset outside
// the resource writes zeros. Issued through inline assembly so that the
// compiler, which cannot tell the stages of the LDS ring apart, does not wait
// for every outstanding direct load before each LDS read: the K loop waits
// for exactly the stage it reads (dma_wait) and then synchronises the block.
// The statement declares M0 clobbered; nothing else in these kernels keeps a
// value in M0 (a host test checks the assembly for it).
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, uint32_t lds_base, int byte_off) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" ::"s"(lds_base), "v"(byte_off), "s"(r)
               : "memory", "m0");
}
template <int N>
__device__ __forceinline__ void dma_wait() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// ---- K-mode: 8 consecutive k of one row ----------------------------------
// Thread t of NTH loads vectors v = t + NTH i (i < 8 ROWS / NTH): tile row
// v / 8, k chunk t % 8.
// TAPK (convolutions whose channel count is a multiple of BK): every K step
// lies inside one filter tap, so the tap and its pixel shift are uniform for
// the whole block and each vector costs one add and a bounds check.
template <int MODE, bool TAPK, int ROWS, int NTH, bool DMA = false>
struct KLoader {
  static constexpr int V = 8 * ROWS / NTH;   // 16-byte vectors per thread
  static_assert(!DMA || NTH % 128 == 0, "the direct-load chunk permutation assumes 16 | NTH / 8");
  int row_ok[4];
  int base[4];       // byte offset of the row (PLAIN) or of the pixel's channel 0 (CONV)
  int ph[4], pw[4];  // CONV: pixel coordinates
  int kq8;           // this thread's k offset inside a K step

  __device__ void init(const OperandDev& o, int row0, int tid, int /*k0*/) {
    // DMA: vector t + NTH i lands in LDS slot t % 8 of its row, which holds
    // k chunk slot ^ ((row / 2) % 8) (see frag_kd); row / 2 % 8 = t / 16 % 8
    kq8 = DMA ? (((tid & 7) ^ ((tid >> 4) & 7)) * 8) : (tid & 7) * 8;
#pragma unroll
    for (int i = 0; i < V; ++i) {
      const int r = row0 + ((tid + NTH * i) >> 3);
      row_ok[i] = r < o.rows;
      const uint32_t rr = row_ok[i] ? r : 0;
      if (MODE == OP_K_PLAIN) {
        base[i] = static_cast<int>(rr * o.ld * 2);
      } else {
        const uint32_t b = o.fdHW.div(rr);
        const uint32_t rem = rr - b * static_cast<uint32_t>(o.H * o.W);
        const uint32_t h = o.fdW.div(rem);
        ph[i] = h;
        pw[i] = rem - h * o.W;
        base[i] = static_cast<int>(rr) * o.C * 2;
      }
    }
  }

  // Byte offset (OOB for zero padding) of each of the thread's V vectors of
  // the K step starting at k0, handed to f(i, offset).
  template <class F>
  __device__ __forceinline__ void visit(const OperandDev& o, int k0, F&& f) {
    const int k = k0 + kq8;
    const bool kok = k < o.K;
    if (MODE == OP_K_PLAIN) {
#pragma unroll
      for (int i = 0; i < V; ++i) f(i, (row_ok[i] & kok) ? base[i] + k * 2 : OOB);
    } else if (TAPK) {
      const int tap = static_cast<int>(o.fdC.div(k0));     // uniform
      const int kh = (tap * 11) >> 5, kw = tap - 3 * kh;
      const int dh = (MODE == OP_K_CONV_FWD) ? kh - 1 : 1 - kh;
      const int dw = (MODE == OP_K_CONV_FWD) ? kw - 1 : 1 - kw;
      const int shift = ((dh * o.W + dw) * o.C + (k0 - tap * o.C) + kq8) * 2;
#pragma unroll
      for (int i = 0; i < V; ++i) {
        const int hh = ph[i] + dh, ww = pw[i] + dw;
        const bool ok = row_ok[i] & (static_cast<unsigned>(hh) < static_cast<unsigned>(o.H)) &
                        (static_cast<unsigned>(ww) < static_cast<unsigned>(o.W));
        f(i, ok ? base[i] + shift : OOB);
      }
    } else {
      const uint32_t tap = o.fdC.div(kok ? k : 0);
      const int c = k - static_cast<int>(tap) * o.C;
      const int kh = (tap * 11) >> 5;  // tap / 3 for tap < 9
      const int kw = tap - 3 * kh;
      const int dh = (MODE == OP_K_CONV_FWD) ? kh - 1 : 1 - kh;
      const int dw = (MODE == OP_K_CONV_FWD) ? kw - 1 : 1 - kw;
      const int shift = ((dh * o.W + dw) * o.C + c) * 2;
#pragma unroll
      for (int i = 0; i < V; ++i) {
        const int hh = ph[i] + dh, ww = pw[i] + dw;
        const bool ok = row_ok[i] & kok & (static_cast<unsigned>(hh) < static_cast<unsigned>(o.H)) &
                        (static_cast<unsigned>(ww) < static_cast<unsigned>(o.W));
        f(i, ok ? base[i] + shift : OOB);
      }
    }
  }

  __device__ __forceinline__ void load(const OperandDev& o, __amdgpu_buffer_rsrc_t rs, int k0, uint4 (&reg)[4]) {
    visit(o, k0, [&](int i, int off) { reg[i] = bload(rs, off); });
  }

  // DMA: vector i of wave w's lanes lands at tile byte 16 (64 w + NTH i) + 16 lane
  __device__ __forceinline__ void dma(const OperandDev& o, __amdgpu_buffer_rsrc_t rs, int k0, uint32_t tile,
                                      int wave) {
    visit(o, k0, [&](int i, int off) { dma16(rs, tile + 16u * (64 * wave + NTH * i), off); });
  }

  __device__ __forceinline__ void store(bf16_t* lds, const uint4 (&reg)[4], int tid) const {
#pragma unroll
    for (int i = 0; i < V; ++i) {
      const int v = tid + NTH * i;
      *reinterpret_cast<uint4*>(lds + (v >> 3) * PITCH + (v & 7) * 8) = reg[i];
    }
  }
};

// ---- R-mode: 8 consecutive rows of one k ----------------------------------
// The tile is kept in LDS as [k][row] (rows contiguous, RPITCH elements per k)
// exactly as loaded, and the MFMA operand reads transpose it (see frag_r).
// With G = ROWS / 8 row groups, thread t of NTH loads row group t % G (rows
// 8 (t % G) .. + 7) at k = k0 + t / G + (NTH / G) i (i < BK G / NTH): G lanes
// cover one k row of the tile. Loads must be issued for consecutive K steps
// (the filter-gradient gather advances its pixel coordinates by BK per call).
template <int MODE, bool TAPK, int ROWS, int NTH, bool DMA = false>
struct RLoader {
  static constexpr int G = ROWS / 8, KS = NTH / G, V = BK / KS;
  static_assert(!DMA || (G == 16 && NTH % 64 == 0), "direct loads fill 256-byte k rows of 128-row tiles");
  int rows_ok;
  int colb;      // byte offset of the row group (PLAIN, FILTER_T) or of its channel + tap shift (WGRAD)
  int tkh, tkw;  // WGRAD: filter tap of the row group
  int kk0;       // t / G
  int h[4], w[4];

  __device__ void init(const OperandDev& o, int row0, int tid, int k0) {
    kk0 = tid / G;
    // DMA: vector t + NTH i lands in unit slot t % 16 of its k row, which
    // holds row group slot ^ 4 (k % 4) (rcol); k % 4 = t / 16 % 4
    const int grp = DMA ? ((tid & 15) ^ (((tid >> 4) & 3) << 2)) : tid % G;
    const int r = row0 + grp * 8;
    rows_ok = r < o.rows;  // rows are a multiple of 8
    const uint32_t rr = rows_ok ? r : 0;
    tkh = tkw = 0;
    if (MODE == OP_R_CONV_WGRAD) {
      const int tap = static_cast<int>(o.fdC.div(rr));
      tkh = (tap * 11) >> 5;
      tkw = tap - 3 * tkh;
      colb = (((tkh - 1) * o.W + (tkw - 1)) * o.C + static_cast<int>(rr) - tap * o.C) * 2;
#pragma unroll
      for (int i = 0; i < V; ++i) {
        const uint32_t kk = k0 + kk0 + KS * i;
        const uint32_t b = o.fdHW.div(kk);
        const uint32_t rem = kk - b * static_cast<uint32_t>(o.H * o.W);
        h[i] = o.fdW.div(rem);
        w[i] = rem - h[i] * o.W;
      }
    } else {
      colb = static_cast<int>(rr) * 2;
    }
  }

  // Byte offsets of the thread's V vectors of the K step starting at k0
  // (called once per K step, in order: the filter-gradient gather advances
  // its pixel coordinates by BK per call).
  template <class F>
  __device__ __forceinline__ void visit(const OperandDev& o, int k0, F&& f) {
    int t0 = 0, c0 = 0;
    if (MODE == OP_R_FILTER_T && TAPK) {
      t0 = static_cast<int>(o.fdC2.div(k0));  // uniform
      c0 = k0 - t0 * o.C2;
    }
#pragma unroll
    for (int i = 0; i < V; ++i) {
      const int k = k0 + kk0 + KS * i;
      const bool kok = rows_ok & (k < o.K);
      if (MODE == OP_R_PLAIN) {
        f(i, kok ? static_cast<int>(k * o.ld * 2) + colb : OOB);
      } else if (MODE == OP_R_CONV_WGRAD) {
        const int hh = h[i] + tkh - 1, ww = w[i] + tkw - 1;
        const bool ok = kok & (static_cast<unsigned>(hh) < static_cast<unsigned>(o.H)) &
                        (static_cast<unsigned>(ww) < static_cast<unsigned>(o.W));
        f(i, ok ? k * o.C * 2 + colb : OOB);
        // advance this k by one K step (BK pixels) inside its image
        w[i] += o.step_w;
        const int cw = w[i] >= o.W;
        w[i] -= cw ? o.W : 0;
        h[i] += o.step_h + cw;
        h[i] -= h[i] >= o.H ? o.H : 0;
      } else {  // OP_R_FILTER_T: filter [C2][9][C], k = tap * C2 + c2
        int t, c2;
        if (TAPK) {
          t = t0;
          c2 = c0 + kk0 + KS * i;
        } else {
          t = static_cast<int>(o.fdC2.div(k < o.K ? k : 0));
          c2 = k - t * o.C2;
        }
        f(i, kok ? (c2 * 9 + t) * o.C * 2 + colb : OOB);
      }
    }
  }

  __device__ __forceinline__ void load(const OperandDev& o, __amdgpu_buffer_rsrc_t rs, int k0, uint4 (&reg)[4]) {
    visit(o, k0, [&](int i, int off) { reg[i] = bload(rs, off); });
  }

  __device__ __forceinline__ void dma(const OperandDev& o, __amdgpu_buffer_rsrc_t rs, int k0, uint32_t tile,
                                      int wave) {
    visit(o, k0, [&](int i, int off) { dma16(rs, tile + 16u * (64 * wave + NTH * i), off); });
  }

  __device__ __forceinline__ void store(bf16_t* lds, const uint4 (&reg)[4], int tid) const {
#pragma unroll
    for (int i = 0; i < V; ++i) {
      const int k = tid / G + KS * i;
      *reinterpret_cast<uint4*>(lds + k * RPITCH + rcol(k, (tid % G) * 8)) = reg[i];
    }
  }
};

template <int MODE, bool TAPK, int ROWS, int NTH, bool DMA = false>
struct LoaderFor {
  using type = typename std::conditional<(MODE <= OP_K_CONV_DGRAD), KLoader<MODE, TAPK, ROWS, NTH, DMA>,
                                         RLoader<MODE, TAPK, ROWS, NTH, DMA>>::type;
};

// value = acc * alpha + bias + residuals, ReLU, then float32 and/or bf16 stores
// (the bf16 store is zeroed where the mask is not positive).
__device__ __forceinline__ void epilogue(const EpiDev& e, long idx, int col, float acc) {
  float v = acc * e.alpha;
  if (e.bias) v += e.bias[col];
  else if (e.bias_bf16) v += bf16_to_f32(e.bias_bf16[col]);
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

// The epilogue for four consecutive columns of one row with vector loads and
// stores; needs idx and col multiples of 4 and 16-byte aligned float32 (8-byte
// aligned bf16) tensors, which the host checks.
__device__ __forceinline__ void epilogue4(const EpiDev& e, long idx, int col, float4 a) {
  float v[4] = {a.x, a.y, a.z, a.w};
  if (e.alpha != 1.0f) {
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] *= e.alpha;
  }
  auto unpack = [](uint2 u, float (&f)[4]) {
    f[0] = bf16_to_f32(static_cast<bf16_t>(u.x & 0xffff));
    f[1] = bf16_to_f32(static_cast<bf16_t>(u.x >> 16));
    f[2] = bf16_to_f32(static_cast<bf16_t>(u.y & 0xffff));
    f[3] = bf16_to_f32(static_cast<bf16_t>(u.y >> 16));
  };
  float t[4];
  if (e.bias) {
    const float4 b = *reinterpret_cast<const float4*>(e.bias + col);
    v[0] += b.x; v[1] += b.y; v[2] += b.z; v[3] += b.w;
  } else if (e.bias_bf16) {
    unpack(*reinterpret_cast<const uint2*>(e.bias_bf16 + col), t);
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] += t[q];
  }
  if (e.res_f32) {
    const float4 r = *reinterpret_cast<const float4*>(e.res_f32 + idx);
    v[0] += r.x; v[1] += r.y; v[2] += r.z; v[3] += r.w;
  }
  if (e.res_bf16) {
    unpack(*reinterpret_cast<const uint2*>(e.res_bf16 + idx), t);
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] += t[q];
  }
  if (e.relu) {
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = fmaxf(v[q], 0.0f);
  }
  if (e.out_f32) {
    float4* o = reinterpret_cast<float4*>(e.out_f32 + idx);
    if (e.accumulate) {
      const float4 old = *o;
      v[0] += old.x; v[1] += old.y; v[2] += old.z; v[3] += old.w;
    }
    *o = make_float4(v[0], v[1], v[2], v[3]);
  }
  if (e.out_bf16) {
    if (e.mask) {
      unpack(*reinterpret_cast<const uint2*>(e.mask + idx), t);
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] = t[q] > 0.0f ? v[q] : 0.0f;
    }
    *reinterpret_cast<uint2*>(e.out_bf16 + idx) = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
  }
}

// The epilogue values of four consecutive columns with the bf16 bias,
// residual and mask already loaded (bb, rb, mk: four bf16 each; read only
// where the epilogue has that operand): stores the float32 output if there
// is one and returns the four bf16 results (zero where the mask is not
// positive).
__device__ __forceinline__ uint2 epilogue4_values(const EpiDev& e, long idx, int col, float4 a, uint2 bb, uint2 rb,
                                                  uint2 mk) {
  float v[4] = {a.x, a.y, a.z, a.w};
  if (e.alpha != 1.0f) {
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] *= e.alpha;
  }
  auto unpack = [](uint2 u, float (&f)[4]) {
    f[0] = bf16_to_f32(static_cast<bf16_t>(u.x & 0xffff));
    f[1] = bf16_to_f32(static_cast<bf16_t>(u.x >> 16));
    f[2] = bf16_to_f32(static_cast<bf16_t>(u.y & 0xffff));
    f[3] = bf16_to_f32(static_cast<bf16_t>(u.y >> 16));
  };
  float t[4];
  if (e.bias) {
    const float4 b = *reinterpret_cast<const float4*>(e.bias + col);
    v[0] += b.x; v[1] += b.y; v[2] += b.z; v[3] += b.w;
  } else if (e.bias_bf16) {
    unpack(bb, t);
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] += t[q];
  }
  if (e.res_f32) {
    const float4 r = *reinterpret_cast<const float4*>(e.res_f32 + idx);
    v[0] += r.x; v[1] += r.y; v[2] += r.z; v[3] += r.w;
  }
  if (e.res_bf16) {
    unpack(rb, t);
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] += t[q];
  }
  if (e.relu) {
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = fmaxf(v[q], 0.0f);
  }
  if (e.out_f32) {
    float4* o = reinterpret_cast<float4*>(e.out_f32 + idx);
    if (e.accumulate) {
      const float4 old = *o;
      v[0] += old.x; v[1] += old.y; v[2] += old.z; v[3] += old.w;
    }
    *o = make_float4(v[0], v[1], v[2], v[3]);
  }
  if (e.mask) {
    unpack(mk, t);
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = t[q] > 0.0f ? v[q] : 0.0f;
  }
  return make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
}

// epilogue4 with the bf16 operands already loaded (see epilogue4_values).
__device__ __forceinline__ void epilogue4_pre(const EpiDev& e, long idx, int col, float4 a, uint2 bb, uint2 rb,
                                              uint2 mk) {
  const uint2 h = epilogue4_values(e, idx, col, a, bb, rb, mk);
  if (e.out_bf16) *reinterpret_cast<uint2*>(e.out_bf16 + idx) = h;
}

// Stores a block's 128 x 128 accumulator tile: float32 partials of its K
// split, or the epilogue into the outputs.
template <int NJ>
__device__ __forceinline__ void write_tile(const KArgs& args, f32x16_t (&acc)[2][NJ], int row0, int col0, int wm,
                                           int wn, int lane, int split, int z, int z1, int z2) {
  // With B as the first MFMA operand, lane l holds row (l % 32) and columns
  // 8 (r / 4) + 4 (l / 32) + r % 4 of each 32 x 32 tile: four consecutive
  // columns per register group.
  if (args.splits > 1) {
    float* part = args.partial + (static_cast<long>(split) * args.batch + z) * args.M * args.N;
    const bool vec = (args.N & 3) == 0;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int row = row0 + wm * 64 + i * 32 + (lane & 31);
        if (row >= args.M) continue;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int col = col0 + wn * (32 * NJ) + j * 32 + 8 * g + 4 * (lane >> 5);
          float* o = part + static_cast<long>(row) * args.N + col;
          if (vec && col + 3 < args.N) {
            *reinterpret_cast<float4*>(o) =
                make_float4(acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
          } else {
#pragma unroll
            for (int q = 0; q < 4; ++q)
              if (col + q < args.N) o[q] = acc[i][j][4 * g + q];
          }
        }
      }
    return;
  }
  const long coff = z1 * args.c_bs1 + z2 * args.c_bs2;
  const EpiDev& e = args.e;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int row = row0 + wm * 64 + i * 32 + (lane & 31);
    if (row >= args.M) continue;
    // The bf16 epilogue operands (bias, residual, ReLU mask) of this lane's
    // 4 NJ column groups are all loaded before the first store: the output
    // may alias nothing the compiler can prove, so a load issued after a
    // store waits for it, and one memory round trip per group would
    // serialise the epilogue. Loading first is exact also for an output
    // that overwrites its own residual element by element.
    uint2 bb[NJ][4], rb[NJ][4], mk[NJ][4];
    if (args.vec_epi) {
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int col = col0 + wn * (32 * NJ) + j * 32 + 8 * g + 4 * (lane >> 5);
          const long idx = coff + static_cast<long>(row) * e.ldc + col;
          const bool ok = col + 3 < args.N;
          bb[j][g] = rb[j][g] = mk[j][g] = make_uint2(0, 0);
          if (ok && !e.bias && e.bias_bf16) bb[j][g] = *reinterpret_cast<const uint2*>(e.bias_bf16 + col);
          if (ok && e.res_bf16) rb[j][g] = *reinterpret_cast<const uint2*>(e.res_bf16 + idx);
          if (ok && e.mask) mk[j][g] = *reinterpret_cast<const uint2*>(e.mask + idx);
        }
    }
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int col = col0 + wn * (32 * NJ) + j * 32 + 8 * g + 4 * (lane >> 5);
        const long idx = coff + static_cast<long>(row) * e.ldc + col;
        const float4 v = make_float4(acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
        if (args.vec_epi && col + 3 < args.N) {
          epilogue4_pre(e, idx, col, v, bb[j][g], rb[j][g], mk[j][g]);
        } else {
          if (col < args.N) epilogue(e, idx, col, v.x);
          if (col + 1 < args.N) epilogue(e, idx + 1, col + 1, v.y);
          if (col + 2 < args.N) epilogue(e, idx + 2, col + 2, v.z);
          if (col + 3 < args.N) epilogue(e, idx + 3, col + 3, v.w);
        }
      }
    }
  }
}

// The bf16 operands of the staged epilogue (below) for one thread: the bias
// of its 8 columns and the residual and mask of its NP row segments (8
// columns each, rows erl + RPP p of the tile).
template <int BNT, int NTH>
struct EpiOperands {
  static constexpr int TPR = BNT / 8;   // threads per row
  static constexpr int RPP = NTH / TPR; // rows per pass
  static constexpr int NP = 128 / RPP;  // rows per thread
  uint4 bb, rb[NP], mk[NP];

  __device__ __forceinline__ void load(const KArgs& args, int row0, int col0, int tid, long coff) {
    const EpiDev& e = args.e;
    const int ecol = col0 + (tid % TPR) * 8, erl = tid / TPR;
    const bool colok = ecol < args.N;
    bb = make_uint4(0, 0, 0, 0);
    if (colok && !e.bias && e.bias_bf16) bb = *reinterpret_cast<const uint4*>(e.bias_bf16 + ecol);
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const int row = row0 + erl + p * RPP;
      const long idx = coff + static_cast<long>(row) * e.ldc + ecol;
      rb[p] = mk[p] = make_uint4(0, 0, 0, 0);
      if (colok && row < args.M) {
        if (e.res_bf16) rb[p] = *reinterpret_cast<const uint4*>(e.res_bf16 + idx);
        if (e.mask) mk[p] = *reinterpret_cast<const uint4*>(e.mask + idx);
      }
    }
  }
};

// The staged epilogue's rows for one combination of bf16 operands known at
// compile time (bias, residual, ReLU, mask; alpha 1, no float32 output) on a
// tile inside the output: straight-line code whose NP rows the compiler can
// interleave. The operations and their order are those of epilogue4_values,
// so both paths give the same bits.
template <int BNT, int NTH, bool BIAS, bool RES, bool RELU, bool MASK>
__device__ __forceinline__ void staged_rows(const EpiDev& e, const float* tile, const EpiOperands<BNT, NTH>& eop,
                                            bf16_t* out, int ecl, int erl) {
  constexpr int EP = BNT + 4, RPP = EpiOperands<BNT, NTH>::RPP, NP = EpiOperands<BNT, NTH>::NP;
  auto unpack8 = [](uint4 u, float (&f)[8]) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      f[2 * q] = __uint_as_float(w[q] << 16);
      f[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);
    }
  };
  float bias[8];
  if constexpr (BIAS) unpack8(eop.bb, bias);
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int rr = erl + p * RPP;
    const float4 a0 = *reinterpret_cast<const float4*>(tile + rr * EP + ecl);
    const float4 a1 = *reinterpret_cast<const float4*>(tile + rr * EP + ecl + 4);
    float v[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
    if constexpr (BIAS) {
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] += bias[q];
    }
    if constexpr (RES) {
      float r[8];
      unpack8(eop.rb[p], r);
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] += r[q];
    }
    if constexpr (RELU) {
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = fmaxf(v[q], 0.0f);
    }
    if constexpr (MASK) {
      float m[8];
      unpack8(eop.mk[p], m);
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = m[q] > 0.0f ? v[q] : 0.0f;
    }
    *reinterpret_cast<uint4*>(out + static_cast<long>(rr) * e.ldc) =
        make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7]));
  }
}

// BNT: block tile width in N (128, or 64 for launches whose 128-wide tiles
// cannot give every CU two blocks); each wave owns 64 x (BNT / 2).
// KSL: waves per output sub-tile. With KSL = 2 (8 waves, 128-wide tiles
// only) waves w and w + 4 own the same sub-tile and take the first and the
// second half of every K step; their accumulators are added through LDS at
// the end (first half + second half), so one block per CU keeps two waves
// on every SIMD without the narrow tile's extra operand traffic.
// DMA (128-wide tiles, 4- or 8-wave blocks): the operand tiles go from
// global memory straight into a two-stage LDS ring (buffer loads with the
// LDS flag), with no register stage and no LDS store instruction; a stage is
// read after its own loads are counted complete and the block has
// synchronised. A wave that issues its share of a stage's direct loads
// waits for the memory pipeline to accept them, about as long as its MFMAs
// of a K step take; on 8-wave blocks the two waves of a SIMD issue half as
// many loads each and one multiplies while the other waits.
template <int MA, int MB, bool TAPK, int BNT, int KSL, bool DMA = false>
__global__ __launch_bounds__(NT * KSL, 2) void gemm_bf16_kernel(KArgs args) {
  constexpr int NJ = BNT / 64;   // 32-column MFMA tiles per wave
  constexpr int NTH = NT * KSL;
  constexpr int KW = BK / KSL;   // k of each K step that one wave multiplies
  static_assert(KSL == 1 || BNT == 128, "K-sliced waves use the 128-wide tile");
  static_assert(!DMA || BNT == 128, "direct loads serve the 128-wide tile");
  static_assert(KSL == 1 || DMA, "8-wave blocks load their operands directly");
  __shared__ __attribute__((aligned(16))) bf16_t lds[2][2][TILE_ELEMS];  // [buffer][A|B]

  const int tid = threadIdx.x;
  // XCD-aware tile order: consecutive blocks land on consecutive XCDs; give
  // each XCD a contiguous run of tiles (tiles sharing A rows share an L2).
  // A launch of batch x split slices enumerates (slice, tile) slice-major;
  // each XCD takes a contiguous run of that order, so an XCD works on the
  // same K slice (and batch entry) of neighbouring tiles and reads each
  // slice of both operands once, instead of every XCD fetching the operand
  // shared by its tiles for every slice.
  const int bid = blockIdx.x;
  int tile = bid, zs = blockIdx.y;
  const int blocks = gridDim.x * gridDim.y;
  if ((blocks & 7) == 0) {
    const int lin = blockIdx.y * gridDim.x + bid;
    const int ord = (lin & 7) * (blocks >> 3) + (lin >> 3);
    zs = ord / args.tiles_total;
    tile = ord - zs * args.tiles_total;
  } else if ((args.tiles_total & 7) == 0) {
    tile = (bid & 7) * (args.tiles_total >> 3) + (bid >> 3);
  }
  const int tm = tile / args.tiles_n, tn = tile - tm * args.tiles_n;
  const int row0 = tm * BM, col0 = tn * BNT;

  const int z = zs / args.splits, split = zs - z * args.splits;
  const int z1 = z / args.zdiv, z2 = z - z1 * args.zdiv;
  OperandDev A = args.A, B = args.B;
  const long aoff = z1 * args.a_bs1 + z2 * args.a_bs2, boff = z1 * args.b_bs1 + z2 * args.b_bs2;
  A.p += aoff;
  B.p += boff;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(A.p, A.extent - aoff);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(B.p, B.extent - boff);

  const int kbeg = split * args.k_per_split;
  const int kend = min(args.K, kbeg + args.k_per_split);
  const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;

  typename LoaderFor<MA, TAPK, BM, NTH, DMA>::type la;
  typename LoaderFor<MB, TAPK, BNT, NTH, DMA>::type lb;
  la.init(A, row0, tid, kbeg);
  lb.init(B, col0, tid, kbeg);

  // The staged epilogue's operands do not depend on the product: the
  // direct-load 4-wave kernels, which hold no operand tiles in registers,
  // issue their loads before the first K step so that they arrive while the
  // block multiplies (the register-staged loop, and the 8-wave blocks with
  // half the registers per wave, have none to spare for them and load them
  // in the epilogue). Issued before the first direct loads, they are older
  // than every stage the K loop waits for.
  const bool staged_epi = args.splits == 1 && args.vec8;
  const long coff = z1 * args.c_bs1 + z2 * args.c_bs2;
  EpiOperands<BNT, NTH> eop;
  if constexpr (DMA && KSL == 1) {
    if (staged_epi) eop.load(args, row0, col0, tid, coff);
  }

  const int wave = tid >> 6, lane = tid & 63;
  const int wm = (wave >> 1) & 1, wn = wave & 1, kslice = wave >> 2;

  f32x16_t acc[2][NJ];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  auto compute = [&](const bf16_t* sa, const bf16_t* sb) {
    // data gradient reading the filter through the transposing LDS reads: the
    // wave issuing MFMAs goes first while it does (measured faster for that
    // operand pair only; slower against the transposed filter copy)
    if constexpr (MA == OP_K_CONV_DGRAD && MB == OP_R_FILTER_T) __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int kk = kslice * KW; kk < (kslice + 1) * KW; kk += 16) {
      bf16x8_t fa[2], fb[NJ];
      const int kl = kk + (lane >> 5) * 8;
#pragma unroll
      for (int i = 0; i < 2; ++i)
        fa[i] = (MA <= OP_K_CONV_DGRAD)
                    ? (DMA ? frag_kd(sa, wm * 64 + i * 32 + (lane & 31), kl) : frag_k(sa, wm * 64 + i * 32 + (lane & 31), kl))
                    : frag_r(sa, wm * 64 + i * 32, kk, lane);
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        fb[j] = (MB <= OP_K_CONV_DGRAD)
                    ? (DMA ? frag_kd(sb, wn * (32 * NJ) + j * 32 + (lane & 31), kl)
                           : frag_k(sb, wn * (32 * NJ) + j * 32 + (lane & 31), kl))
                    : frag_r(sb, wn * (32 * NJ) + j * 32, kk, lane);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[j], fa[i], acc[i][j], 0, 0, 0);
    }
    __builtin_amdgcn_iglp_opt(0);
    if constexpr (MA == OP_K_CONV_DGRAD && MB == OP_R_FILTER_T) __builtin_amdgcn_s_setprio(0);
  };

  if constexpr (DMA) {
    if (nk > 0) {
      // stage b (b = 0, 1) at elements [2 b BK 128, ...): A tile then B tile,
      // 128 x 64 each; the prefetch of the two steps past the end reads zeros
      // or data that is never multiplied, and is drained before the LDS is
      // reused by the epilogue
      constexpr int TE = BM * BK, SE = 2 * TE;
      static_assert(sizeof(lds) >= 2 * SE * sizeof(bf16_t), "two stages fit the operand buffers");
      constexpr int VS = decltype(la)::V + decltype(lb)::V;   // direct loads per thread per stage
      bf16_t* const l0 = &lds[0][0][0];
      const uint32_t lbase = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) bf16_t*)l0));
      const int wv = __builtin_amdgcn_readfirstlane(wave);
      auto issue = [&](int buf, int k0) {
        const uint32_t t = lbase + static_cast<uint32_t>(buf * SE * 2);
        la.dma(A, ra, k0, t, wv);
        lb.dma(B, rb, k0, t + TE * 2, wv);
      };
      issue(0, kbeg);
      issue(1, kbeg + BK);
      dma_wait<VS>();
      __syncthreads();
      for (int kt = 0; kt < nk; ++kt) {
        const bf16_t* sa = l0 + (kt & 1) * SE;
        compute(sa, sa + TE);
        __syncthreads();
        issue(kt & 1, kbeg + (kt + 2) * BK);
        dma_wait<VS>();
        __syncthreads();
      }
      dma_wait<0>();
    }
  } else if (nk > 0) {
    uint4 ra0[4], rb0[4], ra1[4], rb1[4];
    // Prefetch loads are issued unconditionally (a step past the end reads
    // zeros or data that is never stored), so the compiler can count the
    // outstanding loads exactly and wait only for the older register set.
    la.load(A, ra, kbeg, ra0);
    lb.load(B, rb, kbeg, rb0);
    la.load(A, ra, kbeg + BK, ra1);
    lb.load(B, rb, kbeg + BK, rb1);
    la.store(lds[0][0], ra0, tid);
    lb.store(lds[0][1], rb0, tid);
    __syncthreads();
    // Register sets 0 / 1 hold K steps of even / odd index; LDS buffer b holds
    // the step being multiplied. The loop body covers a pair of steps and has
    // no exit in the middle, so the accumulators keep one register home.
    int kt = 0;
    for (; kt + 2 <= nk; kt += 2) {
      la.load(A, ra, kbeg + (kt + 2) * BK, ra0);
      lb.load(B, rb, kbeg + (kt + 2) * BK, rb0);
      compute(lds[0][0], lds[0][1]);
      la.store(lds[1][0], ra1, tid);
      lb.store(lds[1][1], rb1, tid);
      __syncthreads();
      la.load(A, ra, kbeg + (kt + 3) * BK, ra1);
      lb.load(B, rb, kbeg + (kt + 3) * BK, rb1);
      compute(lds[1][0], lds[1][1]);
      if (kt + 2 < nk) {
        la.store(lds[0][0], ra0, tid);
        lb.store(lds[0][1], rb0, tid);
      }
      __syncthreads();
    }
    if (kt < nk) compute(lds[0][0], lds[0][1]);   // odd step count: the last step is in buffer 0
  }

  if constexpr (KSL == 2) {
    // second-half waves hand their sums to the first-half waves through LDS
    // (register r of tile (i, j) of lane l at [sub-tile][i][j][r][l])
    float* red = reinterpret_cast<float*>(&lds[0][0][0]);
    static_assert(sizeof(lds) >= 4 * 2 * NJ * 16 * 64 * sizeof(float), "the reduction fits the operand buffers");
    float* mine = red + (wave & 3) * (2 * NJ * 16 * 64) + lane;
    __syncthreads();
    if (kslice == 1) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) mine[((i * NJ + j) * 16 + r) * 64] = acc[i][j][r];
    }
    __syncthreads();
    if (kslice == 0) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] += mine[((i * NJ + j) * 16 + r) * 64];
    }
    if (!staged_epi) {
      if (kslice == 1) return;
      write_tile<NJ>(args, acc, row0, col0, wm, wn, lane, split, z, z1, z2);
      return;
    }
    __syncthreads();   // the sums are read before the staged tile overwrites them
  }
  {
    if (staged_epi) {
      // float32 tile [128][BNT] in LDS (row pitch BNT + 4 floats), then each
      // thread takes 8 consecutive columns of NP rows: every load and store
      // of the epilogue covers whole row segments. All of a thread's operand
      // loads are issued before the tile is staged and before its first
      // store: loads and stores share one counter of outstanding memory
      // operations, so a load issued after a store would wait for the store
      // to complete and every row would cost a memory round trip.
      constexpr int EP = BNT + 4;
      using EO = EpiOperands<BNT, NTH>;
      constexpr int TPR = EO::TPR, RPP = EO::RPP, NP = EO::NP;
      const int ecl = (tid % TPR) * 8, erl = tid / TPR;
      const int ecol = col0 + ecl;
      const EpiDev& e = args.e;
      const bool colok = ecol < args.N;
      if constexpr (!(DMA && KSL == 1)) eop.load(args, row0, col0, tid, coff);
      const uint4 ebb = eop.bb;
      const uint4 (&erb)[NP] = eop.rb;
      const uint4 (&emk)[NP] = eop.mk;
      float* tile = reinterpret_cast<float*>(&lds[0][0][0]);
      static_assert(sizeof(lds) >= 128 * (BNT + 4) * sizeof(float), "the float32 tile fits the operand buffers");
      if constexpr (KSL == 1) __syncthreads();   // every wave has read its last operand tile
      if (kslice == 0) {                         // 8-wave blocks: the first-half waves hold the sums
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const int r = wm * 64 + i * 32 + (lane & 31);
              const int c = wn * (32 * NJ) + j * 32 + 8 * g + 4 * (lane >> 5);
              *reinterpret_cast<float4*>(tile + r * EP + c) =
                  make_float4(acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
            }
      }
      __syncthreads();
      // whole tiles with only bf16 operands: the specialised rows
      if (e.out_bf16 && !e.out_f32 && !e.bias && !e.res_f32 && e.alpha == 1.0f && row0 + 128 <= args.M &&
          col0 + BNT <= args.N) {
        bf16_t* const out = e.out_bf16 + coff + static_cast<long>(row0) * e.ldc + ecol;   // row rr at + rr ldc
        const int kind = (e.bias_bf16 ? 1 : 0) | (e.res_bf16 ? 2 : 0) | (e.relu ? 4 : 0) | (e.mask ? 8 : 0);
        bool done = true;
        switch (kind) {
          case 0: staged_rows<BNT, NTH, false, false, false, false>(e, tile, eop, out, ecl, erl); break;
          case 1: staged_rows<BNT, NTH, true, false, false, false>(e, tile, eop, out, ecl, erl); break;
          case 2: staged_rows<BNT, NTH, false, true, false, false>(e, tile, eop, out, ecl, erl); break;
          case 3: staged_rows<BNT, NTH, true, true, false, false>(e, tile, eop, out, ecl, erl); break;
          case 4: staged_rows<BNT, NTH, false, false, true, false>(e, tile, eop, out, ecl, erl); break;
          case 5: staged_rows<BNT, NTH, true, false, true, false>(e, tile, eop, out, ecl, erl); break;
          case 6: staged_rows<BNT, NTH, false, true, true, false>(e, tile, eop, out, ecl, erl); break;
          case 8: staged_rows<BNT, NTH, false, false, false, true>(e, tile, eop, out, ecl, erl); break;
          case 10: staged_rows<BNT, NTH, false, true, false, true>(e, tile, eop, out, ecl, erl); break;
          default: done = false;
        }
        if (done) return;
      }
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        const int rr = erl + p * RPP, row = row0 + rr;
        if (row >= args.M || !colok) continue;
        const long idx = coff + static_cast<long>(row) * e.ldc + ecol;
        const float4 a0 = *reinterpret_cast<const float4*>(tile + rr * EP + ecl);
        const float4 a1 = *reinterpret_cast<const float4*>(tile + rr * EP + ecl + 4);
        const uint2 h0 = epilogue4_values(e, idx, ecol, a0, make_uint2(ebb.x, ebb.y), make_uint2(erb[p].x, erb[p].y),
                                          make_uint2(emk[p].x, emk[p].y));
        const uint2 h1 = epilogue4_values(e, idx + 4, ecol + 4, a1, make_uint2(ebb.z, ebb.w),
                                          make_uint2(erb[p].z, erb[p].w), make_uint2(emk[p].z, emk[p].w));
        if (e.out_bf16) *reinterpret_cast<uint4*>(e.out_bf16 + idx) = make_uint4(h0.x, h0.y, h1.x, h1.y);
      }
      return;
    }
  }
  write_tile<NJ>(args, acc, row0, col0, wm, wn, lane, split, z, z1, z2);
}

// Sum the split partials in split order and apply the epilogue. Four
// consecutive columns per thread (N % 4 == 0) with 16-byte partial loads, all
// of a thread's loads issued before the ordered sum. The partial plane is
// below 2^31 elements (the workspace bounds it), so indices are 32-bit.
template <bool VEC_EPI>
__global__ __launch_bounds__(256) void splitk_reduce4_kernel(KArgs args) {
  const uint32_t mn = static_cast<uint32_t>(args.M) * args.N;
  const uint32_t plane = static_cast<uint32_t>(args.batch) * mn;
  const uint32_t total4 = plane >> 2;
  for (uint32_t t = blockIdx.x * 256 + threadIdx.x; t < total4; t += gridDim.x * 256) {
    const uint32_t e = t << 2;
    float4 v[MAX_SPLITS];
#pragma unroll
    for (int sp = 0; sp < MAX_SPLITS; ++sp)
      if (sp < args.splits) v[sp] = *reinterpret_cast<const float4*>(args.partial + sp * plane + e);
    float4 acc = v[0];
#pragma unroll
    for (int sp = 1; sp < MAX_SPLITS; ++sp)
      if (sp < args.splits) {
        acc.x += v[sp].x;
        acc.y += v[sp].y;
        acc.z += v[sp].z;
        acc.w += v[sp].w;
      }
    uint32_t z = 0, rem = e;
    if (args.batch > 1) {
      z = e / mn;
      rem = e - z * mn;
    }
    const uint32_t row = rem / static_cast<uint32_t>(args.N), col = rem - row * args.N;
    const uint32_t z1 = z / args.zdiv, z2 = z - z1 * args.zdiv;
    const long o = z1 * args.c_bs1 + z2 * args.c_bs2 + static_cast<long>(row) * args.e.ldc + col;
    if (VEC_EPI) {
      epilogue4(args.e, o, col, acc);
    } else {
      epilogue(args.e, o, col, acc.x);
      epilogue(args.e, o + 1, col + 1, acc.y);
      epilogue(args.e, o + 2, col + 2, acc.z);
      epilogue(args.e, o + 3, col + 3, acc.w);
    }
  }
}

// Scalar variant for N % 4 != 0.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(KArgs args) {
  const long mn = static_cast<long>(args.M) * args.N;
  const long plane = static_cast<long>(args.batch) * mn;
  for (long t = static_cast<long>(blockIdx.x) * 256 + threadIdx.x; t < plane;
       t += static_cast<long>(gridDim.x) * 256) {
    float s = 0.0f;
    for (int sp = 0; sp < args.splits; ++sp) s += args.partial[sp * plane + t];
    const int z = static_cast<int>(t / mn);
    const long rem = t - z * mn;
    const int row = static_cast<int>(rem / args.N), col = static_cast<int>(rem - static_cast<long>(row) * args.N);
    const int z1 = z / args.zdiv, z2 = z - z1 * args.zdiv;
    epilogue(args.e, z1 * args.c_bs1 + z2 * args.c_bs2 + static_cast<long>(row) * args.e.ldc + col, col, s);
  }
}

// Elements a correct launch may read from the batch-0 base: the operand of
// the last batch at its largest row and k (or the whole gathered tensor).
long operand_extent(const Operand& o, int rows, int K, int batch, int zdiv) {
  if (o.extent > 0) return o.extent;
  long per;
  switch (o.mode) {
    case OP_K_PLAIN: per = static_cast<long>(rows - 1) * o.ld + K; break;
    case OP_R_PLAIN: per = static_cast<long>(K - 1) * o.ld + rows; break;
    case OP_R_FILTER_T: per = static_cast<long>(o.g.C2) * 9 * o.g.C; break;
    default: per = static_cast<long>(o.g.B) * o.g.H * o.g.W * o.g.C; break;
  }
  const long z1max = (batch - 1) / zdiv;
  const long z2max = batch > zdiv ? zdiv - 1 : batch - 1;
  return per + z1max * o.bs1 + z2max * o.bs2;
}

OperandDev make_operand(const Operand& o, int rows, int K, long extent) {
  OperandDev d{};
  d.p = static_cast<const bf16_t*>(o.ptr);
  d.ld = o.ld;
  d.extent = extent;
  d.rows = rows;
  d.K = K;
  d.H = o.g.H;
  d.W = o.g.W;
  d.C = o.g.C;
  d.C2 = o.g.C2;
  const int hw = o.g.H * o.g.W;
  if (hw > 0) {
    const int rem = BK % hw;
    d.step_h = rem / o.g.W;
    d.step_w = rem % o.g.W;
  }
  d.fdC = FastDiv(o.g.C > 0 ? o.g.C : 1);
  d.fdC2 = FastDiv(o.g.C2 > 0 ? o.g.C2 : 1);
  d.fdHW = FastDiv(o.g.H * o.g.W > 0 ? o.g.H * o.g.W : 1);
  d.fdW = FastDiv(o.g.W > 0 ? o.g.W : 1);
  return d;
}

template <int MA, int MB, bool TAPK = false>
hipError_t launch(const KArgs& a, hipStream_t s) {
  dim3 grid(a.tiles_total, a.batch * a.splits);
  if (a.bn == 64) {
    hipLaunchKernelGGL((gemm_bf16_kernel<MA, MB, TAPK, 64, 1>), grid, dim3(NT), 0, s, a);
  } else if (a.ksl == 2) {
    hipLaunchKernelGGL((gemm_bf16_kernel<MA, MB, TAPK, 128, 2, true>), grid, dim3(2 * NT), 0, s, a);
  } else {
    hipLaunchKernelGGL((gemm_bf16_kernel<MA, MB, TAPK, 128, 1, true>), grid, dim3(NT), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace

namespace {

constexpr long kCUs = 256;
constexpr long kTargetBlocks = 2 * kCUs;   // two resident 4-wave blocks per CU

// Kernel of a launch (block tile width bn, waves per output sub-tile ksl)
// and its K split.
//  * 4-wave blocks, two per CU: 128-wide tiles, or 64-wide ones where
//    128-wide tiles cannot fill the two-per-CU slots but 64-wide ones fill
//    at least three quarters of them without a K split.
//  * A convolution gather against a row-major filter (the forward, or the
//    data gradient against a transposed filter copy) of that narrow kind
//    whose 128-wide tiles give between 7/8 of the CUs and every CU one block
//    runs them on 8-wave blocks instead (ksl = 2; its gathered A operand is
//    then loaded once per 128 x 128 outputs). Other operand pairs, and
//    launches filling fewer CUs, were measured slower on 8-wave blocks (with
//    direct loads too: every launch of at most one 128-wide block per CU on
//    8-wave blocks made the 1x1 and filter-gradient launches no faster or
//    slower alone, and the concurrent bottleneck step 20 % slower, its
//    8-wave blocks leaving no room on their CUs for the other pass).
//  * A split gives each slice at least 12 K steps (shorter slices cost more
//    in the reduction than they gain), at most MAX_SPLITS slices and no more
//    partials than the workspace holds.
//  * concurrent: the launch shares the GPU with another pass's launches (a
//    forward beside a backward), which fill the CUs its own grid leaves
//    idle. It keeps the 128-wide tile (a third less LDS traffic per MFMA
//    than the 64-wide one) instead of narrowing, and splits K only for grids
//    of fewer than 128 tiles or for K of 64 steps or more (measured: the
//    bottleneck and transformer stages 3.6 % and 3.9 % faster per step than
//    with the rules above; run alone, the narrow tiles stay faster).
struct Shape {
  int bn, ksl, splits;
};

Shape shape_of(int M, int N, int K, int batch, size_t workspace_bytes, bool conv_fwd, bool concurrent) {
  const long rows = static_cast<long>((M + BM - 1) / BM) * batch;
  const long t128 = rows * ((N + 127) / 128), t64 = rows * ((N + 63) / 64);
  Shape sh{128, 1, 1};
  if (t128 < kTargetBlocks && 4 * t64 >= 3 * kTargetBlocks) {
    if (conv_fwd && t128 <= kCUs && 8 * t128 >= 7 * kCUs) {
      sh.ksl = 2;
      return sh;
    }
    if (!concurrent) {
      sh.bn = 64;
      return sh;
    }
  }
  if (t128 >= kTargetBlocks || K < 2 * 12 * BK) return sh;
  if (concurrent && t128 >= kCUs / 2 && K < 64 * BK) return sh;
  int splits = static_cast<int>(kTargetBlocks / t128);   // all blocks resident in one round
  splits = std::min(splits, K / (12 * BK));
  splits = std::min(splits, MAX_SPLITS);
  const long per = static_cast<long>(batch) * M * N * 4;
  while (splits > 1 && per * splits > static_cast<long>(workspace_bytes)) --splits;
  sh.splits = std::max(splits, 1);
  return sh;
}

// Launch parameters of one GEMM: kernel, tile counts, the split of K and the
// device view of both operands. Returns false (with err set) for a shape the
// kernel cannot address; err stays hipSuccess for an empty problem.
bool plan(const GemmDesc& d, KArgs& a, hipError_t& err) {
  err = hipSuccess;
  if (d.M <= 0 || d.N <= 0 || d.batch <= 0) return false;
  const int zdiv = d.zdiv > 0 ? d.zdiv : 1;
  const long ext_a = operand_extent(d.A, d.M, d.K, d.batch, zdiv);
  const long ext_b = operand_extent(d.B, d.N, d.K, d.batch, zdiv);
  if (d.K <= 0 || ext_a <= 0 || ext_b <= 0 || ext_a >= (1L << 30) || ext_b >= (1L << 30)) {
    err = hipErrorInvalidValue;   // operands are addressed with 32-bit byte offsets
    return false;
  }
  a = KArgs{};
  a.M = d.M;
  a.N = d.N;
  a.K = d.K;
  a.batch = d.batch;
  a.zdiv = zdiv;
  const bool gather = (d.A.mode == OP_K_CONV_FWD || d.A.mode == OP_K_CONV_DGRAD) && d.B.mode == OP_K_PLAIN;
  const Shape sh = shape_of(d.M, d.N, d.K, d.batch, d.workspace ? d.workspace_bytes : 0, gather, d.concurrent);
  a.bn = sh.bn;
  a.ksl = sh.ksl;
  a.dma = sh.bn == 128;
  a.tiles_n = (d.N + a.bn - 1) / a.bn;
  a.tiles_total = a.tiles_n * ((d.M + BM - 1) / BM);
  const int splits = sh.splits;
  const int ksteps = (d.K + BK - 1) / BK;
  a.k_per_split = ((ksteps + splits - 1) / splits) * BK;
  a.splits = splits;
  a.partial = d.workspace;
  a.A = make_operand(d.A, d.M, d.K, ext_a);
  a.B = make_operand(d.B, d.N, d.K, ext_b);
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
  auto al = [](const void* p, uintptr_t n) { return (reinterpret_cast<uintptr_t>(p) & (n - 1)) == 0; };
  const EpiDev& e = a.e;
  a.vec_epi = e.ldc % 4 == 0 && a.c_bs1 % 4 == 0 && a.c_bs2 % 4 == 0 && al(e.out_f32, 16) && al(e.out_bf16, 8) &&
              al(e.bias, 16) && al(e.bias_bf16, 8) && al(e.res_f32, 16) && al(e.res_bf16, 8) && al(e.mask, 8);
  a.vec8 = a.vec_epi && d.N % 8 == 0 && e.ldc % 8 == 0 && a.c_bs1 % 8 == 0 && a.c_bs2 % 8 == 0 &&
           al(e.out_f32, 32) && al(e.out_bf16, 16) && al(e.bias, 32) && al(e.bias_bf16, 16) && al(e.res_f32, 32) &&
           al(e.res_bf16, 16) && al(e.mask, 16) && !e.res_f32 && !e.bias;
  return true;
}

hipError_t launch_main(const GemmDesc& d, const KArgs& a, hipStream_t s) {
  const int ma = d.A.mode, mb = d.B.mode;
  if (ma == OP_K_PLAIN && mb == OP_K_PLAIN) return launch<OP_K_PLAIN, OP_K_PLAIN>(a, s);
  if (ma == OP_K_PLAIN && mb == OP_R_PLAIN) return launch<OP_K_PLAIN, OP_R_PLAIN>(a, s);
  if (ma == OP_R_PLAIN && mb == OP_R_PLAIN) return launch<OP_R_PLAIN, OP_R_PLAIN>(a, s);
  if (ma == OP_K_CONV_FWD && mb == OP_K_PLAIN)
    return (d.A.g.C % BK == 0) ? launch<OP_K_CONV_FWD, OP_K_PLAIN, true>(a, s)
                               : launch<OP_K_CONV_FWD, OP_K_PLAIN>(a, s);
  if (ma == OP_K_CONV_DGRAD && mb == OP_R_FILTER_T)
    return (d.A.g.C % BK == 0 && d.B.g.C2 % BK == 0) ? launch<OP_K_CONV_DGRAD, OP_R_FILTER_T, true>(a, s)
                                                    : launch<OP_K_CONV_DGRAD, OP_R_FILTER_T>(a, s);
  if (ma == OP_K_CONV_DGRAD && mb == OP_K_PLAIN)
    return (d.A.g.C % BK == 0) ? launch<OP_K_CONV_DGRAD, OP_K_PLAIN, true>(a, s)
                               : launch<OP_K_CONV_DGRAD, OP_K_PLAIN>(a, s);
  if (ma == OP_R_PLAIN && mb == OP_R_CONV_WGRAD) return launch<OP_R_PLAIN, OP_R_CONV_WGRAD>(a, s);
  return hipErrorInvalidValue;
}

hipError_t launch_reduce(const KArgs& a, hipStream_t s) {
  const long total = static_cast<long>(a.batch) * a.M * a.N;
  if (a.N % 4 == 0) {
    const long blocks = std::min<long>((total / 4 + 255) / 256, 8192);
    if (a.vec_epi) hipLaunchKernelGGL(splitk_reduce4_kernel<true>, dim3(static_cast<int>(blocks)), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(splitk_reduce4_kernel<false>, dim3(static_cast<int>(blocks)), dim3(256), 0, s, a);
  } else {
    const long blocks = std::min<long>((total + 255) / 256, 8192);
    hipLaunchKernelGGL(splitk_reduce_kernel, dim3(static_cast<int>(blocks)), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace

const char* gemm_bf16_kernel_name(const GemmDesc& d) {
  KArgs a;
  hipError_t err;
  if (!plan(d, a, err)) return "gemm_bf16_kernel";
  const int ma = d.A.mode, mb = d.B.mode;
  bool tapk = false;
  if (ma == OP_K_CONV_FWD || (ma == OP_K_CONV_DGRAD && mb == OP_K_PLAIN)) tapk = d.A.g.C % BK == 0;
  if (ma == OP_K_CONV_DGRAD && mb == OP_R_FILTER_T) tapk = d.A.g.C % BK == 0 && d.B.g.C2 % BK == 0;
  // the kernel's template arguments as a profiler prints the instantiation
  static thread_local char buf[64];
  std::snprintf(buf, sizeof(buf), "gemm_bf16_kernel<%d, %d, %s, %d, %d, %s>", ma, mb, tapk ? "true" : "false",
                a.bn == 64 ? 64 : 128, a.bn == 64 ? 1 : a.ksl, a.dma ? "true" : "false");
  return buf;
}

const char* gemm_bf16_reduce_name(const GemmDesc& d) {
  KArgs a;
  hipError_t err;
  if (!plan(d, a, err)) return "splitk_reduce_kernel";
  if (a.N % 4) return "splitk_reduce_kernel";
  return a.vec_epi ? "splitk_reduce4_kernel<true>" : "splitk_reduce4_kernel<false>";
}

int gemm_bf16_split_rule(int M, int N, int K, int batch, size_t workspace_bytes, bool concurrent) {
  if (M <= 0 || N <= 0 || K <= 0 || batch <= 0) return 1;
  return shape_of(M, N, K, batch, workspace_bytes, false, concurrent).splits;
}

int gemm_bf16_splits(const GemmDesc& d) {
  KArgs a;
  hipError_t err;
  return plan(d, a, err) ? a.splits : 1;
}

hipError_t gemm_bf16(const GemmDesc& d, hipStream_t s, int phases) {
  KArgs a;
  hipError_t err;
  if (!plan(d, a, err)) return err;
  if (phases & GEMM_MAIN) {
    err = launch_main(d, a, s);
    if (err != hipSuccess) return err;
  }
  if ((phases & GEMM_REDUCE) && a.splits > 1) return launch_reduce(a, s);
  return hipSuccess;
}

}  // namespace spx
