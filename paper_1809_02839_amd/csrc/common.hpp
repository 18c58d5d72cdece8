// Shared device/host helpers of the SpecTrain stage library (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>

namespace spx {

// bf16 is carried as its raw 16 bits; arithmetic is always float32.
typedef uint16_t bf16_t;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef uint16_t u16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float sigmoidf(float x) { return 1.0f / (1.0f + expf(-x)); }

__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two floats to two bf16 (lo in the low half), rounded to nearest, ties to
// even, by the conversion instruction (v_cvt_pk_bf16_f32). Over all 2^32
// float inputs it returns what the integer formulation returns: u + 0x7fff
// + bit 16 of u, shifted right by 16, for every non-NaN u, and u >> 16 with
// the quiet bit 0x40 set for a NaN.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// Round to nearest, ties to even (NaN stays NaN), as pack_bf16x2.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return static_cast<bf16_t>(pack_bf16x2(f, 0.0f) & 0xffffu);
}

// Unsigned division by a run-time constant d >= 1 for numerators below 2^31:
// q = (umulhi(n, magic) + n) >> shift with magic = floor(2^32 (2^shift - d) / d) + 1,
// shift = ceil(log2 d) (Granlund and Montgomery, PLDI 1994).
struct FastDiv {
  uint32_t d, magic, shift;
  FastDiv() : d(1), magic(0), shift(0) {}
  explicit FastDiv(uint32_t div) : d(div) {
    shift = 0;
    while ((1ull << shift) < div) ++shift;
    magic = static_cast<uint32_t>(((1ull << 32) * ((1ull << shift) - div)) / div + 1);
  }
  __host__ __device__ __forceinline__ uint32_t div(uint32_t n) const {
#if defined(__HIP_DEVICE_COMPILE__)
    uint32_t hi = __umulhi(n, magic);
#else
    uint32_t hi = static_cast<uint32_t>((static_cast<uint64_t>(n) * magic) >> 32);
#endif
    return static_cast<uint32_t>((static_cast<uint64_t>(hi) + n) >> shift);
  }
};

}  // namespace spx
