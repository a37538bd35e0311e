// Device-side helpers shared by the SparSTAR kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "launch.h"

namespace sparstar {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Two floats -> packed bf16 pair (round to nearest even, hardware convert).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  __bf16 a = (__bf16)lo;
  __bf16 b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

__device__ __forceinline__ bool keep_block(const KeepBlocks& kb, int j) {
  bool r = false;
#pragma unroll
  for (int t = 0; t < kMaxKeep; ++t) {
    if (t >= kb.n) break;  // uniform: a kernel argument
    r |= (j >= kb.begin[t]) & (j < kb.end[t]);
  }
  return r;
}

// Work-group id -> linear work index, so that consecutive linear indices land
// on the same XCD (work-groups are dispatched round-robin over the 8 XCDs).
// A bijection on [0, n).
__device__ __forceinline__ int64_t xcd_linear(int64_t id, int64_t n) {
  const int64_t q = n / 8, rem = n % 8;
  const int64_t x = id % 8, r = id / 8;
  return x * q + (x < rem ? x : rem) + r;
}

}  // namespace sparstar
