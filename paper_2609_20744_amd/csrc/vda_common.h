// Internal definitions shared by the VDA kernels and the host library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vda {

// RMSNorm epsilon of the linear-branch epilogue (Eq. 1c); the paper does
// not state a value.
constexpr float kRmsEps = 1e-6f;

// Workgroup size of every kernel: four 64-wide wavefronts, one per SIMD.
constexpr int kThreads = 256;

// Token tile of the frame-statistics kernels; split ranges are multiples.
constexpr int kStatsTile = 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// Two floats -> packed bf16 pair, round-to-nearest-even (low half = a).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Byte permute: result byte i = byte sel_i of the 8-byte value {hi:lo}.
__device__ __forceinline__ uint32_t perm_b32(uint32_t hi, uint32_t lo, uint32_t sel) {
  return __builtin_amdgcn_perm(hi, lo, sel);
}

// Map a linear workgroup id onto a logical id so that consecutive logical
// ids land on the same XCD.  Workgroups are dispatched round-robin over the
// 8 XCDs (id % 8), each with its own L2; grouping logically adjacent work
// (for example the row blocks of one scan chain, which read the same
// matrices) on one XCD lets it share that L2.  Identity when the count is not
// a multiple of 8.
__device__ __forceinline__ unsigned xcd_grouped_id(unsigned id, unsigned count) {
  if (count % 8u != 0u) return id;
  const unsigned per_xcd = count / 8u;
  return (id % 8u) * per_xcd + id / 8u;
}

}  // namespace vda
