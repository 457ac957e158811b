// Internal definitions shared by the VDA kernels and the host library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vda {

// RMSNorm epsilon of the linear-branch epilogue (Eq. 1c); the paper does
// not state a value.
constexpr float kRmsEps = 1e-6f;

// L2-normalisation epsilon of the feature map (Sec. 2.3), x / sqrt(|x|^2 +
// eps); the paper states none.
constexpr float kL2Eps = 1e-6f;

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

// Buffer resource over [base, base + bytes): buffer loads outside the range
// return zero and buffer stores outside it are dropped, with no branch, so
// the compiler can keep counting outstanding memory operations precisely.
// The last word is the gfx9-family raw-buffer configuration.
// The base and size must be workgroup-uniform; they are passed through
// readfirstlane so the descriptor lives in scalar registers even when the
// address arithmetic ran on the vector ALU.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
  void* p = reinterpret_cast<void*>(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(p, (short)0, (int)__builtin_amdgcn_readfirstlane(bytes),
                                           0x00020000);
}

// Split-bf16 operand tiles of a d_k x d_k fp32 matrix X (the inverse
// (I + A_t)^{-1} on the bf16 storage path, written by the inverse and read
// by the state scan).  The scan's product x X of a 16-row block x on
// v_mfma_f32_16x16x32_bf16 takes, for output columns 16 nb .. 16 nb + 15
// and k step ks, one 8-element B-operand per lane (li, lg) =
// (lane % 16, lane / 16):
//     X[32 ks + 4 lg + r][16 nb + li] for r < 4, then
//     X[32 ks + 16 + 4 lg + r][16 nb + li] for r < 4
// (the k order the scan uses in both operands).  Each operand is stored as
// its bf16 part hi = RNE(x) in plane 0 and lo = RNE(x - hi) in plane 1, so
// one wave's operand of one (nb, ks) tile is 1 KB of contiguous memory.  The
// layout has d_k * d_k * 4 bytes, as many as the fp32 matrix.
__host__ __device__ constexpr uint32_t operand_tile_offset(int dk, int plane, int nb, int ks,
                                                           int lane) {
  return (uint32_t)plane * (uint32_t)(dk * dk * 2) +
         ((uint32_t)(nb * (dk / 32) + ks) * 64u + (uint32_t)lane) * 16u;
}

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Any offset at or past this is outside every buffer range used here.
constexpr uint32_t kOutOfRange = 0xfffffff0u;

__device__ __forceinline__ uint4 load_b128(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  const u32x4 v = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)byte_off, 0, 0));
  return make_uint4(v[0], v[1], v[2], v[3]);
}

__device__ __forceinline__ float load_f32(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)byte_off, 0, 0));
}

__device__ __forceinline__ void store_b64(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, uint2 v) {
  __builtin_amdgcn_raw_buffer_store_b64(u32x2{v.x, v.y}, r, (int)byte_off, 0, 0);
}

__device__ __forceinline__ void store_b128(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, (int)byte_off, 0, 0);
}

// 16-byte store of streamed output (cache policy sc0 | nt | sc1: written
// through at system scope, not kept).  An output much larger than the
// caches is then written back while it is produced, instead of being left
// dirty for the next kernel's reads to evict.
__device__ __forceinline__ void store_b128_stream(__amdgpu_buffer_rsrc_t r, uint32_t byte_off,
                                                  u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, (int)byte_off, 0, 1 | 2 | 16);
}

// Workgroup-uniform integer kept in a scalar register.  Integer division by
// a runtime value is expanded on the vector ALU; without this the compiler
// may treat values derived from it (such as buffer descriptors) as varying
// per lane.
__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Workgroup barrier after which LDS written before it by any wave is
// visible.  Each wave first waits for its own outstanding LDS operations
// (s_waitcnt lgkmcnt(0); the immediate leaves the other counters at their
// maximum): the compiler is relied on for that wait inside __syncthreads(),
// but it has been seen to drop it where a loop's back edge reaches the
// barrier right after LDS stores, which lets another wave read stale data.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __syncthreads();
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
