// Step a2: Inv_t = (I + A_t)^{-1} for every frame of every head (Eq. 5).
//
// I + A_t is symmetric positive definite with every eigenvalue >= 1 (A_t is
// a Gram matrix weighted by beta >= 0; Appendix A.1), so Gauss-Jordan
// elimination needs no pivoting.  One workgroup inverts one matrix in fp32:
// the d_k x d_k matrix stays in registers, each of the 256 threads owning a
// (d_k/16) x (d_k/16) block.  At pivot p the owners of row p and column p
// publish them through LDS (double-buffered, so one barrier per pivot) and
// every thread applies the rank-1 elimination to its block, then the pivot
// row and column take their final values.  The partial statistics of the
// token splits are summed (in split order) while loading.
#include "vda_common.h"
#include "vda_launch.h"

namespace vda {
namespace {

template <int DK>
__global__ __launch_bounds__(kThreads)
void inverse_kernel(const float* A_part, int splits, size_t part_stride,
                    float* Inv) {  // Inv may alias A_part (in place)
  constexpr int BS = DK / 16;
  static_assert(BS % 2 == 0, "pivot buffers alternate with the pivot parity");
  __shared__ __align__(16) float rowbuf[2][DK];
  __shared__ __align__(16) float colbuf[2][DK];

  const size_t base = (size_t)blockIdx.x * (DK * DK);
  const int tid = threadIdx.x;
  const int ri = tid >> 4;  // row block
  const int cj = tid & 15;  // column block

  float m[BS][BS];
#pragma unroll
  for (int a = 0; a < BS; ++a) {
    const int gi = ri * BS + a;
#pragma unroll
    for (int b = 0; b < BS; ++b) m[a][b] = 0.f;
    for (int s = 0; s < splits; ++s) {
      const float* src = A_part + s * part_stride + base + (size_t)gi * DK + cj * BS;
#pragma unroll
      for (int b = 0; b < BS; b += 2) {
        const float2 x = *reinterpret_cast<const float2*>(src + b);
        m[a][b] += x.x;
        m[a][b + 1] += x.y;
      }
    }
#pragma unroll
    for (int b = 0; b < BS; ++b)
      if (gi == cj * BS + b) m[a][b] += 1.0f;
  }

  for (int pb = 0; pb < 16; ++pb) {
#pragma unroll
    for (int pc = 0; pc < BS; ++pc) {
      const int p = pb * BS + pc;
      const int buf = pc & 1;
      if (ri == pb) {
#pragma unroll
        for (int b = 0; b < BS; ++b) rowbuf[buf][cj * BS + b] = m[pc][b];
      }
      if (cj == pb) {
#pragma unroll
        for (int a = 0; a < BS; ++a) colbuf[buf][ri * BS + a] = m[a][pc];
      }
      __syncthreads();
      const float piv = rowbuf[buf][p];
      const float inv = 1.0f / piv;
      float g[BS], f[BS];
#pragma unroll
      for (int b = 0; b < BS; ++b) g[b] = rowbuf[buf][cj * BS + b];      // old row p
#pragma unroll
      for (int a = 0; a < BS; ++a) f[a] = colbuf[buf][ri * BS + a] * inv;  // old column p / piv
#pragma unroll
      for (int a = 0; a < BS; ++a)
#pragma unroll
        for (int b = 0; b < BS; ++b) m[a][b] = fmaf(-f[a], g[b], m[a][b]);
      if (ri == pb) {  // pivot row: old row / piv, diagonal 1 / piv
#pragma unroll
        for (int b = 0; b < BS; ++b) m[pc][b] = (cj * BS + b == p) ? inv : g[b] * inv;
      }
      if (cj == pb) {  // pivot column: -old column / piv, diagonal 1 / piv
#pragma unroll
        for (int a = 0; a < BS; ++a) m[a][pc] = (ri * BS + a == p) ? inv : -f[a];
      }
    }
  }

#pragma unroll
  for (int a = 0; a < BS; ++a) {
    float* dst = Inv + base + (size_t)(ri * BS + a) * DK + cj * BS;
#pragma unroll
    for (int b = 0; b < BS; b += 2) *reinterpret_cast<float2*>(dst + b) = make_float2(m[a][b], m[a][b + 1]);
  }
}

}  // namespace

hipError_t launch_frame_inverse(const float* A_part, int splits, long long count, int d_k,
                                float* Inv, hipStream_t stream) {
  const size_t part_stride = (size_t)count * d_k * d_k;
  const dim3 grid((unsigned)count);
  switch (d_k) {
    case 32:
      hipLaunchKernelGGL(inverse_kernel<32>, grid, dim3(kThreads), 0, stream, A_part, splits, part_stride, Inv);
      break;
    case 64:
      hipLaunchKernelGGL(inverse_kernel<64>, grid, dim3(kThreads), 0, stream, A_part, splits, part_stride, Inv);
      break;
    case 128:
      hipLaunchKernelGGL(inverse_kernel<128>, grid, dim3(kThreads), 0, stream, A_part, splits, part_stride, Inv);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace vda
