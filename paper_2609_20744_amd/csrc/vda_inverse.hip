// Step a2 as a stand-alone kernel: Inv_t = (I + A_t)^{-1} for every frame
// of every head (Eq. 5), one workgroup per matrix.  The algorithm is
// described in vda_inverse_body.h.
#include "vda_common.h"
#include "vda_inverse_body.h"
#include "vda_launch.h"

namespace vda {
namespace {

template <int DK>
__global__ __launch_bounds__(64 * (DK / 16 < 4 ? DK / 16 : 4))
void inverse_kernel(const float* A_part, int splits, size_t part_stride,
                    float* Inv,  // may alias A_part (in place)
                    float* B_part, size_t b_mat, size_t b_stride) {
  constexpr int NB = DK / 16;
  constexpr int W = NB < 4 ? NB : 4;
  __shared__ __align__(16) float piv[2][NB][64 * 4];  // [buffer][block j][lane][4]

  const size_t base = (size_t)blockIdx.x * (DK * DK);
  const int tid = threadIdx.x;

  // Fold the token-split partials of B_t into the first partial (in place).
  if (splits > 1)
    inv::fold_b_partials(B_part + (size_t)blockIdx.x * b_mat, splits, b_mat, b_stride, tid, 64 * W);

  inv::invert_matrix<DK>(A_part, splits, part_stride, base, Inv, &piv[0][0][0], tid);
}

}  // namespace

hipError_t launch_frame_inverse(const float* A_part, float* B_part, int splits, long long count,
                                int d_k, int d_v, float* Inv, hipStream_t stream) {
  const size_t part_stride = (size_t)count * d_k * d_k;
  const size_t b_mat = (size_t)d_v * d_k;
  const size_t b_stride = (size_t)count * b_mat;
  const dim3 grid((unsigned)count);
  switch (d_k) {
    case 32:
      hipLaunchKernelGGL(inverse_kernel<32>, grid, dim3(64 * 2), 0, stream, A_part, splits,
                         part_stride, Inv, B_part, b_mat, b_stride);
      break;
    case 64:
      hipLaunchKernelGGL(inverse_kernel<64>, grid, dim3(64 * 4), 0, stream, A_part, splits,
                         part_stride, Inv, B_part, b_mat, b_stride);
      break;
    case 128:
      hipLaunchKernelGGL(inverse_kernel<128>, grid, dim3(64 * 4), 0, stream, A_part, splits,
                         part_stride, Inv, B_part, b_mat, b_stride);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace vda
