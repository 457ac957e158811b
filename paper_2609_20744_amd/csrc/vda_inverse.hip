// Step a2 as a stand-alone kernel: Inv_t = (I + A_t)^{-1} for every frame
// of every head (Eq. 5), one workgroup per matrix.  The algorithm is
// described in vda_inverse_body.h.  The result is written as an fp32
// matrix, or (TILED, for the split-bf16 state scan) as split-bf16 operand
// tiles (operand_tile_offset).
#include "vda_common.h"
#include "vda_inverse_body.h"
#include "vda_launch.h"

namespace vda {
namespace {

// Three workgroups per SIMD (the registers of the tiled store would
// otherwise push it to two), so one matrix's serial pivot work hides behind
// the others' products.
template <int DK, bool TILED>
__global__ __launch_bounds__(64 * (DK / 16 < 4 ? DK / 16 : 4))
__attribute__((amdgpu_waves_per_eu(3)))
void inverse_kernel(const float* A_part, unsigned first_split, int plan_splits, unsigned extra,
                    size_t part_stride,
                    float* Inv,  // may alias A_part (in place)
                    float* B_part, size_t b_mat, size_t b_stride) {
  constexpr int NB = DK / 16;
  constexpr int W = NB < 4 ? NB : 4;
  __shared__ __align__(16) float piv[3][NB][64 * 4];  // [buffer][block j][lane][4]

  const int tid = threadIdx.x;
  if (blockIdx.x >= gridDim.x - extra) {
    // One of the workgroups past the matrices: fold the token-range partials
    // of B_t of split frame first_split + (its index) / 4, quarter (its
    // index) % 4 of the matrix, into the first partial (in place), alongside
    // the inversions.
    const unsigned e = blockIdx.x - (gridDim.x - extra);
    const size_t f = first_split + e / 4;
    const size_t quarter = b_mat / 4;
    inv::fold_b_partials(B_part + f * b_mat, plan_splits, (e % 4) * quarter,
                         (e % 4 + 1) * quarter, b_stride, tid, 64 * W);
    return;
  }
  const size_t base = (size_t)blockIdx.x * (DK * DK);
  // Frames from first_split on were split into plan_splits token ranges.
  const int splits = blockIdx.x >= first_split ? plan_splits : 1;
  inv::invert_matrix<DK, TILED>(A_part, splits, part_stride, base, Inv, &piv[0][0][0], tid);
}

}  // namespace

hipError_t launch_frame_inverse(const float* A_part, float* B_part, SplitPlan plan,
                                long long count, int d_k, int d_v, bool tiled, float* Inv,
                                hipStream_t stream) {
  const int splits = plan.splits > 1 && plan.tail > 0 ? plan.splits : 1;
  const unsigned first_split = splits > 1 ? (unsigned)(count - plan.tail) : (unsigned)count;
  // Partial p of frame f is matrix f + p * tail.
  const size_t part_stride = (size_t)plan.tail * d_k * d_k;
  const size_t b_mat = (size_t)d_v * d_k;
  const size_t b_stride = (size_t)plan.tail * b_mat;
  // One workgroup per matrix, then four per split frame to fold its B
  // partials (a quarter of the matrix each, one memory round trip).
  const unsigned extra = splits > 1 ? 4u * (unsigned)plan.tail : 0u;
  const dim3 grid((unsigned)count + extra);
  switch (d_k) {
    case 32:
      if (tiled)
        hipLaunchKernelGGL((inverse_kernel<32, true>), grid, dim3(64 * 2), 0, stream, A_part,
                           first_split, splits, extra, part_stride, Inv, B_part, b_mat, b_stride);
      else
        hipLaunchKernelGGL((inverse_kernel<32, false>), grid, dim3(64 * 2), 0, stream, A_part,
                           first_split, splits, extra, part_stride, Inv, B_part, b_mat, b_stride);
      break;
    case 64:
      if (tiled)
        hipLaunchKernelGGL((inverse_kernel<64, true>), grid, dim3(64 * 4), 0, stream, A_part,
                           first_split, splits, extra, part_stride, Inv, B_part, b_mat, b_stride);
      else
        hipLaunchKernelGGL((inverse_kernel<64, false>), grid, dim3(64 * 4), 0, stream, A_part,
                           first_split, splits, extra, part_stride, Inv, B_part, b_mat, b_stride);
      break;
    case 128:
      if (tiled)
        hipLaunchKernelGGL((inverse_kernel<128, true>), grid, dim3(64 * 4), 0, stream, A_part,
                           first_split, splits, extra, part_stride, Inv, B_part, b_mat, b_stride);
      else
        hipLaunchKernelGGL((inverse_kernel<128, false>), grid, dim3(64 * 4), 0, stream, A_part,
                           first_split, splits, extra, part_stride, Inv, B_part, b_mat, b_stride);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace vda
