// Step a2: Inv_t = (I + A_t)^{-1} for every frame of every head (Eq. 5).
//
// I + A_t is symmetric positive definite with every eigenvalue >= 1 (A_t is
// a Gram matrix weighted by beta >= 0; Appendix A.1), so Gauss-Jordan
// elimination needs no pivoting and every leading block is invertible.
//
// One wavefront inverts one d_k x d_k matrix in fp32 by blocked Gauss-Jordan
// with 16 x 16 blocks, the whole matrix held in MFMA accumulator layout
// (block (i, j): lane (c, g) holds rows 4g..4g+3, column c).  No LDS and no
// barriers are needed, because symmetry puts every operand in the lane's own
// registers.  After eliminating block columns 0..kb-1 the matrix is
// [[X, Y], [Z, S]] with X and S symmetric and Z = -Y^T, so block (i, kb) is
// the transpose of the stored block (kb, i), negated when i < kb.  The
// v_mfma_f32_16x16x4_f32 operand a lane supplies at k = 4g + s is then
// element s of its own accumulator of that transposed block.  Block step kb:
//   1. D^{-1} of the pivot block D = M[kb][kb] by scalar Gauss-Jordan (rows
//      and columns exchanged by cross-lane shuffles);
//   2. R_j = D^{-1} M[kb][j] for j != kb (D^{-1} is symmetric, so it is its
//      own A-operand);
//   3. M[i][j] -= M[i][kb] R_j and M[i][kb] = -M[i][kb] D^{-1} for i != kb;
//   4. M[kb][j] = R_j, M[kb][kb] = D^{-1}.
// Only the pivot row of each step is ever read, so a block (i, j) with
// j > kb that step j will overwrite (i < kb, or i > j) is not updated: about
// a third of the Gauss-Jordan products are skipped.
// Both A_t and its inverse are symmetric, so the column segments of the
// accumulator layout are loaded and stored as contiguous row segments of the
// transposed block (the result is the transpose of the computed inverse,
// which equals it up to rounding).
// The token-split partials of A_t are summed in split order while loading;
// the kernel also folds the split partials of B_t into the first partial for
// the state scan.  All products and sums are fp32.
#include "vda_common.h"
#include "vda_launch.h"

namespace vda {
namespace {

template <int DK>
__global__ __launch_bounds__(64)
void inverse_kernel(const float* A_part, int splits, size_t part_stride,
                    float* Inv,  // may alias A_part (in place)
                    float* B_part, size_t b_mat, size_t b_stride) {
  constexpr int NB = DK / 16;  // 16-wide blocks per side
  const size_t base = (size_t)blockIdx.x * (DK * DK);
  const int lane = threadIdx.x;
  const int li = lane & 15;
  const int lg = lane >> 4;

  // Fold the token-split partials of B_t into the first partial (in place).
  if (splits > 1) {
    float* b0 = B_part + (size_t)blockIdx.x * b_mat;
    for (size_t idx = (size_t)lane * 4; idx < b_mat; idx += 64 * 4) {
      float4 a4 = *reinterpret_cast<const float4*>(b0 + idx);
      for (int s = 1; s < splits; ++s) {
        const float4 x = *reinterpret_cast<const float4*>(b0 + s * b_stride + idx);
        a4.x += x.x;
        a4.y += x.y;
        a4.z += x.z;
        a4.w += x.w;
      }
      *reinterpret_cast<float4*>(b0 + idx) = a4;
    }
  }

  // The accumulator of block (i, j) holds the column segment
  // M[16i + 4lg .. +3][16j + li]; A_t is symmetric, so it is read as the
  // contiguous row segment M[16j + li][16i + 4lg .. +3] with 16-byte loads
  // (and the result is written back the same way).
  floatx4 acc[NB][NB];
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      floatx4 v = {0.f, 0.f, 0.f, 0.f};
      for (int s = 0; s < splits; ++s) {
        const float4 x = *reinterpret_cast<const float4*>(
            A_part + s * part_stride + base + (size_t)(16 * j + li) * DK + 16 * i + 4 * lg);
        v[0] += x.x;
        v[1] += x.y;
        v[2] += x.z;
        v[3] += x.w;
      }
      if (i == j) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (4 * lg + r == li) v[r] += 1.0f;
      }
      acc[i][j] = v;
    }

#pragma unroll
  for (int kb = 0; kb < NB; ++kb) {
    // 1. D^{-1}: lane holds D[4*lg + r][li] in d[r].
    float d[4] = {acc[kb][kb][0], acc[kb][kb][1], acc[kb][kb][2], acc[kb][kb][3]};
#pragma unroll
    for (int p = 0; p < 16; ++p) {
      const float rowv = __shfl(d[p & 3], li + 16 * (p >> 2));   // D[p][li]
      float colv[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) colv[r] = __shfl(d[r], p + 16 * lg);  // D[4lg+r][p]
      const float piv = __shfl(rowv, p);                           // D[p][p]
      // Hardware reciprocal refined by one Newton step (error <= 1 ulp); the
      // IEEE division sequence would sit 128 times on the serial path.
      float inv = __builtin_amdgcn_rcpf(piv);
      inv = inv * fmaf(-piv, inv, 2.0f);
      const float rs = rowv * inv;
#pragma unroll
      for (int r = 0; r < 4; ++r) d[r] = fmaf(-colv[r], rs, d[r]);
      if (lg == (p >> 2)) d[p & 3] = (li == p) ? inv : rs;          // pivot row
      if (li == p) {                                               // pivot column
#pragma unroll
        for (int r = 0; r < 4; ++r) d[r] = (4 * lg + r == p) ? inv : -colv[r] * inv;
      }
    }

    // 2. R_j = D^{-1} M[kb][j]; A-operand D^{-1}[li][4lg+s] = d[s] (symmetric).
    floatx4 R[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) R[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        if (j == kb) continue;
        R[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(d[s], acc[kb][j][s], R[j], 0, 0, 0);
      }

    // 3. rows i != kb.  A-operand of -M[i][kb] at k = 4lg + s:
    //    i > kb: -acc[kb][i][s];  i < kb: +acc[kb][i][s].
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      if (i == kb) continue;
      float a[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) a[s] = (i > kb) ? -acc[kb][i][s] : acc[kb][i][s];
      // Independent accumulators innermost, so consecutive products do not
      // wait on each other.
      floatx4 o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 4; ++s) {
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          // Block (i, j), j > kb, is overwritten at step j (from the pivot
          // row's transpose) unless kb < i <= j: skip those dead updates.
          if (j == kb || (j > kb && (i > j || i < kb))) continue;
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], R[j][s], acc[i][j], 0, 0, 0);
        }
        o = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], d[s], o, 0, 0, 0);
      }
      acc[i][kb] = o;
    }

    // 4. pivot row.
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if (j == kb)
        acc[kb][j] = floatx4{d[0], d[1], d[2], d[3]};
      else
        acc[kb][j] = R[j];
    }
  }

#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
      *reinterpret_cast<float4*>(Inv + base + (size_t)(16 * j + li) * DK + 16 * i + 4 * lg) =
          make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
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
      hipLaunchKernelGGL(inverse_kernel<32>, grid, dim3(64), 0, stream, A_part, splits,
                         part_stride, Inv, B_part, b_mat, b_stride);
      break;
    case 64:
      hipLaunchKernelGGL(inverse_kernel<64>, grid, dim3(64), 0, stream, A_part, splits,
                         part_stride, Inv, B_part, b_mat, b_stride);
      break;
    case 128:
      hipLaunchKernelGGL(inverse_kernel<128>, grid, dim3(64), 0, stream, A_part, splits,
                         part_stride, Inv, B_part, b_mat, b_stride);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace vda
