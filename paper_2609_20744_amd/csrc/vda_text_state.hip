// The prompt state S_T (Sec. 2.2, Eq. 1b): the prompt enters as a leading
// frame updated from the zero state (Sec. 4), so after the statistics and
// the inverse of that one frame per head, S_T = B_T (I + A_T)^{-1} for the
// joint rule (Eq. 5) or B_T / sqrt(L) for the frozen rule (Eq. 3c, U = L).
// This last step is one small d_v x d_k x d_k product per head, run once
// per prompt, so it is a plain fp32 loop: a thread per output element,
// lanes along the output column so that the Inv reads of a wave are
// contiguous and the B reads are broadcasts.
#include "vda_common.h"
#include "vda_launch.h"

namespace vda {
namespace {

// S[h][r][c] = sum_{j < d_k} B[h][r][j] Inv[h][j][c] (Inv != null), else
// B[h][r][c] * scale, for r < d_v and c < d_k.  B is [H][pv][pk] and Inv
// [H][pk][pk] (pk >= d_k, pv >= d_v: zero-padded heads); S is [H][d_v][d_k].
__global__ __launch_bounds__(kThreads)
void text_state_kernel(const float* __restrict__ B, const float* __restrict__ Inv, int H, int pk,
                       int pv, int d_k, int d_v, float scale, float* __restrict__ S) {
  const long long total = (long long)H * d_v * d_k;
  for (long long i = (long long)blockIdx.x * kThreads + threadIdx.x; i < total;
       i += (long long)gridDim.x * kThreads) {
    const int c = (int)(i % d_k);
    const long long hr = i / d_k;
    const int r = (int)(hr % d_v);
    const long long h = hr / d_v;
    const float* b = B + ((size_t)h * pv + r) * pk;
    float acc;
    if (Inv) {
      const float* m = Inv + (size_t)h * pk * pk + c;
      acc = 0.0f;
      for (int j = 0; j < d_k; ++j) acc = fmaf(b[j], m[(size_t)j * pk], acc);
    } else {
      acc = b[c] * scale;
    }
    S[i] = acc;
  }
}

}  // namespace

hipError_t launch_text_state(const float* B, const float* Inv, int H, int pk, int pv, int d_k,
                             int d_v, float scale, float* S, hipStream_t stream) {
  long long g = ((long long)H * d_v * d_k + kThreads - 1) / kThreads;
  if (g > 8192) g = 8192;
  hipLaunchKernelGGL(text_state_kernel, dim3((unsigned)g), dim3(kThreads), 0, stream, B, Inv, H,
                     pk, pv, d_k, d_v, scale, S);
  return hipGetLastError();
}

}  // namespace vda
