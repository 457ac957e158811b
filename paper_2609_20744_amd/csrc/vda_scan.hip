// Steps a3/a4: the forward and reverse state scans of Eq. A.1 (alpha = 1),
// Algorithm 1 step 5, from a zero initial state:
//     P_t = (P_{t-1} + B_t) Inv_t,    R_t = (R_{t+1} + B_t) Inv_t.
// The entering state of every frame (P_{t-1} forward, R_{t+1} reverse) is
// stored for the readout.
//
// The rows of the d_v x d_k state evolve independently (each is a row vector
// times Inv_t), so a chain (head, direction) is split into 16-row blocks,
// one workgroup each, and the frame loop runs inside the workgroup with the
// 16 x d_k block resident in LDS (double-buffered, fp32).  Per frame the four
// wavefronts multiply the block by Inv_t with v_mfma_f32_16x16x4_f32, each
// producing d_k/64 16-column slices.  The next frame's Inv_t and B_t are
// loaded into registers one step ahead, so only the matrix product and two
// barriers sit on the serial path.  Workgroups of one chain are placed on one
// XCD so they share Inv_t in its L2.
#include "vda_common.h"
#include "vda_launch.h"

namespace vda {
namespace {

template <int DK>
__global__ __launch_bounds__(kThreads)
void scan_kernel(const float* __restrict__ Inv, const float* __restrict__ B_part, int splits,
                 size_t part_stride, int F, int DV, unsigned nwg,
                 float* __restrict__ S_fwd, float* __restrict__ S_rev) {
  constexpr int XLD = DK + 4;        // LDS row stride (floats)
  constexpr int NB = DK / 16;        // 16-column output slices
  constexpr int NBW = (NB + 3) / 4;  // slices per wave
  constexpr int KS = DK / 4;         // k values per lane group
  constexpr int E = DK / 16;         // state elements per thread in the row-wise phase
  static_assert(E % 2 == 0, "float2 granularity");
  __shared__ __align__(16) float xs[2][16 * XLD];

  const int nrb = DV / 16;
  const unsigned L = xcd_grouped_id(blockIdx.x, nwg);
  const int rb = L % nrb;
  const unsigned chain = L / nrb;
  const int dir = chain & 1;
  const unsigned hb = chain >> 1;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int li = lane & 15;
  const int lg = lane >> 4;

  // Row-wise phase role: row pr of the block, columns pc .. pc+E-1.
  const int pr = tid >> 4;
  const int pc = (tid & 15) * E;

  for (int i = tid; i < 16 * XLD; i += kThreads) xs[0][i] = 0.f;

  float* Sout = dir == 0 ? S_fwd : S_rev;
  const size_t mat_b = (size_t)DV * DK;  // one B / state matrix
  const size_t row_off = (size_t)(rb * 16 + pr) * DK + pc;

  auto frame_of = [&](int step) { return dir == 0 ? step : F - 1 - step; };

  // B-operand of the MFMA: Inv_t[lg*KS + s][nb*16 + li].
  float opc[NBW][KS], opn[NBW][KS];
  float bc[E], bn[E];
  auto load_ops = [&](int step, float (&op)[NBW][KS], float (&bb)[E]) {
    const size_t fh = (size_t)hb * F + frame_of(step);
    const float* inv = Inv + fh * (DK * DK);
#pragma unroll
    for (int m = 0; m < NBW; ++m) {
      const int nb = wave + 4 * m;
      if (nb < NB) {
#pragma unroll
        for (int s = 0; s < KS; ++s) op[m][s] = inv[(lg * KS + s) * DK + nb * 16 + li];
      }
    }
#pragma unroll
    for (int e = 0; e < E; ++e) bb[e] = 0.f;
    for (int sp = 0; sp < splits; ++sp) {
      const float* src = B_part + sp * part_stride + fh * mat_b + row_off;
#pragma unroll
      for (int e = 0; e < E; e += 2) {
        const float2 x = *reinterpret_cast<const float2*>(src + e);
        bb[e] += x.x;
        bb[e + 1] += x.y;
      }
    }
  };

  load_ops(0, opc, bc);
  int cur = 0;
  for (int step = 0; step < F; ++step) {
    const size_t fh = (size_t)hb * F + frame_of(step);
    if (step + 1 < F) load_ops(step + 1, opn, bn);
    __syncthreads();  // xs[cur] holds the entering state
    {
      float* x = &xs[cur][pr * XLD + pc];
      float* dst = Sout + fh * mat_b + row_off;
#pragma unroll
      for (int e = 0; e < E; e += 2) {
        float2 v = *reinterpret_cast<float2*>(x + e);
        *reinterpret_cast<float2*>(dst + e) = v;
        v.x += bc[e];
        v.y += bc[e + 1];
        *reinterpret_cast<float2*>(x + e) = v;
      }
    }
    __syncthreads();
    if (wave < NB) {
      float a[KS];
      const float* xr = &xs[cur][li * XLD + lg * KS];
#pragma unroll
      for (int s = 0; s < KS; s += 4) {
        const float4 v = *reinterpret_cast<const float4*>(xr + s);
        a[s] = v.x;
        a[s + 1] = v.y;
        a[s + 2] = v.z;
        a[s + 3] = v.w;
      }
#pragma unroll
      for (int m = 0; m < NBW; ++m) {
        const int nb = wave + 4 * m;
        if (nb < NB) {
          floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int s = 0; s < KS; ++s)
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], opc[m][s], acc, 0, 0, 0);
#pragma unroll
          for (int i = 0; i < 4; ++i) xs[cur ^ 1][(lg * 4 + i) * XLD + nb * 16 + li] = acc[i];
        }
      }
    }
    cur ^= 1;
#pragma unroll
    for (int m = 0; m < NBW; ++m)
#pragma unroll
      for (int s = 0; s < KS; ++s) opc[m][s] = opn[m][s];
#pragma unroll
    for (int e = 0; e < E; ++e) bc[e] = bn[e];
  }
}

template <int DK>
hipError_t launch_scan_t(const float* Inv, const float* B_part, int splits, int F, int H, int d_v,
                         float* S_fwd, float* S_rev, hipStream_t stream) {
  const unsigned nwg = (unsigned)H * 2u * (unsigned)(d_v / 16);
  const size_t part_stride = (size_t)H * F * d_v * DK;
  hipLaunchKernelGGL(scan_kernel<DK>, dim3(nwg), dim3(kThreads), 0, stream, Inv, B_part, splits,
                     part_stride, F, d_v, nwg, S_fwd, S_rev);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_state_scan(const float* Inv, const float* B_part, int splits, int F, int H,
                             int d_k, int d_v, float* S_fwd, float* S_rev, hipStream_t stream) {
  switch (d_k) {
    case 32: return launch_scan_t<32>(Inv, B_part, splits, F, H, d_v, S_fwd, S_rev, stream);
    case 64: return launch_scan_t<64>(Inv, B_part, splits, F, H, d_v, S_fwd, S_rev, stream);
    case 128: return launch_scan_t<128>(Inv, B_part, splits, F, H, d_v, S_fwd, S_rev, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace vda
