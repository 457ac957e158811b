// Step a1: per-frame statistics A_t = K_t^T Diag(beta_t) K_t and
// B_t = V_t^T Diag(beta_t) K_t (Eq. 3b), computed in one pass over K and V.
//
// Both products contract over the token axis, which is the slow (row) axis
// of the frame-major [token][channel] layout, so the matrix-core operands
// need the transposed view.  Each workgroup streams 64-token tiles: every
// thread loads an 8-token x 8-channel block with 16-byte coalesced loads,
// transposes it in registers (16-bit shuffles), and writes it channel-major
// into LDS; beta * k is formed in fp32 and rounded to bf16 on the way.  The
// stacked product [K | V]^T (beta K) is then one (d_k + d_v) x d_k output,
// accumulated in fp32 by v_mfma_f32_16x16x32_bf16 with operands read as
// 16-byte rows of the transposed tiles.  The next tile's global loads are
// issued before the current tile's matrix work, so HBM traffic overlaps the
// MFMA phase.
#include "vda_common.h"
#include "vda_launch.h"

namespace vda {
namespace {

constexpr int kLd = kStatsTile + 8;  // bf16 row stride of the transposed tiles (144 B)

// 8x8 transpose of 16-bit elements: in[e] holds channels 0..7 of token e,
// out[c] holds tokens 0..7 of channel c (low half first).
__device__ __forceinline__ void transpose8x8(const uint4 (&in)[8], uint4 (&out)[8]) {
  const uint32_t* w = reinterpret_cast<const uint32_t*>(in);
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int j = c >> 1;
    uint32_t r[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t lo = w[(2 * i) * 4 + j];
      const uint32_t hi = w[(2 * i + 1) * 4 + j];
      r[i] = (c & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
    }
    out[c] = make_uint4(r[0], r[1], r[2], r[3]);
  }
}

__device__ __forceinline__ uint32_t scale_pair(uint32_t w, float b) {
  return pack_bf16x2(bf16_lo(w) * b, bf16_hi(w) * b);
}

template <int DK, int DV>
__global__ __launch_bounds__(kThreads, 2)
void stats_bf16_kernel(const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
                       const float* __restrict__ beta, int N, int tokens_per_split,
                       int splits, unsigned fh_count,
                       float* __restrict__ A_part, float* __restrict__ B_part) {
  constexpr int DX = DK + DV;
  constexpr int CGK = DK / 8;      // 8-channel groups of K
  constexpr int CGH = DX / 32;     // 32-channel slices of [K | V]
  constexpr int RB = DX / 16;      // 16-row output blocks
  constexpr int CB = DK / 16;      // 16-column output blocks
  constexpr int RPW = (RB + 3) / 4;
  static_assert(CGH <= 8, "one 8x8 block per thread per tile");

  __shared__ __align__(16) uint16_t xt[DX * kLd];  // [K | V]^T tile, [channel][token]
  __shared__ __align__(16) uint16_t yt[DK * kLd];  // (beta K)^T tile

  const unsigned fh = blockIdx.x / splits;
  const int split = blockIdx.x % splits;
  const int n_begin = split * tokens_per_split;
  const int n_end = min(N, n_begin + tokens_per_split);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;

  // Loader role: channel group cg (8 channels), token group tg (8 tokens).
  const int cgh = (lane >> 5) + 2 * wave;
  const bool active = cgh < CGH;
  const int cg = (lane & 3) + 4 * cgh;
  const int tg = (lane >> 2) & 7;
  const bool is_k = cg < CGK;
  const int ld = is_k ? DK : DV;
  const uint16_t* src = is_k ? K + (size_t)fh * N * DK + cg * 8
                             : V + (size_t)fh * N * DV + (cg - CGK) * 8;
  const float* bsrc = beta + (size_t)fh * N;

  uint4 raw[8];
  float bw[8];
  auto load_tile = [&](int n0) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int n = n0 + tg * 8 + e;
      const bool ok = active && n < n_end;
      raw[e] = ok ? *reinterpret_cast<const uint4*>(src + (size_t)n * ld) : make_uint4(0, 0, 0, 0);
      bw[e] = (ok && is_k) ? bsrc[n] : 0.0f;
    }
  };

  const int li = lane & 15;
  const int lg = lane >> 4;
  floatx4 acc[RPW][CB];
#pragma unroll
  for (int r = 0; r < RPW; ++r)
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) acc[r][cb] = floatx4{0.f, 0.f, 0.f, 0.f};

  if (n_begin < n_end) load_tile(n_begin);
  for (int n0 = n_begin; n0 < n_end; n0 += kStatsTile) {
    __syncthreads();  // previous tile's operand reads are done
    if (active) {
      uint4 tr[8];
      transpose8x8(raw, tr);
#pragma unroll
      for (int c = 0; c < 8; ++c)
        *reinterpret_cast<uint4*>(&xt[(cg * 8 + c) * kLd + tg * 8]) = tr[c];
      if (is_k) {
        uint4 sc[8];
#pragma unroll
        for (int e = 0; e < 8; ++e)
          sc[e] = make_uint4(scale_pair(raw[e].x, bw[e]), scale_pair(raw[e].y, bw[e]),
                             scale_pair(raw[e].z, bw[e]), scale_pair(raw[e].w, bw[e]));
        transpose8x8(sc, tr);
#pragma unroll
        for (int c = 0; c < 8; ++c)
          *reinterpret_cast<uint4*>(&yt[(cg * 8 + c) * kLd + tg * 8]) = tr[c];
      }
    }
    __syncthreads();
    if (n0 + kStatsTile < n_end) load_tile(n0 + kStatsTile);

#pragma unroll
    for (int ks = 0; ks < kStatsTile / 32; ++ks) {
      bf16x8 bop[CB];
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        bop[cb] = *reinterpret_cast<const bf16x8*>(&yt[(cb * 16 + li) * kLd + ks * 32 + lg * 8]);
#pragma unroll
      for (int r = 0; r < RPW; ++r) {
        const int rb = wave + 4 * r;
        if (rb < RB) {
          const bf16x8 aop =
              *reinterpret_cast<const bf16x8*>(&xt[(rb * 16 + li) * kLd + ks * 32 + lg * 8]);
#pragma unroll
          for (int cb = 0; cb < CB; ++cb)
            acc[r][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aop, bop[cb], acc[r][cb], 0, 0, 0);
        }
      }
    }
  }

  // Output block (rb, cb): lane holds rows rb*16 + 4*lg + i, column cb*16 + li.
  float* Ab = A_part + ((size_t)split * fh_count + fh) * (DK * DK);
  float* Bb = B_part + ((size_t)split * fh_count + fh) * (DV * DK);
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const int rb = wave + 4 * r;
    if (rb < RB) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int x = rb * 16 + lg * 4 + i;
          const int col = cb * 16 + li;
          if (rb * 16 < DK)
            Ab[x * DK + col] = acc[r][cb][i];
          else
            Bb[(x - DK) * DK + col] = acc[r][cb][i];
        }
    }
  }
}

// fp32 storage: plain fp32 products and sums (no rounding of beta * k).
template <int DK, int DV>
__global__ __launch_bounds__(kThreads)
void stats_f32_kernel(const float* __restrict__ K, const float* __restrict__ V,
                      const float* __restrict__ beta, int N, int tokens_per_split,
                      int splits, unsigned fh_count,
                      float* __restrict__ A_part, float* __restrict__ B_part) {
  constexpr int DX = DK + DV;
  constexpr int T = 32;
  constexpr int OPT = DX * DK / kThreads;  // outputs per thread
  __shared__ float xs[T][DX];
  __shared__ float ys[T][DK];

  const unsigned fh = blockIdx.x / splits;
  const int split = blockIdx.x % splits;
  const int n_begin = split * tokens_per_split;
  const int n_end = min(N, n_begin + tokens_per_split);
  const int tid = threadIdx.x;

  float acc[OPT];
#pragma unroll
  for (int m = 0; m < OPT; ++m) acc[m] = 0.f;

  for (int n0 = n_begin; n0 < n_end; n0 += T) {
    __syncthreads();
    for (int idx = tid; idx < T * DX; idx += kThreads) {
      const int e = idx / DX, c = idx % DX;
      const int n = n0 + e;
      float x = 0.f;
      if (n < n_end)
        x = c < DK ? K[((size_t)fh * N + n) * DK + c] : V[((size_t)fh * N + n) * DV + (c - DK)];
      xs[e][c] = x;
      if (c < DK) ys[e][c] = n < n_end ? x * beta[(size_t)fh * N + n] : 0.f;
    }
    __syncthreads();
    for (int e = 0; e < T; ++e) {
#pragma unroll
      for (int m = 0; m < OPT; ++m) {
        const int o = tid + m * kThreads;
        acc[m] = fmaf(xs[e][o / DK], ys[e][o % DK], acc[m]);
      }
    }
  }
  float* Ab = A_part + ((size_t)split * fh_count + fh) * (DK * DK);
  float* Bb = B_part + ((size_t)split * fh_count + fh) * (DV * DK);
#pragma unroll
  for (int m = 0; m < OPT; ++m) {
    const int o = tid + m * kThreads;
    const int x = o / DK, j = o % DK;
    if (x < DK)
      Ab[x * DK + j] = acc[m];
    else
      Bb[(x - DK) * DK + j] = acc[m];
  }
}

template <int DK, int DV>
hipError_t launch_stats_t(bool is_f32, const void* k, const void* v, const float* beta,
                          int F, int N, int H, int splits, float* A_part, float* B_part,
                          hipStream_t stream) {
  const unsigned fh_count = (unsigned)H * (unsigned)F;
  const int tps = stats_tokens_per_split(N, splits);
  const dim3 grid(fh_count * (unsigned)splits);
  if (is_f32)
    hipLaunchKernelGGL((stats_f32_kernel<DK, DV>), grid, dim3(kThreads), 0, stream,
                       static_cast<const float*>(k), static_cast<const float*>(v), beta, N, tps,
                       splits, fh_count, A_part, B_part);
  else
    hipLaunchKernelGGL((stats_bf16_kernel<DK, DV>), grid, dim3(kThreads), 0, stream,
                       static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), beta, N,
                       tps, splits, fh_count, A_part, B_part);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_frame_stats(bool is_f32, const void* k, const void* v, const float* beta,
                              int F, int N, int H, int d_k, int d_v, int splits,
                              float* A_part, float* B_part, hipStream_t stream) {
#define VDA_STATS_CASE(DKV, DVV)                                                         \
  if (d_k == DKV && d_v == DVV)                                                          \
    return launch_stats_t<DKV, DVV>(is_f32, k, v, beta, F, N, H, splits, A_part, B_part, \
                                    stream);
  VDA_STATS_CASE(32, 32) VDA_STATS_CASE(32, 64) VDA_STATS_CASE(32, 128)
  VDA_STATS_CASE(64, 32) VDA_STATS_CASE(64, 64) VDA_STATS_CASE(64, 128)
  VDA_STATS_CASE(128, 32) VDA_STATS_CASE(128, 64) VDA_STATS_CASE(128, 128)
#undef VDA_STATS_CASE
  return hipErrorInvalidValue;
}

}  // namespace vda
