// Step a1: per-frame statistics A_t = K_t^T Diag(beta_t) K_t and
// B_t = V_t^T Diag(beta_t) K_t (Eq. 3b), computed in one pass over K and V.
//
// Two workgroups share a frame (and a token range): workgroup half h owns
// the output rows of K channels [h*d_k/2, (h+1)*d_k/2) (rows of A_t) and of
// V channels [h*d_v/2, ...) (rows of B_t), against all d_k columns of
// beta*K.  So no partial sums are written, each lane holds half the
// accumulators, and the two halves (placed on one XCD) read the same K
// tiles, which the second one finds in L2.
//
// Both products contract over tokens, the slow axis of the frame-major
// [token][channel] layout.  Tiles of 64 tokens are copied into LDS in that
// natural layout (16-byte coalesced loads, two tiles in flight in
// registers; beta*k is formed per token row in fp32 and rounded to bf16 on
// the way), and the matrix-core operands are read with gfx950's transposing
// LDS read ds_read_b64_tr_b16: within a 16-lane group, lane i returns
// element (i mod 4) of the 64-bit chunks addressed by lanes floor(i/4) + 4e,
// e = 0..3.  If lane j addresses token t0 + floor(j/4) at channel
// c0 + 4 (j mod 4), lane i receives tokens t0..t0+3 of channel c0 + i: one
// half of a v_mfma_f32_16x16x32_bf16 operand column.  Lane group g takes the
// tokens {4g + e} and {16 + 4g + e} of each 32-token step (the same order in
// both operands), which with a row stride of 288 bytes (32 mod 256) keeps
// the 32 lanes of one LDS pass on distinct banks.  Tokens past the range are
// read through range-checked buffer loads as zero, so they contribute
// nothing and no load sits behind a branch or feeds a select.
#include "vda_common.h"
#include "vda_launch.h"

namespace vda {
namespace {

typedef short v4i16 __attribute__((ext_vector_type(4)));

// Row stride (bf16 elements) of a natural-layout tile with `ch` channels:
// the row rounded up to a multiple of 256 bytes, plus 32 bytes.
__host__ __device__ constexpr int tile_ld(int ch) { return ((ch * 2 + 255) / 256) * 128 + 16; }

// One v_mfma_f32_16x16x32_bf16 operand: channels c0..c0+15 (lane i: c0 + i)
// at the 32 tokens k0.. of a natural-layout tile, in the token order above.
template <int LD>
__device__ __forceinline__ bf16x8 tr_operand(const uint16_t* tile, int k0, int c0, int li, int lg) {
  const int tok = k0 + 4 * lg + (li >> 2);
  const int ch = c0 + 4 * (li & 3);
  typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
  const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(tile + tok * LD + ch));
  const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(tile + (tok + 16) * LD + ch));
  typedef short v8i16 __attribute__((ext_vector_type(8)));
  const v8i16 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ uint32_t scale_pair(uint32_t w, float b) {
  return pack_bf16x2(bf16_lo(w) * b, bf16_hi(w) * b);
}

template <int DK, int DV>
__global__ __launch_bounds__(kThreads, 2)
void stats_bf16_kernel(const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
                       const float* __restrict__ beta, int N, int tokens_per_split,
                       int splits, unsigned fh_count, unsigned nwg,
                       float* __restrict__ A_part, float* __restrict__ B_part) {
  constexpr int KH = DK / 2;          // K channels (A rows) owned by a half
  constexpr int VH = DV / 2;          // V channels (B rows) owned by a half
  constexpr int XC = KH + VH;         // channels of the X tile [K_h | V_h]
  constexpr int LDX = tile_ld(XC);
  constexpr int LDY = tile_ld(DK);
  constexpr int RB = XC / 16;         // 16-row output blocks
  constexpr int CB = DK / 16;         // 16-column output blocks
  // The four waves split the workgroup's XC x DK output 2 x 2: wave (wr, wc)
  // owns row blocks wr*RPW .. and column blocks wc*CPW .. .  Per token a wave
  // reads RPW + CPW operand blocks from LDS, fewer than a 4 x 1 split.
  constexpr int RPW = (RB + 1) / 2;   // output row blocks per wave
  constexpr int CPW = CB / 2;         // output column blocks per wave
  constexpr int KCH = DK / 8;         // 16-byte chunks per K row
  constexpr int VCH = VH / 8;         // 16-byte chunks per V-half row
  constexpr int NKC = kStatsTile * KCH / kThreads;                // K chunks per thread
  constexpr int NVC = (kStatsTile * VCH + kThreads - 1) / kThreads;  // V chunks per thread
  static_assert(kStatsTile * KCH % kThreads == 0, "K chunks divide evenly");

  // One extra row absorbs the stores of lanes with nothing to store, so the
  // stores need no branch.
  __shared__ __align__(16) uint16_t xt[(kStatsTile + 1) * LDX];  // [token][K_h | V_h]
  __shared__ __align__(16) uint16_t yt[kStatsTile * LDY];  // [token][beta * K]

  // Logical id: (frame-head, split, half), halves adjacent on one XCD.
  const unsigned L = xcd_grouped_id(blockIdx.x, nwg);
  const int half = uniform(L & 1);
  const unsigned fs = L >> 1;
  const unsigned fh = (unsigned)uniform((int)(fs / splits));
  const int split = uniform((int)(fs % splits));
  const int n_begin = split * tokens_per_split;
  const int n_end = uniform(min(N, n_begin + tokens_per_split));

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int wr = wave & 1;
  const int wc = wave >> 1;
  const int li = lane & 15;
  const int lg = lane >> 4;

  // Range-checked views of this frame's rows [0, n_end): rows past the end
  // read as zero (so they add nothing to either product), with no clamp or
  // select between a load and its use.
  const __amdgpu_buffer_rsrc_t krsrc = make_rsrc(K + (size_t)fh * N * DK, (uint32_t)(n_end * DK * 2));
  const __amdgpu_buffer_rsrc_t vrsrc =
      make_rsrc(V + (size_t)fh * N * DV + half * VH, (uint32_t)(n_end * DV * 2 - half * VH * 2));
  const __amdgpu_buffer_rsrc_t brsrc = make_rsrc(beta + (size_t)fh * N, (uint32_t)(n_end * 4));

  // Loader roles: K chunk i of this thread is (row kr0 + i*kRowStep, col kc),
  // consecutive lanes reading consecutive 16-byte chunks of a row.
  constexpr int KROWS = kThreads / KCH;  // K rows covered per pass
  const int kc = tid % KCH;
  const int kr0 = tid / KCH;
  const bool kc_in_half = (kc / (KH / 8)) == half;
  const int vch = tid % VCH;
  const int vr0 = tid / VCH;
  constexpr int VROWS = kThreads / VCH;

  // Two-tile register ring, as separately named arrays so that every access
  // has a compile-time index (a two-dimensional ring was moved to scratch).
  u32x4 kraw0[NKC], kraw1[NKC];
  float kb0[NKC], kb1[NKC];
  u32x4 vraw0[NVC], vraw1[NVC];
  auto load_tile = [&](int n0, u32x4 (&kr)[NKC], float (&kbv)[NKC], u32x4 (&vr)[NVC]) {
#pragma unroll
    for (int i = 0; i < NKC; ++i) {
      const uint32_t n = (uint32_t)(n0 + kr0 + i * KROWS);
      kr[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                            krsrc, (int)(n * (DK * 2) + kc * 16), 0, 0));
      kbv[i] = load_f32(brsrc, n * 4u);
    }
#pragma unroll
    for (int i = 0; i < NVC; ++i) {
      const int r = vr0 + i * VROWS;  // >= kStatsTile only when the tile needs fewer chunks
      const uint32_t off = r < kStatsTile ? (uint32_t)(n0 + r) * (DV * 2) + vch * 16 : kOutOfRange;
      vr[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(vrsrc, (int)off, 0, 0));
    }
  };
  auto store_tile = [&](const u32x4 (&kr)[NKC], const float (&kbv)[NKC], const u32x4 (&vr)[NVC]) {
#pragma unroll
    for (int i = 0; i < NKC; ++i) {
      const int r = kr0 + i * KROWS;
      const u32x4 w = kr[i];
      const float b = kbv[i];
      *reinterpret_cast<u32x4*>(&yt[r * LDY + kc * 8]) =
          u32x4{scale_pair(w[0], b), scale_pair(w[1], b), scale_pair(w[2], b), scale_pair(w[3], b)};
      const int xo = kc_in_half ? r * LDX + (kc * 8 - half * KH) : kStatsTile * LDX;
      *reinterpret_cast<u32x4*>(&xt[xo]) = w;
    }
#pragma unroll
    for (int i = 0; i < NVC; ++i) {
      const int r = vr0 + i * VROWS;
      const int xo = r < kStatsTile ? r * LDX + KH + vch * 8 : kStatsTile * LDX;
      *reinterpret_cast<u32x4*>(&xt[xo]) = vr[i];
    }
  };

  floatx4 acc[RPW][CPW];
#pragma unroll
  for (int r = 0; r < RPW; ++r)
#pragma unroll
    for (int c = 0; c < CPW; ++c) acc[r][c] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Consume one tile from the ring, then refill its slot with tile n_next.
  auto tile_step = [&](int n_next, u32x4 (&kr)[NKC], float (&kbv)[NKC], u32x4 (&vr)[NVC]) {
    lds_barrier();  // previous tile's operand reads are done
    store_tile(kr, kbv, vr);
    lds_barrier();
    load_tile(n_next, kr, kbv, vr);
#pragma unroll
    for (int ks = 0; ks < kStatsTile / 32; ++ks) {
      bf16x8 bop[CPW];
#pragma unroll
      for (int c = 0; c < CPW; ++c)
        bop[c] = tr_operand<LDY>(yt, ks * 32, (wc * CPW + c) * 16, li, lg);
#pragma unroll
      for (int r = 0; r < RPW; ++r) {
        const int rb = wr * RPW + r;
        if (RB % 2 == 0 || rb < RB) {
          const bf16x8 aop = tr_operand<LDX>(xt, ks * 32, rb * 16, li, lg);
#pragma unroll
          for (int c = 0; c < CPW; ++c)
            acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aop, bop[c], acc[r][c], 0, 0, 0);
        }
      }
    }
  };

  if (n_begin < n_end) {
    load_tile(n_begin, kraw0, kb0, vraw0);
    __builtin_amdgcn_sched_barrier(0);
    load_tile(n_begin + kStatsTile, kraw1, kb1, vraw1);
    __builtin_amdgcn_sched_barrier(0);
  }
  // Pairs of tiles per iteration (a surplus tile has beta = 0 everywhere).
  for (int n0 = n_begin; n0 < n_end; n0 += 2 * kStatsTile) {
    tile_step(n0 + 2 * kStatsTile, kraw0, kb0, vraw0);
    tile_step(n0 + 3 * kStatsTile, kraw1, kb1, vraw1);
  }

  // Output block (rb, cb): lane holds rows rb*16 + 4*lg + i, column cb*16 + li.
  float* Ab = A_part + ((size_t)split * fh_count + fh) * (DK * DK);
  float* Bb = B_part + ((size_t)split * fh_count + fh) * (DV * DK);
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const int rb = wr * RPW + r;
    if (RB % 2 == 0 || rb < RB) {
#pragma unroll
      for (int c = 0; c < CPW; ++c)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int x = rb * 16 + lg * 4 + i;
          const int col = (wc * CPW + c) * 16 + li;
          if (rb * 16 < KH)
            Ab[(half * KH + x) * DK + col] = acc[r][c][i];
          else
            Bb[(half * VH + x - KH) * DK + col] = acc[r][c][i];
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
    lds_barrier();
    for (int idx = tid; idx < T * DX; idx += kThreads) {
      const int e = idx / DX, c = idx % DX;
      const int n = n0 + e;
      float x = 0.f;
      if (n < n_end)
        x = c < DK ? K[((size_t)fh * N + n) * DK + c] : V[((size_t)fh * N + n) * DV + (c - DK)];
      xs[e][c] = x;
      if (c < DK) ys[e][c] = n < n_end ? x * beta[(size_t)fh * N + n] : 0.f;
    }
    lds_barrier();
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
  if (is_f32) {
    const dim3 grid(fh_count * (unsigned)splits);
    hipLaunchKernelGGL((stats_f32_kernel<DK, DV>), grid, dim3(kThreads), 0, stream,
                       static_cast<const float*>(k), static_cast<const float*>(v), beta, N, tps,
                       splits, fh_count, A_part, B_part);
  } else {
    const unsigned nwg = fh_count * (unsigned)splits * 2u;  // two row halves per frame
    hipLaunchKernelGGL((stats_bf16_kernel<DK, DV>), dim3(nwg), dim3(kThreads), 0, stream,
                       static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), beta, N,
                       tps, splits, fh_count, nwg, A_part, B_part);
  }
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
