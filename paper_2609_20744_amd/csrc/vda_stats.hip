// Step a1: per-frame statistics A_t = K_t^T Diag(beta_t) K_t and
// B_t = V_t^T Diag(beta_t) K_t (Eq. 3b), computed in one pass over K and V.
//
// One workgroup per frame (and token range).  A_t is symmetric, so only its
// blocks on or above the diagonal are accumulated (16 x 16 blocks (i, j),
// i <= j); each is written transposed to block (j, i), on or below the
// diagonal (the diagonal blocks as their own transposes), and the blocks
// above the diagonal as they are.  When the inverse is A_t's only reader
// (lower_only), those above the diagonal are not stored: the inverse reads
// only the blocks on and below it.  The four
// waves split the work by output columns (channels of beta*k): with 8 column
// blocks, wave w owns columns w and 7 - w, which carry (w + 1) + (8 - w)
// upper-triangle blocks of A_t and 2 * d_v / 16 blocks of B_t: the same count
// for every wave.  Per 32 tokens a wave reads two beta*k operands and the k
// and v row operands its blocks need, so each operand read from LDS feeds
// one or two matrix products.
//
// Both products contract over tokens, the slow axis of the frame-major
// [token][channel] layout.  Tiles of 64 tokens are copied into LDS in that
// natural layout (16-byte coalesced loads, the next tile in flight in
// registers; beta*k is formed per token row in fp32 and rounded to bf16 on
// the way), and the matrix-core operands are read with gfx950's transposing
// LDS read ds_read_b64_tr_b16: within a 16-lane group, lane i returns
// element (i mod 4) of the 64-bit chunks addressed by lanes floor(i/4) + 4e,
// e = 0..3.  If lane j addresses token t0 + floor(j/4) at channel
// c0 + 4 (j mod 4), lane i receives tokens t0..t0+3 of channel c0 + i: one
// half of a v_mfma_f32_16x16x32_bf16 operand column.  Lane group g takes the
// tokens {4g + e} and {16 + 4g + e} of each 32-token step (the same order in
// both operands), which with a row stride of 32 mod 256 bytes keeps the 32
// lanes of one LDS pass on distinct banks.  Tokens past the range are read
// through range-checked buffer loads as zero, so they contribute nothing and
// no load sits behind a branch or feeds a select.
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

// Work item of statistics workgroup L under a split plan (count frames; the
// last `tail` are split into `splits` token ranges, whose workgroups come
// after those of the unsplit frames so that they fill the end of the launch).
struct StatsItem {
  unsigned fh;    // frame-head
  unsigned slot;  // partial matrix index: fh + piece * tail
  int n_begin;    // token range [n_begin, n_end)
  int n_end;
};

__device__ __forceinline__ StatsItem stats_item(unsigned L, unsigned count, unsigned tail,
                                                int splits, int N, int tokens_per_split) {
  const unsigned head = count - tail;
  if (splits <= 1 || L < head) return StatsItem{L, L, 0, N};
  const unsigned u = L - head;
  const unsigned fh = head + u / (unsigned)splits;
  const int piece = (int)(u % (unsigned)splits);
  const int n_begin = piece * tokens_per_split;
  return StatsItem{fh, fh + (unsigned)piece * tail, n_begin, min(N, n_begin + tokens_per_split)};
}

// Output blocks of wave W (compile time).  CB = d_k / 16 column blocks,
// RBV = d_v / 16 row blocks of B_t.  The wave owns the columns col(c),
// c < ncols; in each it accumulates the A_t blocks i = 0 .. col(c) (when
// has_a) and the B_t blocks v_begin .. v_end - 1.
template <int CB, int RBV, int W>
struct WavePlan {
  static constexpr int ncols = CB == 8 ? 2 : 1;
  static constexpr int col(int c) {
    return CB == 8 ? (c == 0 ? W : 7 - W) : (CB == 4 ? W : (W & 1));
  }
  static constexpr bool has_a = CB != 2 || (W >> 1) == 0;
  static constexpr int v_begin = CB == 2 ? (W >> 1) * (RBV / 2) : 0;
  static constexpr int v_end = CB == 2 ? v_begin + RBV / 2 : RBV;
  static constexpr int imax = ncols == 2 ? (col(0) > col(1) ? col(0) : col(1)) : col(0);
};

template <int DK, int DV>
struct StatsFrame {
  static constexpr int LDK = tile_ld(DK);
  static constexpr int LDV = tile_ld(DV);
  static constexpr int KCH = DK / 8;  // 16-byte chunks per K row
  static constexpr int VCH = DV / 8;  // 16-byte chunks per V row
  static constexpr int NKC = kStatsTile * KCH / kThreads;  // K chunks per thread and tile
  static constexpr int NVC = kStatsTile * VCH / kThreads;  // V chunks per thread and tile
  static constexpr int KROWS = kThreads / KCH;
  static constexpr int VROWS = kThreads / VCH;
  static_assert(NKC * kThreads == kStatsTile * KCH && NVC * kThreads == kStatsTile * VCH,
                "chunks divide evenly");

  uint16_t* kt;  // [token][k]          (LDS)
  uint16_t* yt;  // [token][beta * k]   (LDS)
  uint16_t* vt;  // [token][v]          (LDS)
  __amdgpu_buffer_rsrc_t krsrc, vrsrc, brsrc;
  int kc, kr0, vc, vr0, li, lg;

  // Loader roles: chunk i of this thread is (row r0 + i * ROWS, column c),
  // consecutive lanes reading consecutive 16-byte chunks of a row.
  __device__ void load_tile(int n0, u32x4 (&kr)[NKC], float (&kbv)[NKC], u32x4 (&vr)[NVC]) const {
#pragma unroll
    for (int i = 0; i < NKC; ++i) {
      const uint32_t n = (uint32_t)(n0 + kr0 + i * KROWS);
      kr[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                            krsrc, (int)(n * (DK * 2) + kc * 16), 0, 0));
      kbv[i] = load_f32(brsrc, n * 4u);
    }
#pragma unroll
    for (int i = 0; i < NVC; ++i) {
      const uint32_t n = (uint32_t)(n0 + vr0 + i * VROWS);
      vr[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                            vrsrc, (int)(n * (DV * 2) + vc * 16), 0, 0));
    }
  }

  __device__ void store_tile(const u32x4 (&kr)[NKC], const float (&kbv)[NKC],
                             const u32x4 (&vr)[NVC]) const {
#pragma unroll
    for (int i = 0; i < NKC; ++i) {
      const int r = kr0 + i * KROWS;
      const u32x4 w = kr[i];
      const float b = kbv[i];
      *reinterpret_cast<u32x4*>(&yt[r * LDK + kc * 8]) =
          u32x4{scale_pair(w[0], b), scale_pair(w[1], b), scale_pair(w[2], b), scale_pair(w[3], b)};
      *reinterpret_cast<u32x4*>(&kt[r * LDK + kc * 8]) = w;
    }
#pragma unroll
    for (int i = 0; i < NVC; ++i)
      *reinterpret_cast<u32x4*>(&vt[(vr0 + i * VROWS) * LDV + vc * 8]) = vr[i];
  }

  // The whole token loop and the output stores of wave W.
  template <int W>
  __device__ void run(int n_begin, int n_end, float* Ab, float* Bb, bool lower_only) const {
    using P = WavePlan<DK / 16, DV / 16, W>;
    constexpr int NC = P::ncols;
    floatx4 accA[NC][DK / 16];  // [column c][row block i], i <= col(c)
    floatx4 accB[DV / 16][NC];  // [row block v][column c]
#pragma unroll
    for (int c = 0; c < NC; ++c) {
#pragma unroll
      for (int i = 0; i < DK / 16; ++i) accA[c][i] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int v = 0; v < DV / 16; ++v) accB[v][c] = floatx4{0.f, 0.f, 0.f, 0.f};
    }

    // One tile in flight in registers: the next tile's loads are issued as
    // soon as the current one is in LDS, and land during its products.  (A
    // second tile in flight measured slower: 223 against 218 us at 768p; the
    // extra bytes in flight only queue up.)
    u32x4 kraw[NKC];
    float kb[NKC];
    u32x4 vraw[NVC];

    // Move the tile in registers to LDS, refill the registers with tile
    // n_next, and accumulate the tile's products.
    auto tile_step = [&](int n_next, u32x4 (&kr)[NKC], float (&kbv)[NKC], u32x4 (&vr)[NVC]) {
      lds_barrier();  // previous tile's operand reads are done
      store_tile(kr, kbv, vr);
      lds_barrier();
      load_tile(n_next, kr, kbv, vr);
#pragma unroll
      for (int ks = 0; ks < kStatsTile / 32; ++ks) {
        bf16x8 bop[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) bop[c] = tr_operand<LDK>(yt, ks * 32, P::col(c) * 16, li, lg);
        if (P::has_a) {
#pragma unroll
          for (int i = 0; i <= P::imax; ++i) {
            const bf16x8 aop = tr_operand<LDK>(kt, ks * 32, i * 16, li, lg);
#pragma unroll
            for (int c = 0; c < NC; ++c)
              if (i <= P::col(c))
                accA[c][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aop, bop[c], accA[c][i], 0, 0, 0);
          }
        }
#pragma unroll
        for (int v = P::v_begin; v < P::v_end; ++v) {
          const bf16x8 aop = tr_operand<LDV>(vt, ks * 32, v * 16, li, lg);
#pragma unroll
          for (int c = 0; c < NC; ++c)
            accB[v][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aop, bop[c], accB[v][c], 0, 0, 0);
        }
      }
    };

    // Rows past n_end read as zero; the load issued by the last step (past
    // the range) is never consumed.
    if (n_begin < n_end) load_tile(n_begin, kraw, kb, vraw);
    for (int n0 = n_begin; n0 < n_end; n0 += kStatsTile) tile_step(n0 + kStatsTile, kraw, kb, vraw);

    // Block (rows rb, columns cb): lane holds rows 16 rb + 4 lg + e, column
    // 16 cb + li.  The transposed copy of an off-diagonal A_t block puts the
    // four rows of a lane into one 16-byte row piece.
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int j = P::col(c);
      if (P::has_a) {
#pragma unroll
        for (int i = 0; i <= P::imax; ++i) {
          if (i <= P::col(c)) {
            // Block (j, i), on or below the diagonal, as the transpose of the
            // accumulated block (i, j); the diagonal blocks too, so that the
            // blocks the inverse reads are the same in both modes.
            *reinterpret_cast<floatx4*>(&Ab[(j * 16 + li) * DK + i * 16 + lg * 4]) = accA[c][i];
            if (!lower_only && i < P::col(c)) {
#pragma unroll
              for (int e = 0; e < 4; ++e)
                Ab[(i * 16 + lg * 4 + e) * DK + j * 16 + li] = accA[c][i][e];
            }
          }
        }
      }
#pragma unroll
      for (int v = P::v_begin; v < P::v_end; ++v)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          Bb[(v * 16 + lg * 4 + e) * DK + j * 16 + li] = accB[v][c][e];
    }
  }
};

template <int DK, int DV>
__global__ __launch_bounds__(kThreads, 2)
void stats_bf16_kernel(const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
                       const float* __restrict__ beta, int N, int tokens_per_split,
                       unsigned tail, int splits, unsigned fh_count,
                       float* __restrict__ A_part, float* __restrict__ B_part, int lower_only) {
  using S = StatsFrame<DK, DV>;
  __shared__ __align__(16) uint16_t kt[kStatsTile * S::LDK];
  __shared__ __align__(16) uint16_t yt[kStatsTile * S::LDK];
  __shared__ __align__(16) uint16_t vt[kStatsTile * S::LDV];

  const StatsItem it = stats_item(blockIdx.x, fh_count, tail, splits, N, tokens_per_split);
  const unsigned fh = (unsigned)uniform((int)it.fh);
  const unsigned slot = (unsigned)uniform((int)it.slot);
  const int n_begin = uniform(it.n_begin);
  const int n_end = uniform(it.n_end);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)

  S s;
  s.kt = kt;
  s.yt = yt;
  s.vt = vt;
  // Range-checked views of this frame's rows [0, n_end): rows past the end
  // read as zero (so they add nothing to either product), with no clamp or
  // select between a load and its use.
  s.krsrc = make_rsrc(K + (size_t)fh * N * DK, (uint32_t)(n_end * DK * 2));
  s.vrsrc = make_rsrc(V + (size_t)fh * N * DV, (uint32_t)(n_end * DV * 2));
  s.brsrc = make_rsrc(beta + (size_t)fh * N, (uint32_t)(n_end * 4));
  s.kc = tid % S::KCH;
  s.kr0 = tid / S::KCH;
  s.vc = tid % S::VCH;
  s.vr0 = tid / S::VCH;
  s.li = lane & 15;
  s.lg = lane >> 4;

  float* Ab = A_part + (size_t)slot * (DK * DK);
  float* Bb = B_part + (size_t)slot * (DV * DK);
  // Every branch runs the same number of barriers.
  switch (wave) {
    case 0: s.template run<0>(n_begin, n_end, Ab, Bb, lower_only != 0); break;
    case 1: s.template run<1>(n_begin, n_end, Ab, Bb, lower_only != 0); break;
    case 2: s.template run<2>(n_begin, n_end, Ab, Bb, lower_only != 0); break;
    default: s.template run<3>(n_begin, n_end, Ab, Bb, lower_only != 0); break;
  }
}

// fp32 storage: plain fp32 products and sums (no rounding of beta * k).
// The output X = [A_t; B_t] ((d_k + d_v) x d_k) is dealt out to the threads
// in R x C register tiles (C = 8 columns, 4 for d_k = 32), so each token
// costs a thread R + C LDS reads for R * C fused multiply-adds.  A tile of
// 32 tokens of k, v and beta is loaded by range-checked buffer loads that
// are all in flight together (tokens past the range read as zero), then
// staged in LDS; every output sums its tokens in order.
template <int DK, int DV>
__global__ __launch_bounds__(kThreads)
void stats_f32_kernel(const float* __restrict__ K, const float* __restrict__ V,
                      const float* __restrict__ beta, int N, int tokens_per_split,
                      unsigned tail, int splits, unsigned fh_count,
                      float* __restrict__ A_part, float* __restrict__ B_part) {
  constexpr int DX = DK + DV;
  constexpr int T = 32;
  constexpr int C = DK >= 64 ? 8 : 4;          // columns per thread
  constexpr int CG = DK / C;                   // column groups
  constexpr int R = DX * CG / kThreads;        // rows per thread
  static_assert(R * C * kThreads == DX * DK, "register tiles cover the output");
  constexpr int LPT = T * DX / kThreads;       // loaded elements per thread and tile
  static_assert(LPT * kThreads == T * DX, "tile loads divide evenly");
  __shared__ __align__(16) float xs[T][DX];
  __shared__ __align__(16) float ys[T][DK];

  const StatsItem it = stats_item(blockIdx.x, fh_count, tail, splits, N, tokens_per_split);
  const unsigned fh = (unsigned)uniform((int)it.fh);
  const int n_begin = uniform(it.n_begin);
  const int n_end = uniform(it.n_end);
  const int tid = threadIdx.x;
  const __amdgpu_buffer_rsrc_t krsrc = make_rsrc(K + (size_t)fh * N * DK, (uint32_t)(n_end * DK * 4));
  const __amdgpu_buffer_rsrc_t vrsrc = make_rsrc(V + (size_t)fh * N * DV, (uint32_t)(n_end * DV * 4));
  const __amdgpu_buffer_rsrc_t brsrc = make_rsrc(beta + (size_t)fh * N, (uint32_t)(n_end * 4));
  const int j0 = (tid % CG) * C;
  const int x0 = (tid / CG) * R;

  float acc[R][C];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int c = 0; c < C; ++c) acc[r][c] = 0.f;

  for (int n0 = n_begin; n0 < n_end; n0 += T) {
    float xv[LPT], bv[LPT];
#pragma unroll
    for (int l = 0; l < LPT; ++l) {
      const int idx = tid + l * kThreads;
      const int e = idx / DX, c = idx % DX;
      const uint32_t n = (uint32_t)(n0 + e);
      xv[l] = c < DK ? load_f32(krsrc, (n * DK + c) * 4u) : load_f32(vrsrc, (n * DV + c - DK) * 4u);
      bv[l] = load_f32(brsrc, n * 4u);
    }
    lds_barrier();  // the previous tile's reads are done
#pragma unroll
    for (int l = 0; l < LPT; ++l) {
      const int idx = tid + l * kThreads;
      const int e = idx / DX, c = idx % DX;
      xs[e][c] = xv[l];
      if (c < DK) ys[e][c] = xv[l] * bv[l];
    }
    lds_barrier();
#pragma unroll 4
    for (int e = 0; e < T; ++e) {
      float xr[R], yc[C];
#pragma unroll
      for (int r = 0; r < R; ++r) xr[r] = xs[e][x0 + r];
#pragma unroll
      for (int c = 0; c < C; ++c) yc[c] = ys[e][j0 + c];
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int c = 0; c < C; ++c) acc[r][c] = fmaf(xr[r], yc[c], acc[r][c]);
    }
  }
  float* Ab = A_part + (size_t)it.slot * (DK * DK);
  float* Bb = B_part + (size_t)it.slot * (DV * DK);
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int x = x0 + r;
    float* dst = x < DK ? Ab + (size_t)x * DK + j0 : Bb + (size_t)(x - DK) * DK + j0;
#pragma unroll
    for (int c = 0; c < C; c += 4)
      *reinterpret_cast<float4*>(dst + c) = make_float4(acc[r][c], acc[r][c + 1], acc[r][c + 2],
                                                        acc[r][c + 3]);
  }
}

template <int DK, int DV>
int blocks_per_cu_t(bool is_f32) {
  int n = 0;
  const void* fn = is_f32 ? reinterpret_cast<const void*>(&stats_f32_kernel<DK, DV>)
                          : reinterpret_cast<const void*>(&stats_bf16_kernel<DK, DV>);
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, kThreads, 0) != hipSuccess) return 1;
  return n;
}

template <int DK, int DV>
hipError_t launch_stats_t(bool is_f32, const void* k, const void* v, const float* beta,
                          int F, int N, int H, SplitPlan plan, float* A_part, float* B_part,
                          bool lower_only, hipStream_t stream) {
  const unsigned fh_count = (unsigned)H * (unsigned)F;
  const int splits = plan.splits > 1 && plan.tail > 0 ? plan.splits : 1;
  const unsigned tail = splits > 1 ? (unsigned)plan.tail : 0u;
  const int tps = stats_tokens_per_split(N, splits);
  const dim3 grid((unsigned)stats_workgroups(fh_count, SplitPlan{(int)tail, splits}));
  if (is_f32) {
    hipLaunchKernelGGL((stats_f32_kernel<DK, DV>), grid, dim3(kThreads), 0, stream,
                       static_cast<const float*>(k), static_cast<const float*>(v), beta, N, tps,
                       tail, splits, fh_count, A_part, B_part);
  } else {
    hipLaunchKernelGGL((stats_bf16_kernel<DK, DV>), grid, dim3(kThreads), 0, stream,
                       static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), beta, N,
                       tps, tail, splits, fh_count, A_part, B_part, (int)lower_only);
  }
  return hipGetLastError();
}

}  // namespace

int stats_blocks_per_cu(bool is_f32, int d_k, int d_v) {
#define VDA_OCC_CASE(DKV, DVV) \
  if (d_k == DKV && d_v == DVV) return blocks_per_cu_t<DKV, DVV>(is_f32);
  VDA_OCC_CASE(32, 32) VDA_OCC_CASE(32, 64) VDA_OCC_CASE(32, 128)
  VDA_OCC_CASE(64, 32) VDA_OCC_CASE(64, 64) VDA_OCC_CASE(64, 128)
  VDA_OCC_CASE(128, 32) VDA_OCC_CASE(128, 64) VDA_OCC_CASE(128, 128)
#undef VDA_OCC_CASE
  return 1;
}

hipError_t launch_frame_stats(bool is_f32, const void* k, const void* v, const float* beta,
                              int F, int N, int H, int d_k, int d_v, SplitPlan plan,
                              float* A_part, float* B_part, hipStream_t stream,
                              bool lower_only) {
#define VDA_STATS_CASE(DKV, DVV)                                                       \
  if (d_k == DKV && d_v == DVV)                                                        \
    return launch_stats_t<DKV, DVV>(is_f32, k, v, beta, F, N, H, plan, A_part, B_part, \
                                    lower_only, stream);
  VDA_STATS_CASE(32, 32) VDA_STATS_CASE(32, 64) VDA_STATS_CASE(32, 128)
  VDA_STATS_CASE(64, 32) VDA_STATS_CASE(64, 64) VDA_STATS_CASE(64, 128)
  VDA_STATS_CASE(128, 32) VDA_STATS_CASE(128, 64) VDA_STATS_CASE(128, 128)
#undef VDA_STATS_CASE
  return hipErrorInvalidValue;
}

}  // namespace vda
