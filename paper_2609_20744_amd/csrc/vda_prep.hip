// VDA-Prep (Section 2.3; the fused prep step of Section 4): the linear
// branch's feature map from the QKV projections to the operator's layout.
//     K' = L2(SiLU(T_k * S_k * K)),  V' = SiLU(T_v * S_v * V),  Q' = L2(Q)
// S is a depthwise 5 x 5 spatial filter over the latent grid of each frame,
// T a depthwise five-tap temporal filter over frames (both centred cross-
// correlations with zero padding), L2 the normalisation x / sqrt(|x|^2 +
// eps) over the d channels of one token of one head.  Inputs are the
// token-major projections [B][F][gh*gw][H*d] (bf16); outputs are frame-major
// per head, [B*H][F][gh*gw][d] (bf16), the layout the operator reads.
//
// Convolution kernel: one workgroup of eight waves per (clip, head, 8 x 8
// tile of the grid) streams through all frames.  Per input frame it copies
// the tile and its 2-token halo (12 x 12 tokens x d channels) into LDS,
// expanded to fp32 once, double-buffered: the next frame's tile is in
// flight in registers during this frame's filters.  Wave w owns grid row w
// of the tile (8 tokens) and each lane two channels (one at d = 64), so a
// wave moves whole token rows and the filter taps of a lane's channels stay
// in registers.  The spatial filter reads the 5 x 12 input window row by
// row from LDS.  The temporal filter is a scatter: input frame f adds
// w_t[dt] * S(f) to output frame f - dt + 2, whose running sums sit in a
// five-slot register ring indexed by frame mod 5 (the frame loop is
// unrolled five times so every slot index is a constant); output frame
// f - 2 is then complete and is finished (SiLU, the L2 reduction across the
// wave for K) and stored.  Every input is read from memory once per tile
// that needs it (tiles sharing a halo run on one XCD, so the re-reads hit
// its L2) and every output is written once.  The work is bound by the fp32
// FMAs (25 + 5 per output channel).
//
// Q kernel: each wave normalises four tokens of one head per pass, a lane
// holding eight channels (16-byte loads and stores), with the reduction
// over the 16 lanes of each token.
#include <type_traits>

#include "vda_common.h"
#include "vda_launch.h"

namespace vda {
namespace {

constexpr int kConvThreads = 512;                    // eight waves, one output row each
constexpr int kPTY = 8, kPTX = 8;                    // output tile (rows = waves)
constexpr int kPHY = kPTY + 4, kPHX = kPTX + 4;      // with the 2-token halo
static_assert(kPTX == 8, "the L2 reduction sums eight tokens per wave row");

// SiLU with the hardware reciprocal (1 ulp): for x -> -inf, exp(-x)
// overflows to inf and the result is -0, the limit.
__device__ __forceinline__ float silu(float x) {
  return x * __builtin_amdgcn_rcpf(1.0f + __expf(-x));
}

#define VDA_DPP(v, ctrl) __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), ctrl, 0xf, 0xf, false))

// Sum over all 64 lanes of the two 32-lane halves' and four 16-lane rows'
// copies: lanes 8 apart by DPP row_ror 8, then the 16- and 32-lane row
// swaps of gfx950.  A swap of a register with itself leaves one lane's own
// value in one result and its partner's in the other, so their sum is the
// pair's sum in every lane.
__device__ __forceinline__ float sum_lanes_8_apart(float x) {
  x += VDA_DPP(x, 0x128);  // row_ror 8
  const uint32_t u = __float_as_uint(x);
  const auto r16 = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  x = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);
  const uint32_t w = __float_as_uint(x);
  const auto r32 = __builtin_amdgcn_permlane32_swap(w, w, false, false);
  return __uint_as_float(r32[0]) + __uint_as_float(r32[1]);
}

// Totals over the wave of eight per-token values: v[x] is this lane's part
// of token x; the result in every lane is the total of token lane % 8.
// Three halving exchanges (partners lane ^ 1, lane ^ 2, and lane + 4 within
// each row of 16, which pairs lanes holding the same tokens) leave each lane
// one token's partial sum; adding lanes 8 apart completes it.
__device__ __forceinline__ float token_totals8(const float (&v)[8], int lane) {
  const bool b0 = lane & 1, b1 = lane & 2, b2 = lane & 4;
  float w[4], u[2];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float a = v[2 * j] + VDA_DPP(v[2 * j], 0xb1);          // quad_perm [1,0,3,2]
    const float b = v[2 * j + 1] + VDA_DPP(v[2 * j + 1], 0xb1);
    w[j] = b0 ? b : a;  // token 2j + b0
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const float a = w[2 * i] + VDA_DPP(w[2 * i], 0x4e);          // quad_perm [2,3,0,1]
    const float b = w[2 * i + 1] + VDA_DPP(w[2 * i + 1], 0x4e);
    u[i] = b1 ? b : a;  // token 4i + 2 b1 + b0
  }
  const float a = u[0] + VDA_DPP(u[0], 0x124);                   // row_ror 4
  const float b = u[1] + VDA_DPP(u[1], 0x124);
  return sum_lanes_8_apart(b2 ? b : a);  // token lane % 8
}

#undef VDA_DPP

struct PrepConvArgs {
  const uint16_t* in;  // [B][F][N][H*D] bf16
  const float* ws;     // [H*D][25]
  const float* wt;     // [H*D][5]
  uint16_t* out;       // [B*H][F][N][D] bf16
  int F, gh, gw, H, tiles_y, tiles_x;
};

template <int D, bool NORM>
__global__ __launch_bounds__(kConvThreads, 1)
void prep_conv_kernel(PrepConvArgs a) {
  constexpr int CPL = D / 64;            // channels per lane
  constexpr int TOK = kPHY * kPHX;       // tokens of the haloed tile
  constexpr int CHUNKS = TOK * D * 2 / 16;  // 16-byte bf16 pieces of one frame's tile
  // Two frames of the haloed tile, expanded to fp32 once when written.
  __shared__ __align__(16) float tile[2][TOK * D];

  const int F = a.F, gh = a.gh, gw = a.gw, H = a.H;
  const int N = gh * gw;
  // Consecutive tiles (x fastest) share halos: keep them on one XCD.
  unsigned id = xcd_grouped_id(blockIdx.x, gridDim.x);
  const int tx = id % a.tiles_x;
  id /= a.tiles_x;
  const int ty = id % a.tiles_y;
  id /= a.tiles_y;
  const int h = id % H;
  const int b = id / H;
  const int y0 = ty * kPTY, x0 = tx * kPTX;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // this wave's output row
  const int C = H * D;

  // Filter taps of this lane's channels.
  float wsp[CPL][25], wtp[CPL][5];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int ch = h * D + lane * CPL + c;
#pragma unroll
    for (int i = 0; i < 25; ++i) wsp[c][i] = a.ws[(size_t)ch * 25 + i];
#pragma unroll
    for (int i = 0; i < 5; ++i) wtp[c][i] = a.wt[(size_t)ch * 5 + i];
  }

  // One input frame's haloed tile: chunk q (16 bytes) of the tile is piece
  // q % (D / 8) of token q / (D / 8), token (r, s) of the 12 x 12 window at
  // grid (y0 - 2 + r, x0 - 2 + s); tokens off the grid read as zero.  Each
  // thread moves chunks tid + 512 i, loaded into registers one frame ahead
  // and written to LDS as eight fp32 values after the current frame's
  // filters.
  constexpr int CPT = (CHUNKS + kConvThreads - 1) / kConvThreads;  // chunks per thread
  const __amdgpu_buffer_rsrc_t irsrc =
      make_rsrc(a.in + (size_t)b * F * N * C, (uint32_t)((size_t)F * N * C * 2));
  uint32_t coff[CPT];  // byte offset within a frame, or out of range
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int q = tid + kConvThreads * i;
    const int tok = q / (D / 8), piece = q % (D / 8);
    const int r = tok / kPHX, s = tok % kPHX;
    const int gy = y0 - 2 + r, gx = x0 - 2 + s;
    const bool in = q < CHUNKS && gy >= 0 && gy < gh && gx >= 0 && gx < gw;
    coff[i] = in ? (uint32_t)(((gy * gw + gx) * C + h * D + piece * 8) * 2) : kOutOfRange;
  }
  u32x4 stage[CPT];
  auto load_frame = [&](int f) {
    const uint32_t fb = (uint32_t)f * (uint32_t)(N * C * 2);
#pragma unroll
    for (int i = 0; i < CPT; ++i)
      stage[i] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                     irsrc, (int)(coff[i] == kOutOfRange ? kOutOfRange : fb + coff[i]), 0, 0));
  };
  auto store_frame = [&](float* dst) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int q = tid + kConvThreads * i;
      if (CHUNKS % kConvThreads == 0 || q < CHUNKS) {
        const u32x4 w = stage[i];
        float4* d4 = reinterpret_cast<float4*>(dst + q * 8);
        d4[0] = make_float4(bf16_lo(w[0]), bf16_hi(w[0]), bf16_lo(w[1]), bf16_hi(w[1]));
        d4[1] = make_float4(bf16_lo(w[2]), bf16_hi(w[2]), bf16_lo(w[3]), bf16_hi(w[3]));
      }
    }
  };

  // Output tokens of this wave: grid row y0 + wave, columns x0 .. x0 + 7.
  const int oy = y0 + wave;
  uint16_t* obase = a.out + ((size_t)(b * H + h) * F) * N * D;
  const __amdgpu_buffer_rsrc_t orsrc = make_rsrc(obase, (uint32_t)((size_t)F * N * D * 2));
  // Running sums of the pending output frames: output frame o lives in
  // slot o % 5.  Slots start at zero (outputs 0 and 1 take their first
  // terms by accumulation); the slot of output f + 2 is set, not added to,
  // by input frame f, since output f - 3 left it one frame earlier.
  float ring[5][kPTX][CPL];
#pragma unroll
  for (int s = 0; s < 5; ++s)
#pragma unroll
    for (int x = 0; x < kPTX; ++x)
#pragma unroll
      for (int c = 0; c < CPL; ++c) ring[s][x][c] = 0.f;

  // Input frame f = f0 + P with f0 a multiple of 5, from buffer f % 2:
  // spatial filter, then the temporal scatter (frame f adds w_t[dt] S(f)
  // to output f + 2 - dt); output f - 2 is then complete.
  auto step = [&](auto phase, int f) {
    constexpr int P = decltype(phase)::value;
    const float* tb = tile[f & 1];
    if (f < F) {
      float sp[kPTX][CPL];
#pragma unroll
      for (int x = 0; x < kPTX; ++x)
#pragma unroll
        for (int c = 0; c < CPL; ++c) sp[x][c] = 0.f;
#pragma unroll
      for (int dy = 0; dy < 5; ++dy) {
        float in[kPHX][CPL];
#pragma unroll
        for (int s = 0; s < kPHX; ++s) {
          const float* p = tb + ((wave + dy) * kPHX + s) * D + lane * CPL;
          if constexpr (CPL == 2) {
            const float2 v2 = *reinterpret_cast<const float2*>(p);
            in[s][0] = v2.x;
            in[s][1] = v2.y;
          } else {
            in[s][0] = *p;
          }
        }
#pragma unroll
        for (int dx = 0; dx < 5; ++dx)
#pragma unroll
          for (int x = 0; x < kPTX; ++x)
#pragma unroll
            for (int c = 0; c < CPL; ++c) sp[x][c] = fmaf(wsp[c][dy * 5 + dx], in[x + dx][c], sp[x][c]);
      }
#pragma unroll
      for (int x = 0; x < kPTX; ++x)
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          ring[(P + 2) % 5][x][c] = wtp[c][0] * sp[x][c];
#pragma unroll
          for (int dt = 1; dt < 5; ++dt)
            ring[(P + 2 - dt + 5) % 5][x][c] = fmaf(wtp[c][dt], sp[x][c], ring[(P + 2 - dt + 5) % 5][x][c]);
        }
    }
    const int o = f - 2;
    constexpr int OS = (P + 3) % 5;  // slot of output f - 2
    if (o >= 0 && o < F) {
      float y[kPTX][CPL], scale[kPTX];
#pragma unroll
      for (int x = 0; x < kPTX; ++x) {
        scale[x] = 0.f;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          y[x][c] = silu(ring[OS][x][c]);
          scale[x] = fmaf(y[x][c], y[x][c], scale[x]);
        }
      }
      if constexpr (NORM) {
        // Lane x holds token x's 1 / sqrt(|y|^2 + eps); broadcast all eight.
        const float own = rsqrtf(token_totals8(scale, lane) + kL2Eps);
#pragma unroll
        for (int x = 0; x < kPTX; ++x)
          scale[x] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(own), x));
      } else {
#pragma unroll
        for (int x = 0; x < kPTX; ++x) scale[x] = 1.0f;
      }
      if (oy < gh) {
#pragma unroll
        for (int x = 0; x < kPTX; ++x) {
          if (x0 + x < gw) {
            // Streamed stores (sc0 | nt | sc1): the features are read by the
            // next kernels, not kept dirty in the caches for them to evict.
            const uint32_t off = (uint32_t)((((size_t)o * N + oy * gw + x0 + x) * D + lane * CPL) * 2);
            if constexpr (CPL == 2)
              __builtin_amdgcn_raw_buffer_store_b32(pack_bf16x2(y[x][0] * scale[x], y[x][1] * scale[x]),
                                                    orsrc, (int)off, 0, 1 | 2 | 16);
            else
              __builtin_amdgcn_raw_buffer_store_b16(
                  (uint16_t)(pack_bf16x2(y[x][0] * scale[x], 0.f) & 0xffffu), orsrc, (int)off, 0,
                  1 | 2 | 16);
          }
        }
      }
    }
  };
  // One frame: the next frame's tile is in flight during this frame's
  // filters and is written to the other buffer (read last one frame ago).
  auto frame = [&](auto phase, int f) {
    if (f >= F + 2) return;
    if (f + 1 < F) load_frame(f + 1);
    step(phase, f);
    if (f + 1 < F) store_frame(tile[(f + 1) & 1]);
    lds_barrier();  // next tile complete; this tile's reads done
  };

  load_frame(0);
  store_frame(tile[0]);
  lds_barrier();
  // Two more frames than inputs flush the last two outputs.
  for (int f0 = 0; f0 < F + 2; f0 += 5) {
    frame(std::integral_constant<int, 0>{}, f0);
    frame(std::integral_constant<int, 1>{}, f0 + 1);
    frame(std::integral_constant<int, 2>{}, f0 + 2);
    frame(std::integral_constant<int, 3>{}, f0 + 3);
    frame(std::integral_constant<int, 4>{}, f0 + 4);
  }
}

// Q: L2-normalise each token of each head and lay it out frame-major.
template <int D>
__global__ __launch_bounds__(kThreads)
void prep_qnorm_kernel(const uint16_t* __restrict__ in, uint16_t* __restrict__ out, int F, int N,
                       int H, long long total_groups) {
  constexpr int LPT = D / 8;      // lanes per token (8 channels each)
  constexpr int TPW = 64 / LPT;   // tokens per wave pass
  const int lane = threadIdx.x & 63;
  const long long grp = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);  // one wave pass each
  if (grp >= total_groups) return;
  // Group = (clip, frame, block of TPW tokens, head).
  const int nblocks = (N + TPW - 1) / TPW;
  long long g = grp;
  // Heads fastest: consecutive waves read one token's head slices in turn,
  // so the reads of a frame run sequentially through memory.
  const int h = (int)(g % H);
  g /= H;
  const int nb = (int)(g % nblocks);
  g /= nblocks;
  const long long bf = g;  // clip * F + frame
  const int t = lane / LPT, j = lane % LPT;
  const int n = nb * TPW + t;
  const bool ok = n < N;
  const int C = H * D;
  float x[8];
  if (ok) {
    const uint4 v = *reinterpret_cast<const uint4*>(in + ((size_t)bf * N + n) * C + h * D + j * 8);
    const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = bf16_lo(w4[i]);
      x[2 * i + 1] = bf16_hi(w4[i]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = 0.f;
  }
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) ss = fmaf(x[i], x[i], ss);
#pragma unroll
  for (int m = LPT / 2; m >= 1; m >>= 1) ss += __shfl_xor(ss, m);
  const float sc = rsqrtf(ss + kL2Eps);
  // This wave's TPW output rows, streamed (sc0 | nt | sc1) like the
  // convolutions' outputs; rows past the frame fall outside the range.
  const long long b = bf / F, f = bf % F;
  const uint16_t* wbase = out + (((size_t)(b * H + h) * F + f) * N + (size_t)nb * TPW) * D;
  const __amdgpu_buffer_rsrc_t orsrc =
      make_rsrc(wbase, (uint32_t)((min(N - nb * TPW, TPW)) * D * 2));
  const u32x4 packed = {pack_bf16x2(x[0] * sc, x[1] * sc), pack_bf16x2(x[2] * sc, x[3] * sc),
                        pack_bf16x2(x[4] * sc, x[5] * sc), pack_bf16x2(x[6] * sc, x[7] * sc)};
  store_b128_stream(orsrc, ok ? (uint32_t)((t * D + j * 8) * 2) : kOutOfRange, packed);
}

template <int D, bool NORM>
hipError_t launch_conv_t(const PrepConvArgs& a0, int B, hipStream_t stream) {
  PrepConvArgs a = a0;
  a.tiles_y = (a.gh + kPTY - 1) / kPTY;
  a.tiles_x = (a.gw + kPTX - 1) / kPTX;
  const long long nwg = (long long)B * a.H * a.tiles_y * a.tiles_x;
  hipLaunchKernelGGL((prep_conv_kernel<D, NORM>), dim3((unsigned)nwg), dim3(kConvThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_conv(const PrepConvArgs& a, int B, int D, bool norm, hipStream_t stream) {
  if (D == 128) return norm ? launch_conv_t<128, true>(a, B, stream) : launch_conv_t<128, false>(a, B, stream);
  if (D == 64) return norm ? launch_conv_t<64, true>(a, B, stream) : launch_conv_t<64, false>(a, B, stream);
  return hipErrorInvalidValue;
}

template <int D>
hipError_t launch_qnorm_t(const void* q, void* out, int B, int F, int N, int H, hipStream_t stream) {
  constexpr int TPW = 64 / (D / 8);
  const long long groups = (long long)B * F * H * ((N + TPW - 1) / TPW);
  const long long nwg = (groups + 3) / 4;
  hipLaunchKernelGGL(prep_qnorm_kernel<D>, dim3((unsigned)nwg), dim3(kThreads), 0, stream,
                     static_cast<const uint16_t*>(q), static_cast<uint16_t*>(out), F, N, H, groups);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_prep(const void* q, const void* k, const void* v, const float* wks,
                       const float* wkt, const float* wvs, const float* wvt, int B, int F, int gh,
                       int gw, int H, int d_k, int d_v, void* q_out, void* k_out, void* v_out,
                       hipStream_t stream) {
  const int N = gh * gw;
  hipError_t e = hipSuccess;
  if (d_k != 128 && d_k != 64) return hipErrorInvalidValue;
  if (q && d_k == 128)
    e = launch_qnorm_t<128>(q, q_out, B, F, N, H, stream);
  else if (q)
    e = launch_qnorm_t<64>(q, q_out, B, F, N, H, stream);
  if (e != hipSuccess) return e;
  PrepConvArgs a{};
  a.F = F;
  a.gh = gh;
  a.gw = gw;
  a.H = H;
  a.in = static_cast<const uint16_t*>(k);
  a.ws = wks;
  a.wt = wkt;
  a.out = static_cast<uint16_t*>(k_out);
  e = launch_conv(a, B, d_k, true, stream);
  if (e != hipSuccess) return e;
  a.in = static_cast<const uint16_t*>(v);
  a.ws = wvs;
  a.wt = wvt;
  a.out = static_cast<uint16_t*>(v_out);
  return launch_conv(a, B, d_v, false, stream);
}

}  // namespace vda
