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
// Convolution kernel: one workgroup per (clip, head, 4 x 8 tile of the
// grid) streams through all frames.  Per input frame it copies the tile and
// its 2-token halo (8 x 12 tokens x d channels) into LDS, double-buffered:
// the next frame's tile is in flight in registers during this frame's
// filters.  Wave w owns grid row w of the
// tile (8 tokens) and each lane two channels (one at d = 64), so a wave
// moves whole 256-byte token rows and the filter taps of a lane's channels
// stay in registers.  The spatial filter reads the 5 x 12 input window row
// by row from LDS.  The temporal filter is a scatter: input frame f adds
// w_t[dt] * S(f) to output frame f - dt + 2, whose running sums sit in a
// five-slot register ring; output frame f - 2 is then complete and is
// finished (SiLU, the L2 reduction across the wave for K) and stored.  So
// every input is read from memory once and every output written once.
//
// Q kernel: each wave normalises four tokens of one head per pass, a lane
// holding eight channels (16-byte loads and stores), with the reduction
// over the 16 lanes of each token.
#include "vda_common.h"
#include "vda_launch.h"

namespace vda {
namespace {

constexpr float kL2Eps = 1e-6f;  // the paper states none
constexpr int kPTY = 4, kPTX = 8;                    // output tile (rows = waves)
constexpr int kPHY = kPTY + 4, kPHX = kPTX + 4;      // with the 2-token halo

__device__ __forceinline__ float silu(float x) { return x / (1.0f + __expf(-x)); }

// Sum over the 64 lanes of a wave (every lane gets the total).
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}

struct PrepConvArgs {
  const uint16_t* in;  // [B][F][N][H*D] bf16
  const float* ws;     // [H*D][25]
  const float* wt;     // [H*D][5]
  uint16_t* out;       // [B*H][F][N][D] bf16
  int F, gh, gw, H, tiles_y, tiles_x;
};

template <int D, bool NORM>
__global__ __launch_bounds__(kThreads, 2)
void prep_conv_kernel(PrepConvArgs a) {
  constexpr int CPL = D / 64;            // channels per lane
  constexpr int TOK = kPHY * kPHX;       // tokens of the haloed tile
  constexpr int CHUNKS = TOK * D * 2 / 16;  // 16-byte pieces of one frame's tile
  __shared__ __align__(16) uint16_t tile[2][TOK * D];

  const int F = a.F, gh = a.gh, gw = a.gw, H = a.H;
  const int N = gh * gw;
  unsigned id = blockIdx.x;
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
  // q % (D / 8) of token q / (D / 8), token (r, s) of the 8 x 12 window at
  // grid (y0 - 2 + r, x0 - 2 + s); tokens off the grid read as zero.  Each
  // thread moves chunks tid + 256 i, loaded into registers one frame ahead
  // and written to LDS after the current frame's filters.
  constexpr int CPT = (CHUNKS + kThreads - 1) / kThreads;  // chunks per thread
  const __amdgpu_buffer_rsrc_t irsrc =
      make_rsrc(a.in + (size_t)b * F * N * C, (uint32_t)((size_t)F * N * C * 2));
  uint32_t coff[CPT];  // byte offset within a frame, or out of range
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int q = tid + kThreads * i;
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
  auto store_frame = [&](uint16_t* dst) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int q = tid + kThreads * i;
      if (CHUNKS % kThreads == 0 || q < CHUNKS) reinterpret_cast<u32x4*>(dst)[q] = stage[i];
    }
  };

  // Output tokens of this wave: grid row y0 + wave, columns x0 .. x0 + 7.
  const int oy = y0 + wave;
  uint16_t* obase = a.out + ((size_t)(b * H + h) * F) * N * D;
  // Running sums of the five pending output frames: after input frame f,
  // slot s belongs to output frame f - 2 + s.
  float ring[5][kPTX][CPL];
#pragma unroll
  for (int s = 0; s < 5; ++s)
#pragma unroll
    for (int x = 0; x < kPTX; ++x)
#pragma unroll
      for (int c = 0; c < CPL; ++c) ring[s][x][c] = 0.f;

  // Input frame f (buffer f % 2): spatial filter, scattered into the ring;
  // then output frame f - 2 (slot 0) is complete, and the ring moves on.
  auto step = [&](int f, const uint16_t* tb) {
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
          const uint16_t* p = tb + ((wave + dy) * kPHX + s) * D + lane * CPL;
          if constexpr (CPL == 2) {
            const uint32_t w2 = *reinterpret_cast<const uint32_t*>(p);
            in[s][0] = bf16_lo(w2);
            in[s][1] = bf16_hi(w2);
          } else {
            in[s][0] = __uint_as_float((uint32_t)*p << 16);
          }
        }
#pragma unroll
        for (int dx = 0; dx < 5; ++dx)
#pragma unroll
          for (int x = 0; x < kPTX; ++x)
#pragma unroll
            for (int c = 0; c < CPL; ++c) sp[x][c] = fmaf(wsp[c][dy * 5 + dx], in[x + dx][c], sp[x][c]);
      }
      // Frame f feeds output frame f + 2 - dt: slot 4 - dt.
#pragma unroll
      for (int dt = 0; dt < 5; ++dt)
#pragma unroll
        for (int x = 0; x < kPTX; ++x)
#pragma unroll
          for (int c = 0; c < CPL; ++c)
            ring[4 - dt][x][c] = fmaf(wtp[c][dt], sp[x][c], ring[4 - dt][x][c]);
    }
    const int o = f - 2;
    if (o >= 0 && o < F) {
      float ssq[kPTX];
#pragma unroll
      for (int x = 0; x < kPTX; ++x) {
        ssq[x] = 0.f;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          const float y = silu(ring[0][x][c]);
          ring[0][x][c] = y;
          ssq[x] = fmaf(y, y, ssq[x]);
        }
      }
      if constexpr (NORM) {
#pragma unroll
        for (int x = 0; x < kPTX; ++x) ssq[x] = rsqrtf(wave_sum(ssq[x]) + kL2Eps);
      }
      if (oy < gh) {
#pragma unroll
        for (int x = 0; x < kPTX; ++x) {
          if (x0 + x < gw) {
            uint16_t* dst = obase + ((size_t)o * N + oy * gw + x0 + x) * D + lane * CPL;
            const float sc = NORM ? ssq[x] : 1.0f;
            if constexpr (CPL == 2)
              *reinterpret_cast<uint32_t*>(dst) = pack_bf16x2(ring[0][x][0] * sc, ring[0][x][1] * sc);
            else
              *dst = (uint16_t)(pack_bf16x2(ring[0][x][0] * sc, 0.f) & 0xffffu);
          }
        }
      }
    }
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int x = 0; x < kPTX; ++x)
#pragma unroll
        for (int c = 0; c < CPL; ++c) ring[s][x][c] = ring[s + 1][x][c];
#pragma unroll
    for (int x = 0; x < kPTX; ++x)
#pragma unroll
      for (int c = 0; c < CPL; ++c) ring[4][x][c] = 0.f;
  };

  // Frame 0's tile; then each frame loads the next one during its filters
  // and writes it to the other buffer (read last one frame ago).  Two more
  // steps than frames flush the last two outputs.
  load_frame(0);
  store_frame(tile[0]);
  lds_barrier();
  for (int f = 0; f < F + 2; ++f) {
    if (f + 1 < F) load_frame(f + 1);  // in flight during this frame's filters
    step(f, tile[f & 1]);
    if (f + 1 < F) store_frame(tile[(f + 1) & 1]);
    lds_barrier();  // next tile complete; this tile's reads done
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
  // Group = (clip, frame, head, block of TPW tokens).
  const int nblocks = (N + TPW - 1) / TPW;
  long long g = grp;
  const int nb = (int)(g % nblocks);
  g /= nblocks;
  const int h = (int)(g % H);
  g /= H;
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
  if (ok) {
    const long long b = bf / F, f = bf % F;
    uint16_t* dst = out + (((size_t)(b * H + h) * F + f) * N + n) * D + j * 8;
    *reinterpret_cast<uint4*>(dst) = make_uint4(pack_bf16x2(x[0] * sc, x[1] * sc), pack_bf16x2(x[2] * sc, x[3] * sc),
                                                pack_bf16x2(x[4] * sc, x[5] * sc), pack_bf16x2(x[6] * sc, x[7] * sc));
  }
}

template <int D, bool NORM>
hipError_t launch_conv_t(const PrepConvArgs& a0, int B, hipStream_t stream) {
  PrepConvArgs a = a0;
  a.tiles_y = (a.gh + kPTY - 1) / kPTY;
  a.tiles_x = (a.gw + kPTX - 1) / kPTX;
  const long long nwg = (long long)B * a.H * a.tiles_y * a.tiles_x;
  hipLaunchKernelGGL((prep_conv_kernel<D, NORM>), dim3((unsigned)nwg), dim3(kThreads), 0, stream, a);
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
  hipError_t e;
  if (d_k == 128)
    e = launch_qnorm_t<128>(q, q_out, B, F, N, H, stream);
  else if (d_k == 64)
    e = launch_qnorm_t<64>(q, q_out, B, F, N, H, stream);
  else
    return hipErrorInvalidValue;
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
