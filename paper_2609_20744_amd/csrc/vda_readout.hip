// Steps a5-a7: gather, readout, RMSNorm and gate.
//   S~_t = P_{t-1} + R_{t+1}            (Eq. A.4 with the window [t, t], alpha = 1)
//   o_{t,u} = S~_t q_{t,u}               (Eq. 1a)
//   y_{t,u} = G * o / sqrt(mean(o^2) + eps)      (Eq. 1c)
// G is the per-head gate, or (TOKGATE) the output gate G^L per token and
// channel, read beside the queries.
//
// bf16 path: a workgroup owns one frame of one head and every `chunks`-th
// 64-token super-group of it (the frame's workgroups sweep it together).
// It sums the two fp32 states, rounds S~ to bf16 once into LDS, and
// each wavefront keeps all of S~ as MFMA A-operands in registers.  It then
// streams 16-token groups: the group's queries are the B-operand (16-byte
// loads straight from HBM, two groups in flight per wave), O^T = S~ Q^T is
// accumulated in fp32 by v_mfma_f32_16x16x32_bf16, and the RMSNorm over the
// d_v outputs of a token is a lane-local sum plus two cross-lane exchanges.
// The normalised, gated values are rounded to bf16 into a per-wave LDS tile
// of the group's 16 token rows, from which each 16-byte-per-lane streaming
// store writes consecutive whole token rows (one contiguous run of up to
// 1 KB when the output is frame-major per head; with the token-major output
// of the epilogue's layout conversion, a head's rows sit out_heads * d_v
// apart and each is one run of d_v values).
#include "vda_common.h"
#include "vda_launch.h"

namespace vda {
namespace {

// Local window [lo, hi] of frame f (0-based, clipped to [0, F)): the frame's
// chunk of `chunk` frames (counted from `offset` positions before frame 0)
// and `radius` chunks on each side (Eq. A.4's [l_t, h_t]).
struct Window {
  int lo, hi;
};

__device__ __forceinline__ Window local_window(int f, int F, int chunk, int radius, int offset) {
  const int c = (f + offset) / chunk;
  const int lo = (c - radius) * chunk - offset;
  const int hi = (c + radius + 1) * chunk - offset - 1;
  return Window{max(0, lo), min(F - 1, hi)};
}

// Decay bridge factors of Eq. A.4 for key channels j .. j + W - 1 of head h:
// df = prod_{r = lo..f} alpha_r, dr = prod_{r = f..hi} alpha_r.
template <int W>
__device__ __forceinline__ void bridge_decay(const float* alpha, int h, int F, int DKr, int j,
                                             int f, Window w, float (&df)[W], float (&dr)[W]) {
#pragma unroll
  for (int c = 0; c < W; ++c) df[c] = dr[c] = 1.0f;
  if (alpha == nullptr) return;
  const float* a = alpha + (size_t)h * F * DKr + j;
  for (int r = w.lo; r <= w.hi; ++r) {
#pragma unroll
    for (int c = 0; c < W; ++c) {
      const float x = a[(size_t)r * DKr + c];
      if (r <= f) df[c] *= x;
      if (r >= f) dr[c] *= x;
    }
  }
}

// GENOUT: the general layouts (the token-major output, a padded narrow
// head: row stride and stored channels at run time; a token-major raw query,
// qh heads per clip, L2-normalised here when ql2); otherwise frame-major rows
// of DK and DV channels.
template <int DK, int DV, bool TOKGATE, bool GENOUT>
__global__ __launch_bounds__(kThreads, 2)
void readout_bf16_kernel(const uint16_t* __restrict__ Q, const float* __restrict__ S_fwd,
                         const float* __restrict__ S_rev, const float* __restrict__ gate,
                         int F, int N, int chunks, int tokens_per_chunk, unsigned nwg,
                         int dvo, int oh, int qh, int ql2, const float* __restrict__ alpha,
                         int wchunk, int wradius, int woffset, const uint16_t* __restrict__ gtok,
                         uint16_t* __restrict__ out) {
  constexpr int SLD = DK + 8;  // bf16 row stride of S~ in LDS
  constexpr int MB = DV / 16;  // 16-row blocks of S~ (output channels)
  constexpr int KB = DK / 32;  // 32-wide k steps
  constexpr int OLD = DV + 8;  // bf16 row stride of the output staging tiles
  __shared__ __align__(16) uint16_t st[DV * SLD];
  __shared__ __align__(16) uint16_t otile[4 * 16 * OLD];  // one 16-token tile per wave

  // The chunks of one frame read the same two states: keep them on one XCD.
  const unsigned L = xcd_grouped_id(blockIdx.x, nwg);
  const unsigned fh = L / chunks;
  const int chunk = L % chunks;
  const float g = TOKGATE ? 1.0f : gate[fh / F];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int li = lane & 15;
  const int lg = lane >> 4;

  {
    // Gather (Eq. A.4): the forward state entering the frame's local window
    // and the reverse state leaving it, each decayed across the skipped
    // frames (the own frame only, with alpha = 1, in the core operator).
    const int h = (int)(fh / F), f = (int)(fh % F);
    const Window w = local_window(f, F, wchunk, wradius, woffset);
    const float* sf = S_fwd + ((size_t)h * F + w.lo) * (DV * DK);
    const float* sr = S_rev + ((size_t)h * F + w.hi) * (DV * DK);
    // This thread's columns are the same in every iteration below.
    static_assert((kThreads * 4) % DK == 0, "fixed columns per thread");
    float df[4], dr[4];
    bridge_decay<4>(alpha, h, F, DK, (tid * 4) % DK, f, w, df, dr);
    // Fully unrolled (a compile-time trip count; DV * DK is a multiple of
    // kThreads * 4), so all of a thread's loads are in flight together.
    static_assert((DV * DK) % (kThreads * 4) == 0, "state size");
#pragma unroll
    for (int it = 0; it < (DV * DK) / (kThreads * 4); ++it) {
      const int idx = tid * 4 + it * (kThreads * 4);
      const float4 a = *reinterpret_cast<const float4*>(sf + idx);
      const float4 b = *reinterpret_cast<const float4*>(sr + idx);
      const int i = idx / DK, j = idx % DK;
      *reinterpret_cast<uint2*>(&st[i * SLD + j]) =
          make_uint2(pack_bf16x2(a.x * df[0] + b.x * dr[0], a.y * df[1] + b.y * dr[1]),
                     pack_bf16x2(a.z * df[2] + b.z * dr[2], a.w * df[3] + b.w * dr[3]));
    }
  }
  lds_barrier();

  // S~ as MFMA A-operands: held in registers on the plain frame-major path;
  // the gated and general-layout variants read them from LDS at each group
  // instead, which leaves them the registers for two query groups in flight.
  constexpr bool kSopRegs = !GENOUT && !TOKGATE;
  bf16x8 sop[kSopRegs ? MB : 1][kSopRegs ? KB : 1];
  if constexpr (kSopRegs) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
        sop[mb][kb] = *reinterpret_cast<const bf16x8*>(&st[(mb * 16 + li) * SLD + kb * 32 + lg * 8]);
  }
  const uint16_t* sop_lds = &st[li * SLD + lg * 8];

  // This frame's query rows: DK channels at row stride qh * DK, from head
  // h % qh of clip h / qh (frame-major per head when qh = 1).
  const unsigned qhu = GENOUT ? (unsigned)qh : 1u, hp = fh / F, fr = fh % F;
  const uint32_t qrs = qhu * (uint32_t)DK;
  const uint16_t* qbase = Q + (((size_t)(hp / qhu) * F + fr) * N * qhu + hp % qhu) * DK;
  // This frame's output rows: dvo channels at row stride oh * dvo, likewise.
  const unsigned ohu = GENOUT ? (unsigned)oh : 1u;
  const int dvw = GENOUT ? dvo : DV;
  const uint32_t ors = ohu * (uint32_t)dvw;
  uint16_t* obase = out + (((size_t)(hp / ohu) * F + fr) * N * ohu + hp % ohu) * dvw;
  const float inv_norm = 1.0f / (float)dvw;

  // The frame's tokens go in 64-token super-groups, dealt out to its
  // `chunks` workgroups in turn (super-group c, c + chunks, ...), so the
  // workgroups of one frame sweep it together and the device streams a
  // compact address window; within a super-group wave w takes the 16-token
  // group at 16 w.  The queries of a wave's next kQ groups are in flight in
  // a register ring (slot d: group n0 + S*d, S = 64 * chunks tokens apart).
  // Rows past the frame are clamped onto its last row (always valid
  // memory); their outputs are dropped by the range-checked stores, so
  // loads and stores need no branches.
  constexpr int kQ = 2;
  const int S = 64 * chunks;
  uint4 qr[kQ][KB];
  auto load_q = [&](int nq, uint4 (&qv)[KB]) {
    const int row = min(nq + li, N - 1);
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
      qv[kb] = *reinterpret_cast<const uint4*>(qbase + (size_t)row * qrs + kb * 32 + lg * 8);
  };
  // TOKGATE: a group's output gate, four channels per lane and row block in
  // the accumulators' layout, loaded after the group's products (rows past
  // the frame read as zero).
  const __amdgpu_buffer_rsrc_t grsrc =
      make_rsrc(TOKGATE ? gtok + (size_t)fh * N * DV : Q, TOKGATE ? (uint32_t)N * DV * 2u : 0u);
  const __amdgpu_buffer_rsrc_t orsrc =
      make_rsrc(obase, ((uint32_t)(N - 1) * ors + (uint32_t)dvw) * 2u);

  const int n_first = chunk * 64 + wave * 16;
  if (n_first >= N) return;
  // Issue the ring in slot order (the scheduler must not reorder it), so on
  // loop entry slot 0 is the oldest load and waits stay partial.
#pragma unroll
  for (int d = 0; d < kQ; ++d) {
    load_q(n_first + S * d, qr[d]);
    __builtin_amdgcn_sched_barrier(0);
  }
  for (int n0 = n_first; n0 < N; n0 += S * kQ) {
#pragma unroll
    for (int d = 0; d < kQ; ++d) {
      // Groups past the frame (at most kQ-1 per wave) run on clamped rows;
      // their stores fall outside the buffer range and are dropped.
      const int ng = n0 + S * d;
      floatx4 acc[MB];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) acc[mb] = floatx4{0.f, 0.f, 0.f, 0.f};
      // (An opaque zero offset keeps the compiler from hoisting the LDS
      // operand reads out of the loop into registers.)
      int zero_off = 0;
      if constexpr (!kSopRegs) asm volatile("v_mov_b32 %0, 0" : "=v"(zero_off));
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const bf16x8 qop = __builtin_bit_cast(bf16x8, qr[d][kb]);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          bf16x8 aop;
          if constexpr (kSopRegs)
            aop = sop[mb][kb];
          else
            aop = *reinterpret_cast<const bf16x8*>(sop_lds + zero_off + mb * 16 * SLD + kb * 32);
          acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aop, qop, acc[mb], 0, 0, 0);
        }
      }
      // A raw query: |q|^2 of the lane's token from the operand registers
      // (the token's DK channels are spread over lanes li + 16 lg), so that
      // the L2-normalised query's output is this one divided by
      // sqrt(|q|^2 + eps), which the RMSNorm below takes in.
      float qn2 = 1.0f;
      if constexpr (GENOUT) {
        if (ql2) {
          float s = 0.f;
#pragma unroll
          for (int kb = 0; kb < KB; ++kb) {
            const uint32_t w4[4] = {qr[d][kb].x, qr[d][kb].y, qr[d][kb].z, qr[d][kb].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              s = fmaf(bf16_lo(w4[e]), bf16_lo(w4[e]), s);
              s = fmaf(bf16_hi(w4[e]), bf16_hi(w4[e]), s);
            }
          }
          s += __shfl_xor(s, 16);
          s += __shfl_xor(s, 32);
          qn2 = s + kL2Eps;
        }
      }
      load_q(ng + S * kQ, qr[d]);
      u32x2 gnow[MB];  // this group's gate, in flight during the norm's reduction
      if constexpr (TOKGATE) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
          gnow[mb] = __builtin_bit_cast(
              u32x2, __builtin_amdgcn_raw_buffer_load_b64(
                         grsrc, (int)(((uint32_t)(ng + li) * DV + mb * 16 + 4 * lg) * 2u), 0, 0));
      }
      // lane holds o[token ng + li][mb*16 + 4*lg + i]
      float ss = 0.f;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int i = 0; i < 4; ++i) ss = fmaf(acc[mb][i], acc[mb][i], ss);
      ss += __shfl_xor(ss, 16);
      ss += __shfl_xor(ss, 32);
      // With q / n (n^2 = qn2) in place of q: g (o / n) / sqrt(mean((o / n)^2)
      // + eps) = g o / sqrt(mean(o^2) + eps n^2).
      const float scale = g / sqrtf(ss * inv_norm + kRmsEps * qn2);
      // Stores of whole token rows: the group's outputs (16 tokens x DV,
      // bf16) go through this wave's LDS tile, then each store instruction
      // writes 64 / (DV / 8) consecutive token rows, one contiguous run of
      // up to 1 KB.
      uint16_t* tile = otile + wave * (16 * OLD);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        float sc[4] = {scale, scale, scale, scale};
        if constexpr (TOKGATE) {
          sc[0] *= bf16_lo(gnow[mb][0]);
          sc[1] *= bf16_hi(gnow[mb][0]);
          sc[2] *= bf16_lo(gnow[mb][1]);
          sc[3] *= bf16_hi(gnow[mb][1]);
        }
        *reinterpret_cast<uint2*>(&tile[li * OLD + mb * 16 + 4 * lg]) =
            make_uint2(pack_bf16x2(acc[mb][0] * sc[0], acc[mb][1] * sc[1]),
                       pack_bf16x2(acc[mb][2] * sc[2], acc[mb][3] * sc[3]));
      }
      constexpr int CPR = DV / 8;     // 16-byte chunks per token row
      constexpr int RPI = 64 / CPR;   // token rows per store instruction
#pragma unroll
      for (int r0 = 0; r0 < 16; r0 += RPI) {
        const int tok = r0 + lane / CPR, ch = lane % CPR;
        const u32x4 v = *reinterpret_cast<const u32x4*>(&tile[tok * OLD + ch * 8]);
        // Channels past dvo (zero padding of a narrow head) are not stored.
        store_b128_stream(orsrc, !GENOUT || ch * 8 < dvw ? ((uint32_t)(ng + tok) * ors + ch * 8) * 2u
                                                        : kOutOfRange, v);
      }
    }
  }
}

// fp32 storage: fp32 products and sums.  16 threads per token, each owning
// d_v/16 output channels; S~ in LDS (fp32), queries staged per 16 tokens.
template <int DK, int DV, bool TOKGATE>
__global__ __launch_bounds__(kThreads)
void readout_f32_kernel(const float* __restrict__ Q, const float* __restrict__ S_fwd,
                        const float* __restrict__ S_rev, const float* __restrict__ gate,
                        int F, int N, int chunks, int tokens_per_chunk, int dvo, int oh, int qh,
                        int ql2, const float* __restrict__ alpha, int wchunk, int wradius,
                        int woffset, const float* __restrict__ gtok, float* __restrict__ out) {
  constexpr int SLD = DK + 1;
  constexpr int VPT = DV / 16;  // output channels per thread
  __shared__ float st[DV * SLD];
  __shared__ float qs[16][DK];

  const unsigned fh = blockIdx.x / chunks;
  const int chunk = blockIdx.x % chunks;
  const int n_begin = chunk * tokens_per_chunk;
  const int n_end = min(N, n_begin + tokens_per_chunk);
  const float g = TOKGATE ? 1.0f : gate[fh / F];
  const int tid = threadIdx.x;
  const float inv_norm = 1.0f / (float)dvo;
  // Query and output rows as in readout_bf16_kernel.
  const size_t qrs = (size_t)qh * DK;
  const float* qbase = Q + (((size_t)(fh / F / qh) * F + fh % F) * N * qh + (fh / F) % qh) * DK;
  const size_t ors = (size_t)oh * dvo;
  float* obase = out + (((size_t)(fh / F / oh) * F + fh % F) * N * oh + (fh / F) % oh) * dvo;

  // Gather (Eq. A.4), as in readout_bf16_kernel.
  const int h = (int)(fh / F), f = (int)(fh % F);
  const Window w = local_window(f, F, wchunk, wradius, woffset);
  const float* sf = S_fwd + ((size_t)h * F + w.lo) * (DV * DK);
  const float* sr = S_rev + ((size_t)h * F + w.hi) * (DV * DK);
  static_assert(kThreads % DK == 0, "fixed column per thread");
  float df[1], dr[1];
  bridge_decay<1>(alpha, h, F, DK, tid % DK, f, w, df, dr);
  for (int idx = tid; idx < DV * DK; idx += kThreads)
    st[(idx / DK) * SLD + idx % DK] = sf[idx] * df[0] + sr[idx] * dr[0];

  const int tok = tid >> 4;  // token within the group of 16
  const int part = tid & 15;
  for (int n0 = n_begin; n0 < n_end; n0 += 16) {
    lds_barrier();
    for (int idx = tid; idx < 16 * DK; idx += kThreads) {
      const int e = idx / DK, c = idx % DK;
      const int n = n0 + e;
      qs[e][c] = n < n_end ? qbase[(size_t)n * qrs + c] : 0.f;
    }
    lds_barrier();
    float o[VPT];
#pragma unroll
    for (int m = 0; m < VPT; ++m) o[m] = 0.f;
    for (int c = 0; c < DK; ++c) {
      const float qv = qs[tok][c];
#pragma unroll
      for (int m = 0; m < VPT; ++m) o[m] = fmaf(st[(part + 16 * m) * SLD + c], qv, o[m]);
    }
    float ss = 0.f;
#pragma unroll
    for (int m = 0; m < VPT; ++m) ss = fmaf(o[m], o[m], ss);
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) ss += __shfl_xor(ss, off);
    // A raw query, as in readout_bf16_kernel: |q|^2 over the token's row.
    float qn2 = 1.0f;
    if (ql2) {
      float s = 0.f;
      for (int c = part; c < DK; c += 16) s = fmaf(qs[tok][c], qs[tok][c], s);
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) s += __shfl_xor(s, off);
      qn2 = s + kL2Eps;
    }
    const float scale = g / sqrtf(ss * inv_norm + kRmsEps * qn2);
    const int n = n0 + tok;
    if (n < n_end) {
#pragma unroll
      for (int m = 0; m < VPT; ++m) {
        const int c = part + 16 * m;
        const size_t idx = ((size_t)fh * N + n) * DV + c;
        if (c < dvo) obase[(size_t)n * ors + c] = TOKGATE ? o[m] * scale * gtok[idx] : o[m] * scale;
      }
    }
  }
}

inline int readout_chunks(long long fh_count, int N) {
  // Enough workgroups to cover the chip a few times, each with >= 512 tokens.
  const long long target = 2048;
  long long c = (target + fh_count - 1) / fh_count;
  const long long cap = (N + 511) / 512;
  if (c > cap) c = cap;
  return c < 1 ? 1 : (int)c;
}

template <int DK, int DV>
hipError_t launch_readout_t(bool is_f32, const void* q, const float* S_fwd, const float* S_rev,
                            const float* gate, int F, int N, int H, int d_v_norm,
                            const GatherOptions& go, void* out, hipStream_t stream) {
  const long long fh_count = (long long)H * F;
  const int chunks = readout_chunks(fh_count, N);
  int tpc = (N + chunks - 1) / chunks;
  tpc = ((tpc + 63) / 64) * 64;
  const dim3 grid((unsigned)(fh_count * chunks));
  const bool genout = go.out_heads > 1 || d_v_norm != DV || go.q_heads > 1 || go.q_l2;
  const int ql2 = go.q_l2 ? 1 : 0;
#define VDA_READOUT_LAUNCH(TG, GO)                                                                 \
  if (is_f32)                                                                                      \
    hipLaunchKernelGGL((readout_f32_kernel<DK, DV, TG>), grid, dim3(kThreads), 0, stream,          \
                       static_cast<const float*>(q), S_fwd, S_rev, gate, F, N, chunks, tpc,       \
                       d_v_norm, go.out_heads, go.q_heads, ql2, go.alpha, go.chunk, go.radius,     \
                       go.offset,                                                                  \
                       static_cast<const float*>(go.gate_tokens), static_cast<float*>(out));      \
  else                                                                                             \
    hipLaunchKernelGGL((readout_bf16_kernel<DK, DV, TG, GO>), grid, dim3(kThreads), 0, stream,     \
                       static_cast<const uint16_t*>(q), S_fwd, S_rev, gate, F, N, chunks, tpc,    \
                       (unsigned)(fh_count * chunks), d_v_norm, go.out_heads, go.q_heads, ql2,     \
                       go.alpha, go.chunk,                                                         \
                       go.radius,                                                                  \
                       go.offset, static_cast<const uint16_t*>(go.gate_tokens),                    \
                       static_cast<uint16_t*>(out));
  if (go.gate_tokens != nullptr) {
    if (genout) {
      VDA_READOUT_LAUNCH(true, true)
    } else {
      VDA_READOUT_LAUNCH(true, false)
    }
  } else if (genout) {
    VDA_READOUT_LAUNCH(false, true)
  } else {
    VDA_READOUT_LAUNCH(false, false)
  }
#undef VDA_READOUT_LAUNCH
  return hipGetLastError();
}

}  // namespace

hipError_t launch_readout(bool is_f32, const void* q, const float* S_fwd, const float* S_rev,
                          const float* gate, int F, int N, int H, int d_k, int d_v, int d_v_norm,
                          const GatherOptions& go, void* out, hipStream_t stream) {
#define VDA_READOUT_CASE(DKV, DVV)                                                            \
  if (d_k == DKV && d_v == DVV)                                                               \
    return launch_readout_t<DKV, DVV>(is_f32, q, S_fwd, S_rev, gate, F, N, H, d_v_norm, go, out, \
                                      stream);
  VDA_READOUT_CASE(32, 32) VDA_READOUT_CASE(32, 64) VDA_READOUT_CASE(32, 128)
  VDA_READOUT_CASE(64, 32) VDA_READOUT_CASE(64, 64) VDA_READOUT_CASE(64, 128)
  VDA_READOUT_CASE(128, 32) VDA_READOUT_CASE(128, 64) VDA_READOUT_CASE(128, 128)
#undef VDA_READOUT_CASE
  return hipErrorInvalidValue;
}

}  // namespace vda
