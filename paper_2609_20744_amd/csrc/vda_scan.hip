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
// wavefronts multiply the block by Inv_t, each producing d_k/64 16-column
// slices.  Inv_t is symmetric ((I + A_t)^{-1} of a symmetric A_t), so the
// k-th column slice a lane needs is read as a contiguous piece of row j of
// Inv_t with 16-byte loads.  Inv_t and B_t of the next two frames are in
// flight in a register ring, so memory latency stays off the serial path,
// which holds only the matrix product and two barriers.  Workgroups of one
// chain are placed on one XCD so they share Inv_t in its L2.
//
// Products: with fp32 storage (scan_kernel), v_mfma_f32_16x16x4_f32 (exact
// fp32 products).  With bf16 storage (scan_bf16_kernel, which also stages
// Inv_t through LDS, see there), each fp32 operand x is split into bf16
// hi = bf16(x) and lo = bf16(x - hi), and the product is hi*hi + hi*lo +
// lo*hi on v_mfma_f32_16x16x32_bf16 with fp32 accumulation (about 16
// mantissa bits per operand, relative error ~1e-5), several times the fp32
// matrix rate.
#include "vda_common.h"
#include "vda_launch.h"

namespace vda {
namespace {

__device__ __forceinline__ void split_bf16x8(const float (&x)[8], bf16x8& hi, bf16x8& lo) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const __bf16 h = (__bf16)x[e];
    hi[e] = h;
    lo[e] = (__bf16)(x[e] - (float)h);
  }
}

// The exact fp32 scan (fp32 storage path); DECAY and FROZEN as described at
// scan_bf16_kernel below.
template <int DK, bool FROZEN, bool DECAY>
__global__ __launch_bounds__(kThreads)
void scan_f32_kernel(const float* __restrict__ Mat, const float* __restrict__ Bm,
                     const float* __restrict__ alpha, const float* __restrict__ text_state,
                     int F, int DV, unsigned nwg, float inv_u, float inv_sqrt_u,
                     float* __restrict__ S_fwd, float* __restrict__ S_rev) {
  constexpr int XLD = DK + 4;        // LDS row stride (floats)
  constexpr int NB = DK / 16;        // 16-column output slices
  constexpr int NBW = (NB + 3) / 4;  // slices per wave
  constexpr int KL = DK / 4;         // k values per lane and slice (k = lg * KL + s)
  constexpr int E = DK / 16;         // state elements per thread in the row-wise phase
  static_assert(E % 2 == 0, "float2 granularity");
  // Row-wise accesses in 16-byte pieces where the row slice allows: fewer
  // memory operations keep the prefetch ring within what the hardware's
  // outstanding-load counter can track precisely.
  constexpr int VW = E % 4 == 0 ? 4 : 2;
  __shared__ __align__(16) float xs[2][16 * XLD];
  __shared__ __align__(16) float alds[DECAY ? DK : 4];  // alpha of the coming step

  const int nrb = DV / 16;
  const unsigned L = xcd_grouped_id(blockIdx.x, nwg);
  const int rb = L % nrb;
  const unsigned chain = L / nrb;
  const int dir = chain & 1;
  const unsigned hb = chain >> 1;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int li = lane & 15;
  const int lg = lane >> 4;

  // Row-wise phase role: row pr of the block, columns pc .. pc+E-1.
  const int pr = tid >> 4;
  const int pc = (tid & 15) * E;

  const size_t mat_b = (size_t)DV * DK;  // one B / state matrix
  for (int i = tid; i < 16 * XLD; i += kThreads) {
    const int r = i / XLD, c = i % XLD;
    xs[0][i] = text_state != nullptr && c < DK
                   ? 0.5f * text_state[(size_t)hb * mat_b + (size_t)(rb * 16 + r) * DK + c]
                   : 0.f;
  }

  float* Sout = dir == 0 ? S_fwd : S_rev;
  const size_t row_off = (size_t)(rb * 16 + pr) * DK + pc;
  const __amdgpu_buffer_rsrc_t srsrc =
      make_rsrc(Sout + (size_t)hb * F * mat_b, (uint32_t)(F * mat_b * sizeof(float)));
  const __amdgpu_buffer_rsrc_t brsrc =
      make_rsrc(Bm + (size_t)hb * F * mat_b, (uint32_t)(F * mat_b * sizeof(float)));
  const __amdgpu_buffer_rsrc_t arsrc =
      make_rsrc(DECAY ? alpha + (size_t)hb * F * DK : Bm, DECAY ? (uint32_t)(F * DK * 4) : 0u);

  auto frame_of = [&](int step) { return dir == 0 ? step : F - 1 - step; };

  // Operands of the next two frames are in flight in a register ring: slot
  // d holds frame step0 + d, refilled with frame step0 + d + 2 once
  // consumed.  A deeper ring no longer fits in the vector registers.
  constexpr int kPrefetch = 2;
  float ops[kPrefetch][NBW][KL];
  float bs[kPrefetch][E];
  u32x4 al[kPrefetch];  // alpha, columns 4 tid .. 4 tid + 3 (threads tid < DK / 4)
  auto load_ops = [&](int step, float (&op)[NBW][KL], float (&bb)[E], u32x4& av) {
    const int frame = frame_of(step);
    const int bframe = FROZEN ? frame_of(step - 1) : frame;
    const bool bin = (unsigned)bframe < (unsigned)F;
    const size_t fh = (size_t)hb * F + frame;
    const float* mat = Mat + fh * (DK * DK);
#pragma unroll
    for (int m = 0; m < NBW; ++m) {
      const int nb = wave + 4 * m;
      if (NB >= 4 || nb < NB) {  // compile-time true unless d_k = 32
        // Mat[k][nb*16 + li] == Mat[nb*16 + li][k] (symmetric)
        const float* row = mat + (size_t)(nb * 16 + li) * DK;
#pragma unroll
        for (int s = 0; s < KL; s += 4) {
          const float4 v = *reinterpret_cast<const float4*>(row + lg * KL + s);
          op[m][s] = v.x;
          op[m][s + 1] = v.y;
          op[m][s + 2] = v.z;
          op[m][s + 3] = v.w;
        }
      }
    }
#pragma unroll
    for (int e = 0; e < E; e += VW) {
      const uint32_t off =
          bin ? (uint32_t)(((size_t)bframe * mat_b + row_off + e) * 4u) : kOutOfRange;
      if constexpr (VW == 4) {
        const u32x4 x =
            __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(brsrc, (int)off, 0, 0));
#pragma unroll
        for (int v = 0; v < 4; ++v) bb[e + v] = __uint_as_float(x[v]);
      } else {
        const u32x2 x =
            __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(brsrc, (int)off, 0, 0));
        bb[e] = __uint_as_float(x[0]);
        bb[e + 1] = __uint_as_float(x[1]);
      }
    }
    if constexpr (DECAY) {
      const uint32_t off = tid < DK / 4 ? (uint32_t)(frame * DK + 4 * tid) * 4u : kOutOfRange;
      av = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(arsrc, (int)off, 0, 0));
    }
  };

#pragma unroll
  for (int d = 0; d < kPrefetch; ++d) {
    load_ops(min(d, F - 1), ops[d], bs[d], al[d]);
    __builtin_amdgcn_sched_barrier(0);
  }
  if constexpr (DECAY) {
    if (tid < DK / 4) reinterpret_cast<u32x4*>(alds)[tid] = al[0];
  }

  int cur = 0;
  for (int step0 = 0; step0 < F; step0 += kPrefetch) {
#pragma unroll
    for (int d = 0; d < kPrefetch; ++d) {
      const int step = step0 + d;
      const int frame = dir == 0 ? step : F - 1 - step;
      lds_barrier();  // xs[cur] holds the entering state
      {
        float* x = &xs[cur][pr * XLD + pc];
        const uint32_t off = (uint32_t)((size_t)(unsigned)frame * mat_b + row_off) * 4u;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          if constexpr (FROZEN) x[e] += bs[d][e] * inv_sqrt_u;  // previous frame's write
        }
#pragma unroll
        for (int e = 0; e < E; e += VW) {
          if constexpr (VW == 4) {
            const float4 v = *reinterpret_cast<float4*>(x + e);
            store_b128(srsrc, off + e * 4u,
                       u32x4{__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z),
                             __float_as_uint(v.w)});
          } else {
            const float2 v = *reinterpret_cast<float2*>(x + e);
            store_b64(srsrc, off + e * 4u, make_uint2(__float_as_uint(v.x), __float_as_uint(v.y)));
          }
        }
#pragma unroll
        for (int e = 0; e < E; ++e) {
          float v = x[e];
          if constexpr (DECAY) v *= alds[pc + e];
          if constexpr (!FROZEN) v += bs[d][e];
          x[e] = v;
        }
      }
      lds_barrier();
      if constexpr (DECAY) {  // alpha of the next step (this step's reads are done)
        if (tid < DK / 4) reinterpret_cast<u32x4*>(alds)[tid] = al[(d + 1) % kPrefetch];
      }
      if (NB >= 4 || wave < NB) {
        // A-operand: row li of the block at k = lg * KL + s.
        float a[KL];
        const float* xr = &xs[cur][li * XLD + lg * KL];
#pragma unroll
        for (int s = 0; s < KL; s += 4) {
          const float4 v = *reinterpret_cast<const float4*>(xr + s);
          a[s] = v.x;
          a[s + 1] = v.y;
          a[s + 2] = v.z;
          a[s + 3] = v.w;
        }
#pragma unroll
        for (int m = 0; m < NBW; ++m) {
          const int nb = wave + 4 * m;
          if (NB >= 4 || nb < NB) {
            floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < KL; ++s) {
              float b = ops[d][m][s];
              if constexpr (FROZEN)  // I - A / U
                b = (lg * KL + s == nb * 16 + li ? 1.0f : 0.0f) - b * inv_u;
              acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], b, acc, 0, 0, 0);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) xs[cur ^ 1][(lg * 4 + i) * XLD + nb * 16 + li] = acc[i];
          }
        }
      }
      // Always refill (past the end: a clamped, unused frame) so no branch
      // hides the loads from the wait-count bookkeeping.
      load_ops(min(step + kPrefetch, F - 1), ops[d], bs[d], al[d]);
      cur ^= 1;
    }
  }
}

// 16-byte chunks of the blocks on and above the diagonal of a DK x DK fp32
// matrix (row-major): block row i holds 16 rows of (DK - 16 i) / 4 chunks,
// starting at column 16 i.
template <int DK>
struct UpperChunks {
  static constexpr int NB = DK / 16;
  static constexpr int total = 16 * (NB * DK / 4 - 2 * NB * (NB - 1));
  static constexpr int per_thread = (total + kThreads - 1) / kThreads;
};

// Row and first column of upper-triangle chunk f (f < UpperChunks<DK>::total).
template <int DK>
__device__ __forceinline__ void upper_chunk(int f, int& row, int& col) {
  int start = 0;
  row = 0;
  col = 0;
#pragma unroll
  for (int i = 0; i < DK / 16; ++i) {
    const int cw = (DK - 16 * i) / 4;  // chunks per row in block row i
    if (f >= start && f < start + 16 * cw) {
      const int loc = f - start;
      row = 16 * i + loc / cw;
      col = 16 * i + 4 * (loc % cw);
    }
    start += 16 * cw;
  }
}

// Matrix-core phase of one scan step for wave W (a template, so that which
// operand halves are read along rows and which down columns is fixed at
// compile time and no branch separates the LDS reads): out = x Inv_t for
// this wave's 16-column slices.  x, the 16 x d_k block, comes already split
// into bf16 hi and lo planes (row stride PLD); Inv_t is the upper-triangle
// image (row stride XLD).  Even and odd k steps accumulate separately, which
// halves the chain of dependent matrix products.
template <int DK, int W>
__device__ __forceinline__ void scan_mfma_phase(const uint16_t* __restrict__ xhi,
                                                const uint16_t* __restrict__ xlo,
                                                float* __restrict__ xs_next,
                                                const float* __restrict__ ivs, int li, int lg) {
  constexpr int XLD = DK + 4;
  constexpr int PLD = DK + 8;
  constexpr int NB = DK / 16;
  constexpr int NBW = (NB + 3) / 4;
  constexpr int KB = DK / 32;
  if constexpr (W >= NB) {
    return;  // d_k = 32: two slices, waves 2 and 3 idle
  } else {
    // A-operand: row li of the block at k = 32 ks + 4 lg + e, 32 ks + 16 + 4 lg + e.
    bf16x8 ahi[KB], alo[KB];
#pragma unroll
    for (int ks = 0; ks < KB; ++ks) {
      const int o = li * PLD + 32 * ks + 4 * lg;
      const u32x2 h0 = *reinterpret_cast<const u32x2*>(&xhi[o]);
      const u32x2 h1 = *reinterpret_cast<const u32x2*>(&xhi[o + 16]);
      const u32x2 l0 = *reinterpret_cast<const u32x2*>(&xlo[o]);
      const u32x2 l1 = *reinterpret_cast<const u32x2*>(&xlo[o + 16]);
      ahi[ks] = __builtin_bit_cast(bf16x8, u32x4{h0[0], h0[1], h1[0], h1[1]});
      alo[ks] = __builtin_bit_cast(bf16x8, u32x4{l0[0], l0[1], l1[0], l1[1]});
    }
#pragma unroll
    for (int m = 0; m < NBW; ++m) {
      const int nb = W + 4 * m;
      if (nb < NB) {
        floatx4 acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
        for (int ks = 0; ks < KB; ++ks) {
          // B-operand: Inv[k][16 nb + li] at this lane's k values, in two
          // halves of four, each inside k block kb = 2 ks + h.
          float t[8];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int k0 = 32 * ks + 16 * h + 4 * lg;
            if (2 * ks + h > nb) {  // row 16 nb + li of the stored block (nb, kb)
              const floatx4 v = reinterpret_cast<const floatx4*>(ivs)[((nb * 16 + li) * XLD + k0) / 4];
#pragma unroll
              for (int c = 0; c < 4; ++c) t[4 * h + c] = v[c];
            } else {  // column 16 nb + li of the stored block (kb, nb)
              const float* q = &ivs[k0 * XLD + nb * 16 + li];
#pragma unroll
              for (int c = 0; c < 4; ++c) t[4 * h + c] = q[c * XLD];
            }
          }
          bf16x8 bhi, blo;
          split_bf16x8(t, bhi, blo);
          floatx4& a = acc[ks & 1];
          a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo[ks], bhi, a, 0, 0, 0);
          a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi[ks], blo, a, 0, 0, 0);
          a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi[ks], bhi, a, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
          xs_next[(lg * 4 + i) * XLD + nb * 16 + li] = acc[0][i] + acc[1][i];
      }
    }
  }
}

// The split-bf16 scan (bf16 storage path).  The recurrence, the work split
// (one 16-row block of one chain per workgroup) and the products are those
// of scan_kernel; the difference is how Inv_t reaches the matrix cores.
// Per frame the workgroup copies only the blocks of Inv_t on and above the
// diagonal (36 of 64 at d_k = 128; the others are their transposes, as
// Inv_t is symmetric) with consecutive lanes on consecutive 16-byte chunks
// into an LDS image, and each wave reads its operands from there.  Scattered
// per-lane reads of whole rows of Inv_t from memory are limited by the
// address units, not by bandwidth; the coalesced half-size copy is what
// makes this scan faster.  Inv_t and B_t of the next two frames are in
// flight in a register ring.
//
// Matrix-core k order: in each 32-wide k step, lane group g holds
// k = 4g + e and 16 + 4g + e (e < 4), in both operands.  So each 4-value
// half of an operand lies in one 16 x 16 block of Inv_t: block (kb, nb) with
// kb = 2 ks or 2 ks + 1 for output column block nb, the same for every lane.
// When kb > nb the half is read along row 16 nb + li of the stored block
// (nb, kb) (one 16-byte read), otherwise down column 16 nb + li of the stored
// block (kb, nb) (four 4-byte reads).  With a row stride of 132 floats the
// two lane groups of each 32-lane LDS pass then fall on distinct banks in
// both kinds of read.
//
// Options of the full operator (template switches, so the core path carries
// none of their work):
//   DECAY  - the entering state is decayed, Sbar = S Diag(alpha_t), before
//            the frame's write (Eq. 5 / A.1 with alpha); alpha_t reaches the
//            row-wise phase through a small LDS row written one step ahead.
//   FROZEN - the frozen-state additive rule with 1/sqrt(U) key scaling,
//            S_t = Sbar_t (I - A_t / U) + B_t / sqrt(U) (Eq. 3c): the staged
//            matrix is I - A_t / U, built from A_t on the way into LDS, and
//            the write B_t / sqrt(U) is added after the product, that is at
//            the start of the next step (B is loaded one frame late), so the
//            state kept between steps is S_t - B_t / sqrt(U).  (Not launched:
//            with bf16 storage the frozen rule runs on the tiled scan.)
// Both scans may start from a text state: S_T / 2 (Eq. 1b).
template <int DK, bool FROZEN, bool DECAY>
__global__ __launch_bounds__(kThreads)
void scan_bf16_kernel(const float* __restrict__ Mat, const float* __restrict__ Bm,
                      const float* __restrict__ alpha, const float* __restrict__ text_state,
                      int F, int DV, unsigned nwg, float inv_u, float inv_sqrt_u,
                      float* __restrict__ S_fwd, float* __restrict__ S_rev) {
  constexpr int XLD = DK + 4;        // LDS row stride (floats)
  constexpr int VW = DK >= 64 ? 4 : 2;  // floats per access in the row-wise phase
  constexpr int NG = DK / (16 * VW);    // accesses per thread in the row-wise phase
  using U = UpperChunks<DK>;
  constexpr int CPT = U::per_thread;
  constexpr int PLD = DK + 8;        // bf16 row stride of the split planes
  __shared__ __align__(16) float ivs[(DK + 1) * XLD];  // matrix image, plus a dummy row
  __shared__ __align__(16) float xs[2][16 * XLD];
  __shared__ __align__(16) uint16_t xsp[2][16 * PLD];   // bf16 hi / lo planes of the block
  __shared__ __align__(16) float alds[DECAY ? DK : 4];  // alpha of the coming step

  const int nrb = DV / 16;
  const unsigned L = xcd_grouped_id(blockIdx.x, nwg);
  const int rb = L % nrb;
  const unsigned chain = L / nrb;
  const int dir = chain & 1;
  const unsigned hb = chain >> 1;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int li = lane & 15;
  const int lg = lane >> 4;

  // Row-wise phase role: row pr of the block; access g covers columns
  // pc + g * 16 * VW .. + VW - 1 (16 consecutive lanes on one contiguous run).
  const int pr = tid >> 4;
  const int pc = (tid & 15) * VW;

  const size_t mat_b = (size_t)DV * DK;  // one B / state matrix
  // Initial state: S_T / 2 (rows of this block), or zero.
  for (int i = tid; i < 16 * XLD; i += kThreads) {
    const int r = i / XLD, c = i % XLD;
    xs[0][i] = text_state != nullptr && c < DK
                   ? 0.5f * text_state[(size_t)hb * mat_b + (size_t)(rb * 16 + r) * DK + c]
                   : 0.f;
  }

  float* Sout = dir == 0 ? S_fwd : S_rev;
  const size_t row_off = (size_t)(rb * 16 + pr) * DK + pc;
  // Entering states of this head, [F][d_v][d_k]: a range-checked buffer, so
  // the padded steps past the last frame store nothing.
  const __amdgpu_buffer_rsrc_t srsrc =
      make_rsrc(Sout + (size_t)hb * F * mat_b, (uint32_t)(F * mat_b * sizeof(float)));
  // B of this head, range-checked (frames outside [0, F) read as zero).
  const __amdgpu_buffer_rsrc_t brsrc =
      make_rsrc(Bm + (size_t)hb * F * mat_b, (uint32_t)(F * mat_b * sizeof(float)));
  const __amdgpu_buffer_rsrc_t arsrc =
      make_rsrc(DECAY ? alpha + (size_t)hb * F * DK : Bm, DECAY ? (uint32_t)(F * DK * 4) : 0u);

  auto frame_of = [&](int step) { return dir == 0 ? step : F - 1 - step; };

  // This thread's upper-triangle chunks: byte offsets within a matrix and
  // LDS positions in 16-byte units (chunks past the end: out of range, and
  // the dummy row).
  uint32_t goff[CPT];
  int loff[CPT];
#pragma unroll
  for (int e = 0; e < CPT; ++e) {
    const int f = e * kThreads + tid;
    int row, col;
    upper_chunk<DK>(f, row, col);
    const bool in = f < U::total;
    goff[e] = in ? (uint32_t)(row * DK + col) * 4u : kOutOfRange;
    loff[e] = (in ? row * XLD + col : DK * XLD) / 4;
  }

  // Two-frame register ring, as separately named arrays (compile-time
  // indices only).
  u32x4 ir0[CPT], ir1[CPT];
  float bs0[NG][VW], bs1[NG][VW];
  u32x4 al0, al1;  // alpha_t, columns 4 tid .. 4 tid + 3 (threads tid < DK / 4)
  auto load_step = [&](int step, u32x4 (&ir)[CPT], float (&bb)[NG][VW], u32x4& al) {
    const int frame = frame_of(step);
    // The write added in this step: B of this frame (joint rule) or of the
    // previous one (frozen rule; none before the first frame).
    const int bframe = FROZEN ? frame_of(step - 1) : frame;
    const bool bin = (unsigned)bframe < (unsigned)F;
    // B rows first (they are needed earlier in the step than the matrix),
    // and everything through buffer loads, which the compiler keeps in
    // program order.
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const uint32_t off =
          bin ? (uint32_t)(((size_t)bframe * mat_b + row_off + g * 16 * VW) * 4u) : kOutOfRange;
      if constexpr (VW == 4) {
        const u32x4 x =
            __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(brsrc, (int)off, 0, 0));
#pragma unroll
        for (int v = 0; v < 4; ++v) bb[g][v] = __uint_as_float(x[v]);
      } else {
        const u32x2 x =
            __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(brsrc, (int)off, 0, 0));
        bb[g][0] = __uint_as_float(x[0]);
        bb[g][1] = __uint_as_float(x[1]);
      }
    }
    if constexpr (DECAY) {
      const uint32_t off = tid < DK / 4 ? (uint32_t)(frame * DK + 4 * tid) * 4u : kOutOfRange;
      al = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(arsrc, (int)off, 0, 0));
    }
    const size_t fh = (size_t)hb * F + frame;
    const __amdgpu_buffer_rsrc_t irsrc = make_rsrc(Mat + fh * (DK * DK), DK * DK * 4u);
#pragma unroll
    for (int e = 0; e < CPT; ++e)
      ir[e] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(irsrc, (int)goff[e], 0, 0));
  };

  // The staged matrix: Inv_t as loaded (joint rule), or I - A_t / U from the
  // loaded A_t (frozen rule).
  auto stage = [&](const u32x4 (&ir)[CPT]) {
#pragma unroll
    for (int e = 0; e < CPT; ++e) {
      u32x4 w = ir[e];
      if constexpr (FROZEN) {
        const int elem = (int)(goff[e] / 4u);
        const int row = elem / DK, col = elem % DK;
#pragma unroll
        for (int c = 0; c < 4; ++c)
          w[c] = __float_as_uint((row == col + c ? 1.0f : 0.0f) - __uint_as_float(w[c]) * inv_u);
      }
      reinterpret_cast<u32x4*>(ivs)[loff[e]] = w;
    }
  };

  int cur = 0;
  auto step_body = [&](int step, u32x4 (&ir)[CPT], float (&bb)[NG][VW], u32x4& al,
                       const u32x4& al_next) {
    // Frame index within the head; past the end it is out of the buffer
    // range (>= F forward, negative and so huge as unsigned in reverse).
    const int frame = dir == 0 ? step : F - 1 - step;
    lds_barrier();  // xs[cur] holds the entering state; the last matrix image is consumed
    stage(ir);
    {
      const uint32_t off = (uint32_t)((size_t)(unsigned)frame * mat_b + row_off) * 4u;
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        float* x = &xs[cur][pr * XLD + pc + g * 16 * VW];
        float v[VW];
        if constexpr (VW == 4) {
          const floatx4 xv = reinterpret_cast<const floatx4*>(xs[cur])[(pr * XLD + pc + g * 16 * VW) / 4];
#pragma unroll
          for (int c = 0; c < 4; ++c) v[c] = xv[c];
        } else {
          const float2 xv = *reinterpret_cast<const float2*>(x);
          v[0] = xv.x;
          v[1] = xv.y;
        }
        if constexpr (FROZEN) {  // the previous frame's write, B / sqrt(U)
#pragma unroll
          for (int c = 0; c < VW; ++c) v[c] += bb[g][c] * inv_sqrt_u;
        }
        if constexpr (VW == 4)
          store_b128(srsrc, off + g * 64u * VW,
                     u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]),
                           __float_as_uint(v[3])});
        else
          store_b64(srsrc, off + g * 64u * VW, make_uint2(__float_as_uint(v[0]), __float_as_uint(v[1])));
        if constexpr (DECAY) {
#pragma unroll
          for (int c = 0; c < VW; ++c) v[c] *= alds[pc + g * 16 * VW + c];
        }
        if constexpr (!FROZEN) {
#pragma unroll
          for (int c = 0; c < VW; ++c) v[c] += bb[g][c];
        }
        // The product's A-operand, split once here into bf16 hi and lo
        // (instead of by each of the four waves).
        uint32_t hw[VW / 2], lw[VW / 2];
#pragma unroll
        for (int c = 0; c < VW; c += 2) {
          const uint32_t h = pack_bf16x2(v[c], v[c + 1]);
          hw[c / 2] = h;
          lw[c / 2] = pack_bf16x2(v[c] - bf16_lo(h), v[c + 1] - bf16_hi(h));
        }
        const int po = pr * PLD + pc + g * 16 * VW;
        if constexpr (VW == 4) {
          *reinterpret_cast<u32x2*>(&xsp[0][po]) = u32x2{hw[0], hw[1]};
          *reinterpret_cast<u32x2*>(&xsp[1][po]) = u32x2{lw[0], lw[1]};
        } else {
          *reinterpret_cast<uint32_t*>(&xsp[0][po]) = hw[0];
          *reinterpret_cast<uint32_t*>(&xsp[1][po]) = lw[0];
        }
        (void)x;
      }
    }
    lds_barrier();
    // alpha of the next step, read by its row-wise phase (after the next
    // barrier); this step's reads of alds are complete.
    if constexpr (DECAY) {
      if (tid < DK / 4) reinterpret_cast<u32x4*>(alds)[tid] = al_next;
    }
    // Always refill (past the end: a clamped, unused frame) so no branch
    // hides the loads from the wait-count bookkeeping.
    load_step(min(step + 2, F - 1), ir, bb, al);
    switch (wave) {  // wave-uniform
      case 0: scan_mfma_phase<DK, 0>(xsp[0], xsp[1], xs[cur ^ 1], ivs, li, lg); break;
      case 1: scan_mfma_phase<DK, 1>(xsp[0], xsp[1], xs[cur ^ 1], ivs, li, lg); break;
      case 2: scan_mfma_phase<DK, 2>(xsp[0], xsp[1], xs[cur ^ 1], ivs, li, lg); break;
      default: scan_mfma_phase<DK, 3>(xsp[0], xsp[1], xs[cur ^ 1], ivs, li, lg); break;
    }
    cur ^= 1;
  };

  // Issue the ring in slot order (pinned against rescheduling) so slot 0 is
  // the oldest load on loop entry.
  load_step(0, ir0, bs0, al0);
  __builtin_amdgcn_sched_barrier(0);
  load_step(min(1, F - 1), ir1, bs1, al1);
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (DECAY) {  // alpha of step 0
    if (tid < DK / 4) reinterpret_cast<u32x4*>(alds)[tid] = al0;
  }
  // The step count is padded to an even number; a padded step (step >= F)
  // reads a clamped frame and its stores are dropped, so the loop body has
  // no early exit.
  for (int step0 = 0; step0 < F; step0 += 2) {
    step_body(step0, ir0, bs0, al0, al1);
    step_body(step0 + 1, ir1, bs1, al1, al0);
  }
}

template <int DK, bool FROZEN, bool DECAY>
hipError_t launch_scan_v(bool exact_f32, const float* Mat, const float* Bm, int F, int H, int d_v,
                         const ScanOptions& o, float* S_fwd, float* S_rev, hipStream_t stream) {
  const unsigned nwg = (unsigned)H * 2u * (unsigned)(d_v / 16);
  const float inv_u = FROZEN ? 1.0f / (float)o.tokens : 0.0f;
  const float inv_sqrt_u = FROZEN ? 1.0f / sqrtf((float)o.tokens) : 0.0f;
  if (exact_f32) {
    hipLaunchKernelGGL((scan_f32_kernel<DK, FROZEN, DECAY>), dim3(nwg), dim3(kThreads), 0, stream,
                       Mat, Bm, o.alpha, o.text_state, F, d_v, nwg, inv_u, inv_sqrt_u, S_fwd, S_rev);
  } else {
    // With bf16 storage the frozen rule runs on the tiled scan (map form).
    if constexpr (FROZEN) return hipErrorInvalidValue;
    else
      hipLaunchKernelGGL((scan_bf16_kernel<DK, false, DECAY>), dim3(nwg), dim3(kThreads), 0, stream,
                         Mat, Bm, o.alpha, o.text_state, F, d_v, nwg, inv_u, inv_sqrt_u, S_fwd, S_rev);
  }
  return hipGetLastError();
}

template <int DK>
hipError_t launch_scan_t(bool exact_f32, const float* Mat, const float* Bm, int F, int H, int d_v,
                         const ScanOptions& o, float* S_fwd, float* S_rev, hipStream_t stream) {
  const bool decay = o.alpha != nullptr;
  if (o.frozen)
    return decay ? launch_scan_v<DK, true, true>(exact_f32, Mat, Bm, F, H, d_v, o, S_fwd, S_rev, stream)
                 : launch_scan_v<DK, true, false>(exact_f32, Mat, Bm, F, H, d_v, o, S_fwd, S_rev, stream);
  return decay ? launch_scan_v<DK, false, true>(exact_f32, Mat, Bm, F, H, d_v, o, S_fwd, S_rev, stream)
               : launch_scan_v<DK, false, false>(exact_f32, Mat, Bm, F, H, d_v, o, S_fwd, S_rev, stream);
}

}  // namespace

hipError_t launch_state_scan(bool exact_f32, const float* Mat, const float* Bm, int F, int H,
                             int d_k, int d_v, const ScanOptions& o, float* S_fwd, float* S_rev,
                             hipStream_t stream) {
  switch (d_k) {
    case 32: return launch_scan_t<32>(exact_f32, Mat, Bm, F, H, d_v, o, S_fwd, S_rev, stream);
    case 64: return launch_scan_t<64>(exact_f32, Mat, Bm, F, H, d_v, o, S_fwd, S_rev, stream);
    case 128: return launch_scan_t<128>(exact_f32, Mat, Bm, F, H, d_v, o, S_fwd, S_rev, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace vda
