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

template <int DK, bool EXACT_F32>
__global__ __launch_bounds__(kThreads)
void scan_kernel(const float* __restrict__ Inv, const float* __restrict__ Bm,
                 int F, int DV, unsigned nwg,
                 float* __restrict__ S_fwd, float* __restrict__ S_rev) {
  constexpr int XLD = DK + 4;        // LDS row stride (floats)
  constexpr int NB = DK / 16;        // 16-column output slices
  constexpr int NBW = (NB + 3) / 4;  // slices per wave
  constexpr int KL = DK / 4;         // k values per lane and slice
  constexpr int E = DK / 16;         // state elements per thread in the row-wise phase
  static_assert(E % 2 == 0, "float2 granularity");
  // Row-wise accesses in 16-byte pieces where the row slice allows: fewer
  // memory operations keep the prefetch ring within what the hardware's
  // outstanding-load counter can track precisely.
  constexpr int VW = E % 4 == 0 ? 4 : 2;
  __shared__ __align__(16) float xs[2][16 * XLD];

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

  for (int i = tid; i < 16 * XLD; i += kThreads) xs[0][i] = 0.f;

  float* Sout = dir == 0 ? S_fwd : S_rev;
  const size_t mat_b = (size_t)DV * DK;  // one B / state matrix
  const size_t row_off = (size_t)(rb * 16 + pr) * DK + pc;
  // Entering states of this head, [F][d_v][d_k]: a range-checked buffer, so
  // the padded steps past the last frame store nothing.
  const __amdgpu_buffer_rsrc_t srsrc =
      make_rsrc(Sout + (size_t)hb * F * mat_b, (uint32_t)(F * mat_b * sizeof(float)));

  auto frame_of = [&](int step) { return dir == 0 ? step : F - 1 - step; };

  // k indices held by this lane for the MFMA, in order:
  //   exact fp32 (16x16x4, k = lg*KL + s):           lg*KL .. lg*KL + KL-1
  //   split bf16 (16x16x32, k = ks*32 + 8*lg + e):   ks*32 + 8*lg .. +7, ks = 0..DK/32-1
  auto kidx = [&](int s) {
    return EXACT_F32 ? lg * KL + s : (s / 8) * 32 + 8 * lg + (s % 8);
  };

  // Operands of the next kPrefetch frames are in flight in a register ring:
  // slot d holds frame step0 + d, refilled with frame step0 + d + kPrefetch
  // once consumed.  A deeper ring no longer fits in the vector registers; the
  // compiler then parks slots in accumulation registers and must wait for
  // each load before copying it there, which drains the ring.
  constexpr int kPrefetch = 2;
  float ops[kPrefetch][NBW][KL];
  float bs[kPrefetch][E];
  auto load_ops = [&](int step, float (&op)[NBW][KL], float (&bb)[E]) {
    const size_t fh = (size_t)hb * F + frame_of(step);
    const float* inv = Inv + fh * (DK * DK);
#pragma unroll
    for (int m = 0; m < NBW; ++m) {
      const int nb = wave + 4 * m;
      if (NB >= 4 || nb < NB) {  // compile-time true unless d_k = 32
        // Inv[k][nb*16 + li] == Inv[nb*16 + li][k]
        const float* row = inv + (size_t)(nb * 16 + li) * DK;
#pragma unroll
        for (int s = 0; s < KL; s += 4) {
          const float4 v = *reinterpret_cast<const float4*>(row + kidx(s));
          op[m][s] = v.x;
          op[m][s + 1] = v.y;
          op[m][s + 2] = v.z;
          op[m][s + 3] = v.w;
        }
      }
    }
    const float* src = Bm + fh * mat_b + row_off;
#pragma unroll
    for (int e = 0; e < E; e += VW) {
      if constexpr (VW == 4) {
        const float4 x = *reinterpret_cast<const float4*>(src + e);
        bb[e] = x.x;
        bb[e + 1] = x.y;
        bb[e + 2] = x.z;
        bb[e + 3] = x.w;
      } else {
        const float2 x = *reinterpret_cast<const float2*>(src + e);
        bb[e] = x.x;
        bb[e + 1] = x.y;
      }
    }
  };

  // Issue the ring in slot order (pinned against rescheduling) so slot 0 is
  // the oldest load on loop entry.
#pragma unroll
  for (int d = 0; d < kPrefetch; ++d) {
    load_ops(min(d, F - 1), ops[d], bs[d]);
    __builtin_amdgcn_sched_barrier(0);
  }

  // The step count is padded to a multiple of the ring depth; padded steps
  // (step >= F) read a clamped frame and their stores are dropped, so the
  // loop body has no early exit.
  int cur = 0;
  for (int step0 = 0; step0 < F; step0 += kPrefetch) {
#pragma unroll
    for (int d = 0; d < kPrefetch; ++d) {
      const int step = step0 + d;
      // Frame index within the head; past the end it is out of the buffer
      // range (>= F forward, negative and so huge as unsigned in reverse).
      const int frame = dir == 0 ? step : F - 1 - step;
      lds_barrier();  // xs[cur] holds the entering state
      {
        float* x = &xs[cur][pr * XLD + pc];
        const uint32_t off = (uint32_t)((size_t)(unsigned)frame * mat_b + row_off) * 4u;
#pragma unroll
        for (int e = 0; e < E; e += VW) {
          if constexpr (VW == 4) {
            float4 v = *reinterpret_cast<float4*>(x + e);
            store_b128(srsrc, off + e * 4u,
                       u32x4{__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z),
                             __float_as_uint(v.w)});
            v.x += bs[d][e];
            v.y += bs[d][e + 1];
            v.z += bs[d][e + 2];
            v.w += bs[d][e + 3];
            *reinterpret_cast<float4*>(x + e) = v;
          } else {
            float2 v = *reinterpret_cast<float2*>(x + e);
            store_b64(srsrc, off + e * 4u, make_uint2(__float_as_uint(v.x), __float_as_uint(v.y)));
            v.x += bs[d][e];
            v.y += bs[d][e + 1];
            *reinterpret_cast<float2*>(x + e) = v;
          }
        }
      }
      lds_barrier();
      if (NB >= 4 || wave < NB) {
        // A-operand: row li of the block at this lane's k indices.
        float a[KL];
        const float* xr = &xs[cur][li * XLD];
#pragma unroll
        for (int s = 0; s < KL; s += 4) {
          const float4 v = *reinterpret_cast<const float4*>(xr + kidx(s));
          a[s] = v.x;
          a[s + 1] = v.y;
          a[s + 2] = v.z;
          a[s + 3] = v.w;
        }
        if constexpr (EXACT_F32) {
#pragma unroll
          for (int m = 0; m < NBW; ++m) {
            const int nb = wave + 4 * m;
            if (NB >= 4 || nb < NB) {
              floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
              for (int s = 0; s < KL; ++s)
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], ops[d][m][s], acc, 0, 0, 0);
#pragma unroll
              for (int i = 0; i < 4; ++i) xs[cur ^ 1][(lg * 4 + i) * XLD + nb * 16 + li] = acc[i];
            }
          }
        } else {
          constexpr int KB = DK / 32;
          bf16x8 ahi[KB], alo[KB];
#pragma unroll
          for (int kb = 0; kb < KB; ++kb) {
            float t[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) t[e] = a[kb * 8 + e];
            split_bf16x8(t, ahi[kb], alo[kb]);
          }
#pragma unroll
          for (int m = 0; m < NBW; ++m) {
            const int nb = wave + 4 * m;
            if (NB >= 4 || nb < NB) {
              floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
              for (int kb = 0; kb < KB; ++kb) {
                float t[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) t[e] = ops[d][m][kb * 8 + e];
                bf16x8 bhi, blo;
                split_bf16x8(t, bhi, blo);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo[kb], bhi, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi[kb], blo, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi[kb], bhi, acc, 0, 0, 0);
              }
#pragma unroll
              for (int i = 0; i < 4; ++i) xs[cur ^ 1][(lg * 4 + i) * XLD + nb * 16 + li] = acc[i];
            }
          }
        }
      }
      // Always refill (past the end: a clamped, unused frame) so no branch
      // hides the loads from the wait-count bookkeeping.
      load_ops(min(step + kPrefetch, F - 1), ops[d], bs[d]);
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
// this wave's 16-column slices, x being the 16 x d_k block in LDS (row
// stride XLD) and Inv_t the upper-triangle image.
template <int DK, int W>
__device__ __forceinline__ void scan_mfma_phase(const float* __restrict__ xs_cur,
                                                float* __restrict__ xs_next,
                                                const float* __restrict__ ivs, int li, int lg) {
  constexpr int XLD = DK + 4;
  constexpr int NB = DK / 16;
  constexpr int NBW = (NB + 3) / 4;
  constexpr int KB = DK / 32;
  if constexpr (W >= NB) {
    return;  // d_k = 32: two slices, waves 2 and 3 idle
  } else {
    // A-operand: row li of the block at this lane's k values.
    bf16x8 ahi[KB], alo[KB];
    const floatx4* xr = reinterpret_cast<const floatx4*>(xs_cur) + (li * XLD + 4 * lg) / 4;
#pragma unroll
    for (int ks = 0; ks < KB; ++ks) {
      float t[8];
      const floatx4 v0 = xr[8 * ks];
      const floatx4 v1 = xr[8 * ks + 4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        t[c] = v0[c];
        t[4 + c] = v1[c];
      }
      split_bf16x8(t, ahi[ks], alo[ks]);
    }
#pragma unroll
    for (int m = 0; m < NBW; ++m) {
      const int nb = W + 4 * m;
      if (nb < NB) {
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
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
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo[ks], bhi, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi[ks], blo, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi[ks], bhi, acc, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) xs_next[(lg * 4 + i) * XLD + nb * 16 + li] = acc[i];
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
template <int DK>
__global__ __launch_bounds__(kThreads)
void scan_bf16_kernel(const float* __restrict__ Inv, const float* __restrict__ Bm, int F,
                      int DV, unsigned nwg, float* __restrict__ S_fwd,
                      float* __restrict__ S_rev) {
  constexpr int XLD = DK + 4;        // LDS row stride (floats)
  constexpr int VW = DK >= 64 ? 4 : 2;  // floats per access in the row-wise phase
  constexpr int NG = DK / (16 * VW);    // accesses per thread in the row-wise phase
  using U = UpperChunks<DK>;
  constexpr int CPT = U::per_thread;
  __shared__ __align__(16) float ivs[(DK + 1) * XLD];  // Inv_t image, plus a dummy row
  __shared__ __align__(16) float xs[2][16 * XLD];

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

  for (int i = tid; i < 16 * XLD; i += kThreads) xs[0][i] = 0.f;

  float* Sout = dir == 0 ? S_fwd : S_rev;
  const size_t mat_b = (size_t)DV * DK;  // one B / state matrix
  const size_t row_off = (size_t)(rb * 16 + pr) * DK + pc;
  // Entering states of this head, [F][d_v][d_k]: a range-checked buffer, so
  // the padded steps past the last frame store nothing.
  const __amdgpu_buffer_rsrc_t srsrc =
      make_rsrc(Sout + (size_t)hb * F * mat_b, (uint32_t)(F * mat_b * sizeof(float)));

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
  auto load_step = [&](int step, u32x4 (&ir)[CPT], float (&bb)[NG][VW]) {
    const size_t fh = (size_t)hb * F + frame_of(step);
    // B rows first (they are needed earlier in the step than Inv_t), and
    // both through buffer loads, which the compiler keeps in program order.
    const __amdgpu_buffer_rsrc_t brsrc = make_rsrc(Bm + fh * mat_b, (uint32_t)(mat_b * 4));
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const uint32_t off = (uint32_t)(row_off + g * 16 * VW) * 4u;
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
    const __amdgpu_buffer_rsrc_t irsrc = make_rsrc(Inv + fh * (DK * DK), DK * DK * 4u);
#pragma unroll
    for (int e = 0; e < CPT; ++e)
      ir[e] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(irsrc, (int)goff[e], 0, 0));
  };

  int cur = 0;
  auto step_body = [&](int step, u32x4 (&ir)[CPT], float (&bb)[NG][VW]) {
    // Frame index within the head; past the end it is out of the buffer
    // range (>= F forward, negative and so huge as unsigned in reverse).
    const int frame = dir == 0 ? step : F - 1 - step;
    lds_barrier();  // xs[cur] holds the entering state; the last Inv image is consumed
#pragma unroll
    for (int e = 0; e < CPT; ++e) reinterpret_cast<u32x4*>(ivs)[loff[e]] = ir[e];
    {
      const uint32_t off = (uint32_t)((size_t)(unsigned)frame * mat_b + row_off) * 4u;
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        float* x = &xs[cur][pr * XLD + pc + g * 16 * VW];
        if constexpr (VW == 4) {
          floatx4& xv = reinterpret_cast<floatx4*>(xs[cur])[(pr * XLD + pc + g * 16 * VW) / 4];
          floatx4 v = xv;
          store_b128(srsrc, off + g * 64u * VW,
                     u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]),
                           __float_as_uint(v[3])});
#pragma unroll
          for (int c = 0; c < 4; ++c) v[c] += bb[g][c];
          xv = v;
        } else {
          float2 v = *reinterpret_cast<float2*>(x);
          store_b64(srsrc, off + g * 64u * VW, make_uint2(__float_as_uint(v.x), __float_as_uint(v.y)));
          v.x += bb[g][0];
          v.y += bb[g][1];
          *reinterpret_cast<float2*>(x) = v;
        }
      }
    }
    lds_barrier();
    // Always refill (past the end: a clamped, unused frame) so no branch
    // hides the loads from the wait-count bookkeeping.
    load_step(min(step + 2, F - 1), ir, bb);
    switch (wave) {  // wave-uniform
      case 0: scan_mfma_phase<DK, 0>(xs[cur], xs[cur ^ 1], ivs, li, lg); break;
      case 1: scan_mfma_phase<DK, 1>(xs[cur], xs[cur ^ 1], ivs, li, lg); break;
      case 2: scan_mfma_phase<DK, 2>(xs[cur], xs[cur ^ 1], ivs, li, lg); break;
      default: scan_mfma_phase<DK, 3>(xs[cur], xs[cur ^ 1], ivs, li, lg); break;
    }
    cur ^= 1;
  };

  // Issue the ring in slot order (pinned against rescheduling) so slot 0 is
  // the oldest load on loop entry.
  load_step(0, ir0, bs0);
  __builtin_amdgcn_sched_barrier(0);
  load_step(min(1, F - 1), ir1, bs1);
  __builtin_amdgcn_sched_barrier(0);
  // The step count is padded to an even number; a padded step (step >= F)
  // reads a clamped frame and its stores are dropped, so the loop body has
  // no early exit.
  for (int step0 = 0; step0 < F; step0 += 2) {
    step_body(step0, ir0, bs0);
    step_body(step0 + 1, ir1, bs1);
  }
}

template <int DK>
hipError_t launch_scan_t(bool exact_f32, const float* Inv, const float* Bm, int F, int H, int d_v,
                         float* S_fwd, float* S_rev, hipStream_t stream) {
  const unsigned nwg = (unsigned)H * 2u * (unsigned)(d_v / 16);
  if (exact_f32)
    hipLaunchKernelGGL((scan_kernel<DK, true>), dim3(nwg), dim3(kThreads), 0, stream, Inv, Bm, F,
                       d_v, nwg, S_fwd, S_rev);
  else
    hipLaunchKernelGGL((scan_bf16_kernel<DK>), dim3(nwg), dim3(kThreads), 0, stream, Inv, Bm, F,
                       d_v, nwg, S_fwd, S_rev);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_state_scan(bool exact_f32, const float* Inv, const float* Bm, int F, int H,
                             int d_k, int d_v, float* S_fwd, float* S_rev, hipStream_t stream) {
  switch (d_k) {
    case 32: return launch_scan_t<32>(exact_f32, Inv, Bm, F, H, d_v, S_fwd, S_rev, stream);
    case 64: return launch_scan_t<64>(exact_f32, Inv, Bm, F, H, d_v, S_fwd, S_rev, stream);
    case 128: return launch_scan_t<128>(exact_f32, Inv, Bm, F, H, d_v, S_fwd, S_rev, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace vda
