// Steps a3/a4 on the bf16 storage path for the joint rule: the forward and
// reverse state scans of Eq. A.1 (Algorithm 1 step 5),
//     P_t = (P_{t-1} Diag(alpha_t) + B_t) Inv_t,
//     R_t = (R_{t+1} Diag(alpha_t) + B_t) Inv_t,
// from S_T / 2 (Eq. 1b) or zero, with alpha = 1 unless a decay is given.
// The entering state of every frame (P_{t-1} forward, R_{t+1} reverse) is
// stored for the readout.
//
// Work split as in the other scans: one workgroup per (head, direction,
// 16-row block of the state); the rows of the state evolve independently,
// and the block stays in LDS across all F frames.  The difference is how
// Inv_t reaches the matrix cores: the inverse step wrote it as split-bf16
// operand tiles (operand_tile_offset), in exactly the lane order of the
// B-operands of v_mfma_f32_16x16x32_bf16.  Each wave loads the tiles of its
// own 16-column output slices straight into registers, one contiguous 1 KB
// piece per load instruction, two steps ahead of use, through a three-slot
// register ring whose refills are issued between the products.  No LDS
// image of Inv_t, no per-step split of it and no barrier for it remain on
// the serial path, which is the row-wise update (entering state out, decay,
// B_t in, split into bf16 hi / lo), one barrier, the matrix products and
// another barrier.
//
// Products: the state operand x is split into hi = bf16(x) and
// lo = bf16(x - hi) once per step, and hi*hi + hi*lo + lo*hi runs on the
// bf16 matrix cores with fp32 accumulation (about 16 mantissa bits per
// operand; relative error ~1e-5 per step, which the non-expansive frame maps
// of Prop. 1 keep from growing along the scan).
#include "vda_common.h"
#include "vda_inverse_body.h"
#include "vda_launch.h"

namespace vda {
namespace {

template <int DK>
struct TiledDims {
  static constexpr int NB = DK / 16;           // 16-column output slices
  static constexpr int NBW = (NB + 3) / 4;     // slices per wave
  static constexpr int KB = DK / 32;           // 32-wide k steps
  static constexpr int XLD = DK + 4;           // fp32 state row stride (floats)
  static constexpr int PLD = DK + 8;           // bf16 plane row stride (elements)
  static constexpr int VW = DK >= 64 ? 4 : 2;  // floats per access in the row-wise phase
  static constexpr int NG = DK / (16 * VW);    // accesses per thread in the row-wise phase
};

// One of this wave's tile loads: piece i of its NBW * KB * 2 pieces
// (slice m = i / (2 KB), k step (i / 2) % KB, plane i % 2) of the tiles at
// byte offset fbase of the tile buffer, into register slot t.
template <int DK>
__device__ __forceinline__ void load_tile_piece(
    int i, u32x4 (&t)[TiledDims<DK>::NBW][TiledDims<DK>::KB][2],
    const uint32_t (&toff)[TiledDims<DK>::NBW][TiledDims<DK>::KB][2],
    __amdgpu_buffer_rsrc_t trsrc, uint32_t fbase) {
  constexpr int KB = TiledDims<DK>::KB;
  const int m = i / (2 * KB), ks = (i / 2) % KB, p = i % 2;
  const uint32_t o = toff[m][ks][p];
  t[m][ks][p] = __builtin_bit_cast(
      u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                 trsrc, (int)(o == kOutOfRange ? kOutOfRange : fbase + o), 0, 0));
}

// Matrix-core phase of one step for wave w: xs_next = x Inv_t for this
// wave's output slices nb = w, w + 4, ..., with x from the bf16 hi / lo
// planes and Inv_t from the register tiles t[m][ks][plane].  Even and odd k
// steps accumulate separately (two shorter dependency chains).  After each
// k step's three products the wave issues two of the loads that fill
// another ring slot (tn) with the tiles of a later step (byte offset
// `next`), so the loads stream out between the products rather than in one
// burst that would stall the wave at issue.  (Issuing the products of all
// pairs term by term, with a separate accumulator per pair, measured slower:
// the phase is bound by the loads' issue, not by the products' latency.)
// The wave index is a run-time (scalar) value: one code path for all waves,
// so the compiler's wait-count bookkeeping sees no merging branches and
// keeps its waits partial.
template <int DK>
__device__ __forceinline__ void tiled_mfma_phase(
    const uint16_t* __restrict__ xhi, const uint16_t* __restrict__ xlo,
    float* __restrict__ xs_next, const u32x4 (&t)[TiledDims<DK>::NBW][TiledDims<DK>::KB][2],
    u32x4 (&tn)[TiledDims<DK>::NBW][TiledDims<DK>::KB][2],
    const uint32_t (&toff)[TiledDims<DK>::NBW][TiledDims<DK>::KB][2],
    __amdgpu_buffer_rsrc_t trsrc, uint32_t next, int wave, int li, int lg) {
  using D = TiledDims<DK>;
  constexpr int NBW = D::NBW, KB = D::KB;
  static_assert(D::NB % 4 == 0 || D::NB < 4, "slices are dealt out to four waves");
  if (D::NB < 4 && wave >= D::NB) return;  // d_k = 32: two slices, waves 2 and 3 idle
  // A-operand: row li of the block at k = 32 ks + 4 lg + e, 32 ks + 16 + 4 lg + e.
  bf16x8 ahi[KB], alo[KB];
#pragma unroll
  for (int ks = 0; ks < KB; ++ks) {
    const int o = li * D::PLD + 32 * ks + 4 * lg;
    const u32x2 h0 = *reinterpret_cast<const u32x2*>(&xhi[o]);
    const u32x2 h1 = *reinterpret_cast<const u32x2*>(&xhi[o + 16]);
    const u32x2 l0 = *reinterpret_cast<const u32x2*>(&xlo[o]);
    const u32x2 l1 = *reinterpret_cast<const u32x2*>(&xlo[o + 16]);
    ahi[ks] = __builtin_bit_cast(bf16x8, u32x4{h0[0], h0[1], h1[0], h1[1]});
    alo[ks] = __builtin_bit_cast(bf16x8, u32x4{l0[0], l0[1], l1[0], l1[1]});
  }
#pragma unroll
  for (int m = 0; m < NBW; ++m) {
    const int nb = wave + 4 * m;
    floatx4 acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int ks = 0; ks < KB; ++ks) {
      const bf16x8 bhi = __builtin_bit_cast(bf16x8, t[m][ks][0]);
      const bf16x8 blo = __builtin_bit_cast(bf16x8, t[m][ks][1]);
      floatx4& a = acc[ks & 1];
      a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo[ks], bhi, a, 0, 0, 0);
      a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi[ks], blo, a, 0, 0, 0);
      a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi[ks], bhi, a, 0, 0, 0);
      const int piece = 2 * (m * KB + ks);  // this wave's pieces in (slice, k step, plane) order
      load_tile_piece<DK>(piece, tn, toff, trsrc, next);
      load_tile_piece<DK>(piece + 1, tn, toff, trsrc, next);
      __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);  // the three products
      __builtin_amdgcn_sched_group_barrier(0x020, 2, 0);  // then two loads of the refill
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
      xs_next[(lg * 4 + i) * D::XLD + nb * 16 + li] = acc[0][i] + acc[1][i];
  }
}

// Arguments of the tiled scan.  Frame scans: tiles = Inv_t tiles [H][F],
// add = B [H][F][d_v][d_k].  Map scans (CHUNKED), x <- x M + add_scale J:
// chunk scans take tiles = M_c tiles [H][2][C] and add = J_c
// [H][2][C][d_v][d_k] over the C chunks of the window grid (chunk, offset),
// one set per direction (mats_per_head = 2C, dir_stride = C); the frozen
// rule takes per-frame maps M_t = Diag(alpha_t)(I - A_t / U) and J_t = B_t
// scaled by 1 / sqrt(U), shared by both directions (chunks of one frame,
// mats_per_head = F, dir_stride = 0).
struct TiledScanArgs {
  const uint16_t* tiles;
  const float* add;
  const float* alpha;
  const float* text_state;
  int F, DV;
  unsigned nwg;
  int chunk, offset, C;
  int mats_per_head, dir_stride;
  float add_scale;
  float* S_fwd;
  float* S_rev;
};

// CHUNKED: the same recurrence over the chunk sequence,
//     x <- x M_c + J_c,
// storing the state entering chunk c at its first frame (forward) or its
// last frame (reverse).  The additive term comes after the product here, so
// step j adds J of the previous chunk (loaded one step late) to the product
// before it stores and splits the state; the last step's product is unused.
// At most 256 registers per lane (two waves per SIMD), so two workgroups
// share a compute unit when there are more chains' row blocks than compute
// units (e.g. 24 heads: 384 workgroups) instead of running in two rounds.
template <int DK, bool DECAY, bool CHUNKED>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2)))
void scan_tiled_kernel(TiledScanArgs a) {
  static_assert(!(CHUNKED && DECAY), "chunk maps already hold the decay");
  const int F = a.F, DV = a.DV, C = a.C;
  const float* __restrict__ alpha = a.alpha;
  const float* __restrict__ text_state = a.text_state;
  const unsigned nwg = a.nwg;
  using D = TiledDims<DK>;
  constexpr int XLD = D::XLD, PLD = D::PLD, VW = D::VW, NG = D::NG;
  constexpr int NBW = D::NBW, KB = D::KB;
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

  float* Sout = dir == 0 ? a.S_fwd : a.S_rev;
  const size_t row_off = (size_t)(rb * 16 + pr) * DK + pc;
  // Entering states of this head, [F][d_v][d_k]: a range-checked buffer.
  const __amdgpu_buffer_rsrc_t srsrc =
      make_rsrc(Sout + (size_t)hb * F * mat_b, (uint32_t)(F * mat_b * sizeof(float)));
  // Steps: frames, or chunks; matrices (tiles) and additive terms of this
  // chain, range-checked (indices outside read as zero).
  const int nsteps = CHUNKED ? C : F;
  const size_t chain_mats =
      CHUNKED ? (size_t)hb * a.mats_per_head + (size_t)dir * a.dir_stride : (size_t)hb * F;
  const __amdgpu_buffer_rsrc_t brsrc =
      make_rsrc(a.add + chain_mats * mat_b, (uint32_t)(nsteps * mat_b * sizeof(float)));
  const __amdgpu_buffer_rsrc_t arsrc =
      make_rsrc(DECAY ? alpha + (size_t)hb * F * DK : a.add, DECAY ? (uint32_t)(F * DK * 4) : 0u);
  const __amdgpu_buffer_rsrc_t trsrc = make_rsrc(a.tiles + chain_mats * (DK * DK * 2),
                                                 (uint32_t)nsteps * (uint32_t)(DK * DK * 4));

  // This wave's tile offsets within a frame (out of range for the slices of
  // idle waves at d_k = 32).
  uint32_t toff[NBW][KB][2];
#pragma unroll
  for (int m = 0; m < NBW; ++m) {
    const int nb = wave + 4 * m;
#pragma unroll
    for (int ks = 0; ks < KB; ++ks)
#pragma unroll
      for (int p = 0; p < 2; ++p)
        toff[m][ks][p] = nb < D::NB ? operand_tile_offset(DK, p, nb, ks, lane) : kOutOfRange;
  }

  // Matrix of step `step` (frame or chunk in scan order), the index of its
  // additive term (chunks: the previous chunk's J, none before the first),
  // and the frame whose entering state the step stores (-1: none).
  auto frame_of = [&](int step) { return dir == 0 ? step : nsteps - 1 - step; };
  auto add_of = [&](int step) {
    if constexpr (CHUNKED) return step >= 1 ? frame_of(step - 1) : -1;
    return frame_of(step);
  };
  auto store_frame = [&](int step) {
    if (step >= nsteps) return -1;
    if constexpr (CHUNKED) {
      const int c = frame_of(step);
      return dir == 0 ? max(0, c * a.chunk - a.offset) : min(F - 1, (c + 1) * a.chunk - a.offset - 1);
    }
    return frame_of(step);
  };

  // Three-slot register ring, as separately named arrays (compile-time
  // indices only): step s reads slot s % 3 while the loads of step s + 2
  // fill slot (s + 2) % 3, which step s - 1 has released.
  u32x4 t0[NBW][KB][2], t1[NBW][KB][2], t2[NBW][KB][2];
  float bs0[NG][VW], bs1[NG][VW], bs2[NG][VW];
  u32x4 al0, al1, al2;  // alpha_t, columns 4 tid .. 4 tid + 3 (threads tid < DK / 4)
  auto load_add = [&](int step, float (&bb)[NG][VW], u32x4& al) {
    const int frame = frame_of(step);
    const int ai = add_of(step);
    // B rows first (they are needed earlier in the step than the tiles),
    // and everything through buffer loads, which the compiler keeps in
    // program order.
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const uint32_t off =
          ai >= 0 ? (uint32_t)(((size_t)ai * mat_b + row_off + g * 16 * VW) * 4u) : kOutOfRange;
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
  };
  auto tile_base = [&](int step) { return (uint32_t)frame_of(step) * (uint32_t)(DK * DK * 4); };
  auto load_tiles = [&](int step, u32x4 (&t)[NBW][KB][2]) {
    const uint32_t fbase = tile_base(step);
#pragma unroll
    for (int m = 0; m < NBW; ++m)
#pragma unroll
      for (int ks = 0; ks < KB; ++ks)
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          const uint32_t o = toff[m][ks][p];
          t[m][ks][p] = __builtin_bit_cast(
              u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                         trsrc, (int)(o == kOutOfRange ? kOutOfRange : fbase + o), 0, 0));
        }
  };

  int cur = 0;
  // Step `step` on slot (t, bb); (tn, bn, aln) is the slot the step fills
  // with step + 2 (B and alpha at its start, the tiles between its
  // products; past the end: a clamped, unused step), always, so no
  // branch hides the loads from the wait-count bookkeeping; al_next is the
  // alpha of step + 1, loaded a step ago.
  auto step_body = [&](int step, const u32x4 (&t)[NBW][KB][2], const float (&bb)[NG][VW],
                       const u32x4& al_next, u32x4 (&tn)[NBW][KB][2], float (&bn)[NG][VW],
                       u32x4& aln) {
    // Frame whose entering state this step stores (-1 for a padded step
    // past the end: the stores go out of the buffer's range).
    const int sf = store_frame(step);
    lds_barrier();  // xs[cur] holds the entering state; last step's plane reads are done
    const int refill = min(step + 2, nsteps - 1);
    const uint32_t next = tile_base(refill);
    load_add(refill, bn, aln);
    {
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        const uint32_t off =
            sf >= 0 ? (uint32_t)(((size_t)sf * mat_b + row_off + g * 16 * VW) * 4u) : kOutOfRange;
        const int xo = pr * XLD + pc + g * 16 * VW;
        float v[VW];
        if constexpr (VW == 4) {
          const floatx4 xv = reinterpret_cast<const floatx4*>(xs[cur])[xo / 4];
#pragma unroll
          for (int c = 0; c < 4; ++c) v[c] = xv[c];
        } else {
          const float2 xv = *reinterpret_cast<const float2*>(&xs[cur][xo]);
          v[0] = xv.x;
          v[1] = xv.y;
        }
        if constexpr (CHUNKED) {  // J of the previous chunk, after its product
#pragma unroll
          for (int c = 0; c < VW; ++c) v[c] = fmaf(bb[g][c], a.add_scale, v[c]);
        }
        if constexpr (VW == 4)
          store_b128(srsrc, off,
                     u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]),
                           __float_as_uint(v[3])});
        else
          store_b64(srsrc, off, make_uint2(__float_as_uint(v[0]), __float_as_uint(v[1])));
        if constexpr (DECAY) {
#pragma unroll
          for (int c = 0; c < VW; ++c) v[c] *= alds[pc + g * 16 * VW + c];
        }
        if constexpr (!CHUNKED) {  // B of this frame, before its product
#pragma unroll
          for (int c = 0; c < VW; ++c) v[c] += bb[g][c];
        }
        // The product's A-operand, split once here into bf16 hi and lo.
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
      }
    }
    lds_barrier();
    // alpha of the next step, read by its row-wise phase (after the next
    // barrier); this step's reads of alds are complete.
    if constexpr (DECAY) {
      if (tid < DK / 4) reinterpret_cast<u32x4*>(alds)[tid] = al_next;
    }
    // The products, with the second half of the refill between them.
    tiled_mfma_phase<DK>(xsp[0], xsp[1], xs[cur ^ 1], t, tn, toff, trsrc, next, wave, li, lg);
    cur ^= 1;
  };

  // Issue the ring in slot order (pinned against rescheduling) so slot 0 is
  // the oldest load on loop entry.
  load_add(0, bs0, al0);
  load_tiles(0, t0);
  __builtin_amdgcn_sched_barrier(0);
  load_add(min(1, nsteps - 1), bs1, al1);
  load_tiles(min(1, nsteps - 1), t1);
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (DECAY) {  // alpha of step 0
    if (tid < DK / 4) reinterpret_cast<u32x4*>(alds)[tid] = al0;
  }
  // The step count is padded to a multiple of three; a padded step
  // (step >= nsteps) reads a clamped matrix and stores nothing, so the loop
  // body has no early exit.
  for (int step0 = 0; step0 < nsteps; step0 += 3) {
    step_body(step0, t0, bs0, al1, t2, bs2, al2);
    step_body(step0 + 1, t1, bs1, al2, t0, bs0, al0);
    step_body(step0 + 2, t2, bs2, al0, t1, bs1, al1);
  }
}

// The frozen rule's per-frame maps as operand tiles, in place over A_t:
// M_t = Diag(alpha_t)(I - A_t / U), element [k][n] = alpha_k (delta_kn -
// A_t[k][n] / U), split into bf16 hi and lo planes (operand_tile_offset).
// One workgroup per frame reads its whole A_t (A is symmetric, so the eight
// k values of a lane slot are two contiguous runs of row n) before any
// thread writes.  Under a split plan the frames from first_split on are the
// sums of plan_splits token-range partials (partial s at A + s *
// part_stride), and `extra` workgroups after the frames (four per split
// frame, a quarter of B_t each) fold the B_t partials of those frames in
// place, as the inverse step does.
template <int DK>
__global__ __launch_bounds__(kThreads)
void frozen_tiles_kernel(float* __restrict__ A, const float* __restrict__ alpha, float inv_u,
                         unsigned first_split, int plan_splits, unsigned extra, size_t part_stride,
                         float* __restrict__ B_part, size_t b_mat, size_t b_stride) {
  constexpr int SLOTS = DK * DK / 8;                          // 8 elements per lane slot
  constexpr int SPT = (SLOTS + kThreads - 1) / kThreads;      // slots per thread
  const int tid = threadIdx.x;
  if (blockIdx.x >= gridDim.x - extra) {  // four workgroups per split frame
    const unsigned e = blockIdx.x - (gridDim.x - extra);
    const size_t f = first_split + e / 4;
    const size_t quarter = b_mat / 4;
    inv::fold_b_partials(B_part + f * b_mat, plan_splits, (e % 4) * quarter,
                         (e % 4 + 1) * quarter, b_stride, tid, kThreads);
    return;
  }
  const int splits = blockIdx.x >= first_split ? plan_splits : 1;
  float* a = A + (size_t)blockIdx.x * DK * DK;
  const float* al = alpha != nullptr ? alpha + (size_t)blockIdx.x * DK : nullptr;
  // Row segment (n, k0 .. k0 + 3) of slot i, half h: the eight k values of a
  // lane slot are two contiguous runs of row n (A is symmetric).  All of a
  // partial's segments are loaded in one memory round trip, and the
  // token-range partials are added in split order.
  auto seg = [&](int i, int h) -> size_t {
    const int sl = tid + kThreads * i;
    const int lane = sl % 64, tile = sl / 64;
    const int nb = tile / (DK / 32), ks = tile % (DK / 32);
    const int n = 16 * nb + lane % 16, g = lane / 16;
    return (size_t)n * DK + 32 * ks + 16 * h + 4 * g;
  };
  float4 r[SPT][2];
#pragma unroll
  for (int i = 0; i < SPT; ++i)
#pragma unroll
    for (int h = 0; h < 2; ++h)
      if (tid + kThreads * i < SLOTS) r[i][h] = *reinterpret_cast<const float4*>(a + seg(i, h));
  for (int sp = 1; sp < splits; ++sp) {
    float4 x[SPT][2];
#pragma unroll
    for (int i = 0; i < SPT; ++i)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        if (tid + kThreads * i < SLOTS)
          x[i][h] = *reinterpret_cast<const float4*>(a + sp * part_stride + seg(i, h));
#pragma unroll
    for (int i = 0; i < SPT; ++i)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        if (tid + kThreads * i < SLOTS) {
          r[i][h].x += x[i][h].x;
          r[i][h].y += x[i][h].y;
          r[i][h].z += x[i][h].z;
          r[i][h].w += x[i][h].w;
        }
  }
  float v[SPT][8];
#pragma unroll
  for (int i = 0; i < SPT; ++i) {
    const int sl = tid + kThreads * i;
    if (sl >= SLOTS) continue;
    const int lane = sl % 64, tile = sl / 64;
    const int nb = tile / (DK / 32), ks = tile % (DK / 32);
    const int n = 16 * nb + lane % 16, g = lane / 16;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int k0 = 32 * ks + 16 * h + 4 * g;
      const float rv[4] = {r[i][h].x, r[i][h].y, r[i][h].z, r[i][h].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int k = k0 + e;
        const float m = (k == n ? 1.0f : 0.0f) - rv[e] * inv_u;
        v[i][4 * h + e] = al != nullptr ? al[k] * m : m;
      }
    }
  }
  __syncthreads();  // every read of this frame's A_t is done before it is overwritten
  char* t0 = reinterpret_cast<char*>(a);
#pragma unroll
  for (int i = 0; i < SPT; ++i) {
    const int sl = tid + kThreads * i;
    if (sl >= SLOTS) continue;
    const int lane = sl % 64, tile = sl / 64;
    const int nb = tile / (DK / 32), ks = tile % (DK / 32);
    uint32_t hw[4], lw[4];
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const uint32_t hh = pack_bf16x2(v[i][e], v[i][e + 1]);
      hw[e / 2] = hh;
      lw[e / 2] = pack_bf16x2(v[i][e] - bf16_lo(hh), v[i][e + 1] - bf16_hi(hh));
    }
    *reinterpret_cast<u32x4*>(t0 + operand_tile_offset(DK, 0, nb, ks, lane)) =
        u32x4{hw[0], hw[1], hw[2], hw[3]};
    *reinterpret_cast<u32x4*>(t0 + operand_tile_offset(DK, 1, nb, ks, lane)) =
        u32x4{lw[0], lw[1], lw[2], lw[3]};
  }
}

template <int DK, bool DECAY, bool CHUNKED>
hipError_t launch_tiled_k(TiledScanArgs a, int H, hipStream_t stream) {
  a.nwg = (unsigned)H * 2u * (unsigned)(a.DV / 16);
  hipLaunchKernelGGL((scan_tiled_kernel<DK, DECAY, CHUNKED>), dim3(a.nwg), dim3(kThreads), 0,
                     stream, a);
  return hipGetLastError();
}

template <int DK>
hipError_t launch_tiled_t(const TiledScanArgs& a, int H, bool chunked, hipStream_t stream) {
  if (chunked) return launch_tiled_k<DK, false, true>(a, H, stream);
  if (a.alpha != nullptr) return launch_tiled_k<DK, true, false>(a, H, stream);
  return launch_tiled_k<DK, false, false>(a, H, stream);
}

hipError_t launch_tiled(const TiledScanArgs& a, int H, int d_k, bool chunked, hipStream_t stream) {
  switch (d_k) {
    case 32: return launch_tiled_t<32>(a, H, chunked, stream);
    case 64: return launch_tiled_t<64>(a, H, chunked, stream);
    case 128: return launch_tiled_t<128>(a, H, chunked, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_chunk_sequence_scan(const void* Mt, const float* Jc, const float* text_state,
                                      int F, int H, int d_k, int d_v, int chunk, int offset,
                                      int C, float* S_fwd, float* S_rev, hipStream_t stream) {
  TiledScanArgs a{};
  a.tiles = static_cast<const uint16_t*>(Mt);
  a.add = Jc;
  a.text_state = text_state;
  a.F = F;
  a.DV = d_v;
  a.chunk = chunk;
  a.offset = offset;
  a.mats_per_head = 2 * C;
  a.dir_stride = C;
  a.add_scale = 1.0f;
  a.C = C;
  a.S_fwd = S_fwd;
  a.S_rev = S_rev;
  return launch_tiled(a, H, d_k, true, stream);
}

hipError_t launch_frozen_tiles(float* A, float* B_part, SplitPlan plan, const float* alpha, int F,
                               int H, int d_k, int d_v, int tokens, hipStream_t stream) {
  const long long count = (long long)H * F;
  const int splits = plan.splits > 1 && plan.tail > 0 ? plan.splits : 1;
  const unsigned first_split = splits > 1 ? (unsigned)(count - plan.tail) : (unsigned)count;
  const size_t part_stride = (size_t)plan.tail * d_k * d_k;  // partial p of frame f: f + p * tail
  const size_t b_mat = (size_t)d_v * d_k;
  const size_t b_stride = (size_t)plan.tail * b_mat;
  const unsigned extra = splits > 1 ? 4u * (unsigned)plan.tail : 0u;
  const dim3 grid((unsigned)count + extra);
  const float inv_u = 1.0f / (float)tokens;
#define VDA_FROZEN_TILES(DK)                                                                   \
  hipLaunchKernelGGL(frozen_tiles_kernel<DK>, grid, dim3(kThreads), 0, stream, A, alpha, inv_u, \
                     first_split, splits, extra, part_stride, B_part, b_mat, b_stride)
  switch (d_k) {
    case 32: VDA_FROZEN_TILES(32); break;
    case 64: VDA_FROZEN_TILES(64); break;
    case 128: VDA_FROZEN_TILES(128); break;
    default: return hipErrorInvalidValue;
  }
#undef VDA_FROZEN_TILES
  return hipGetLastError();
}

hipError_t launch_frozen_scan_tiled(const void* M_tiles, const float* Bm, const float* text_state,
                                    int F, int H, int d_k, int d_v, int tokens, float* S_fwd,
                                    float* S_rev, hipStream_t stream) {
  TiledScanArgs a{};
  a.tiles = static_cast<const uint16_t*>(M_tiles);
  a.add = Bm;
  a.text_state = text_state;
  a.F = F;
  a.DV = d_v;
  a.chunk = 1;
  a.offset = 0;
  a.C = F;
  a.mats_per_head = F;
  a.dir_stride = 0;
  a.add_scale = 1.0f / sqrtf((float)tokens);
  a.S_fwd = S_fwd;
  a.S_rev = S_rev;
  return launch_tiled(a, H, d_k, true, stream);
}

hipError_t launch_state_scan_tiled(const void* Inv_tiles, const float* Bm, int F, int H, int d_k,
                                   int d_v, const ScanOptions& o, float* S_fwd, float* S_rev,
                                   hipStream_t stream) {
  if (o.frozen) return hipErrorInvalidValue;
  TiledScanArgs a{};
  a.tiles = static_cast<const uint16_t*>(Inv_tiles);
  a.add = Bm;
  a.alpha = o.alpha;
  a.text_state = o.text_state;
  a.F = F;
  a.DV = d_v;
  a.S_fwd = S_fwd;
  a.S_rev = S_rev;
  return launch_tiled(a, H, d_k, false, stream);
}

}  // namespace vda
