// Device code of step a2, Inv_t = (I + A_t)^{-1} (Eq. 5).
//
// I + A_t is symmetric positive definite with every eigenvalue >= 1 (A_t is
// a Gram matrix weighted by beta >= 0; Appendix A.1), so Gauss-Jordan
// elimination needs no pivoting and every leading block is invertible.
//
// One workgroup inverts one d_k x d_k matrix in fp32 by blocked Gauss-Jordan
// with 16 x 16 blocks on v_mfma_f32_16x16x4_f32.  Block rows are dealt out
// to the waves (wave w owns rows w, w + W, ...), each held in MFMA
// accumulator layout (block (i, j): lane (c, g) holds rows 4g..4g+3, column
// c).  Block step kb:
//   1. the owner of row kb inverts the pivot block D = M[kb][kb] by scalar
//      Gauss-Jordan and publishes D^{-1} and the pivot row P_j = M[kb][j]
//      in LDS;
//   2. for its rows i != kb every wave applies
//        M[i][j] -= M[i][kb] D^{-1} P_j,   M[i][kb] = -M[i][kb] D^{-1},
//      and the owner of row kb sets M[kb][j] = D^{-1} P_j, M[kb][kb] = D^{-1}.
// After eliminating block columns 0..kb-1 the matrix is [[X, Y], [Z, S]]
// with X and S symmetric and Z = -Y^T, so M[i][kb] is the transpose of the
// published P_i, negated when i < kb, and M[i][kb] D^{-1} is (up to that
// sign) the transpose of R_i = D^{-1} P_i.  The A-operands a lane supplies
// at k = 4g + s are therefore element s of its own slot of P_i or R_i, and
// each wave forms R_i only for its own rows.  A block (i, j) with
// j > kb that step j will overwrite (i < kb, or i > j) is not updated:
// about a third of the products are skipped.  The owner of row kb + 1
// publishes step kb + 1's pivot during step kb (it updates that row first,
// then inverts the pivot block while the other waves do their products) and
// applies step kb to its other rows at the start of step kb + 1; the LDS
// pivot rows are triple buffered, so each block step needs one barrier.
// With several matrices' workgroups per SIMD, one wave's serial pivot work
// also hides behind another matrix's products.
// Both A_t and its inverse are symmetric, so the column segments of the
// accumulator layout are loaded (for the blocks on and below the diagonal,
// the only ones read) and stored as contiguous row segments of the
// transposed block (the result is the transpose of the computed inverse,
// which equals it up to rounding).
// The token-split partials of A_t are summed in split order while loading
// (fold_b_partials does the same for B_t).  All products and sums are fp32.
#pragma once

#include "vda_common.h"

namespace vda {
namespace inv {

// Pivot block inverse by scalar Gauss-Jordan: lane (li, lg) holds
// D[4lg + r][li] in d[r] on entry and D^{-1} in the same layout on exit.
// Every cross-lane move is a VALU operation, so a pivot costs no LDS round
// trip: the pivot element comes from one lane (v_readlane), pivot row p
// (held by lane group p/4) is copied to all four lane groups by a 16-lane
// and a 32-lane row swap (v_permlane16_swap, v_permlane32_swap), and pivot
// column p (held by lane p of every group) by a row broadcast (DPP
// row_newbcast).  The reciprocal is the hardware estimate refined by one
// Newton step (error <= 1 ulp); the IEEE division sequence would sit on the
// serial path once per pivot.
template <int P>
__device__ __forceinline__ float row_of_group(float x) {
  constexpr int G = P >> 2;
  const uint32_t u = __float_as_uint(x);
  const auto t = __builtin_amdgcn_permlane16_swap(u, u, false, false);  // [r0 r0 r2 r2], [r1 r1 r3 r3]
  const uint32_t y = (G & 1) ? t[1] : t[0];
  const auto v = __builtin_amdgcn_permlane32_swap(y, y, false, false);  // lower / upper pair
  return __uint_as_float((G & 2) ? v[1] : v[0]);
}

template <int P>
__device__ __forceinline__ void pivot_step(float (&d)[4], int li, int lg) {
  constexpr int G = P >> 2, E = P & 3;
  const float rowv = row_of_group<P>(d[E]);                                // D[P][li]
  float colv[4];
#pragma unroll
  for (int r = 0; r < 4; ++r)                                              // D[4lg+r][P]
    colv[r] = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(d[r]), 0x150 + P, 0xf, 0xf,
                                                      false));
  const float piv = __int_as_float(
      __builtin_amdgcn_readlane(__float_as_int(d[E]), P + 16 * G));        // D[P][P]
  float inv = __builtin_amdgcn_rcpf(piv);
  inv = inv * fmaf(-piv, inv, 2.0f);
  const bool on_col = li == P;
  const float rs = rowv * inv;                                             // new pivot row
  // One fused update for every element off the pivot row: d - colv * s with
  // s = rs, and in the pivot column (where colv = d) s = 1 + inv, which
  // gives -d * inv, the eliminated column.
  const float s = on_col ? 1.0f + inv : rs;
#pragma unroll
  for (int r = 0; r < 4; ++r) d[r] = fmaf(-colv[r], s, d[r]);
  if (lg == G) d[E] = on_col ? inv : rs;                                   // pivot row
}

template <int P = 0>
__device__ __forceinline__ void invert_pivot_block(float (&d)[4], int li, int lg) {
  pivot_step<P>(d, li, lg);
  if constexpr (P + 1 < 16) invert_pivot_block<P + 1>(d, li, lg);
}

// D^{-1} of step kb from the pivot buffer pb: accumulator layout, and (being
// symmetric) its own A-operand D^{-1}[li][4lg+s] = d[s].
__device__ __forceinline__ void read_pivot_inverse(const float* pb, int kb, int lane, float (&d)[4]) {
  const float4 v = *reinterpret_cast<const float4*>(pb + (kb * 64 + lane) * 4);
  d[0] = v.x;
  d[1] = v.y;
  d[2] = v.z;
  d[3] = v.w;
}

// The owner of pivot row kb inverts its pivot block D = row[kb] and
// publishes D^{-1} (in slot kb) and P_j = row[j] (j != kb) in pb.
template <int NB>
__device__ __forceinline__ void publish_pivot(const floatx4 (&row)[NB], int kb, float* pb, int li,
                                              int lg, int lane) {
  const floatx4 dd = row[kb];
  float d[4] = {dd[0], dd[1], dd[2], dd[3]};
  // The pivot block is this matrix's critical path: while it runs, the
  // SIMD's arbiter prefers this wave over the other matrices' waves.
  __builtin_amdgcn_s_setprio(2);
  invert_pivot_block(d, li, lg);
  __builtin_amdgcn_s_setprio(0);
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const floatx4 v = j == kb ? floatx4{d[0], d[1], d[2], d[3]} : row[j];
    *reinterpret_cast<float4*>(pb + (j * 64 + lane) * 4) = make_float4(v[0], v[1], v[2], v[3]);
  }
}

// Block step kb for block row i (held in row[]), from step kb's published
// D^{-1} (d) and pivot row P_j (pb).
template <int NB>
__device__ __forceinline__ void update_row(floatx4 (&row)[NB], int i, int kb, const float* pb,
                                           const float (&d)[4], int lane) {
  if (i == kb) {
    // The pivot row: M[kb][j] = D^{-1} P_j from this wave's own P_j.
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if (j == kb) continue;
      const floatx4 pj = row[j];
      floatx4 r = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 4; ++s) r = __builtin_amdgcn_mfma_f32_16x16x4f32(d[s], pj[s], r, 0, 0, 0);
      row[j] = r;
    }
    row[kb] = floatx4{d[0], d[1], d[2], d[3]};
    return;
  }
  // Row i != kb.  With sigma = +1 for i > kb and -1 for i < kb,
  // M[i][kb] = sigma P_i^T, so C_i = M[i][kb] D^{-1} = sigma R_i^T with
  // R_i = D^{-1} P_i, and
  //   M[i][j] -= C_i P_j  (j != kb),   M[i][kb] = -C_i.
  // A-operands at k = 4lg + s: -M[i][kb] -> -sigma P_i[s] and
  // -C_i -> -sigma R_i[s]; B-operands P_j[s] and D^{-1}: d[s].
  const float4 p4 = *reinterpret_cast<const float4*>(pb + (i * 64 + lane) * 4);
  const float pi[4] = {p4.x, p4.y, p4.z, p4.w};
  const float ms = i > kb ? -1.0f : 1.0f;  // -sigma
  floatx4 o = {0.f, 0.f, 0.f, 0.f};
  floatx4 ri = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    o = __builtin_amdgcn_mfma_f32_16x16x4f32(ms * pi[s], d[s], o, 0, 0, 0);
    ri = __builtin_amdgcn_mfma_f32_16x16x4f32(d[s], pi[s], ri, 0, 0, 0);
  }
  float c[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) c[s] = ms * ri[s];
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    // Block (i, j), j > kb, is overwritten at step j (from the pivot row's
    // transpose) unless kb < i <= j: skip those dead updates.
    if (j == kb || (j > kb && (i > j || i < kb))) continue;
    const float4 pj = *reinterpret_cast<const float4*>(pb + (j * 64 + lane) * 4);
    row[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(c[0], pj.x, row[j], 0, 0, 0);
    row[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(c[1], pj.y, row[j], 0, 0, 0);
    row[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(c[2], pj.z, row[j], 0, 0, 0);
    row[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(c[3], pj.w, row[j], 0, 0, 0);
  }
  row[kb] = o;
}

// The elimination for the block rows of wave WV (rows WV, WV + W, ...); a
// template on the wave so that every row-dependent condition is resolved at
// compile time.  All W waves of the workgroup take the same NB barriers.
template <int DK, int WV, bool TILED>
__device__ __forceinline__ void invert_rows(const float* A_part, int splits, size_t part_stride,
                                            size_t base, float* Inv, float (*piv)[DK / 16][64 * 4],
                                            int lane) {
  constexpr int NB = DK / 16;          // 16-wide blocks per side
  constexpr int W = NB < 4 ? NB : 4;   // waves
  constexpr int RPW = NB / W;          // block rows per wave
  const int li = lane & 15;
  const int lg = lane >> 4;

  // acc[q][j]: block (i, j) with i = WV + W q.  Its accumulator holds the
  // column segment M[16i + 4lg .. +3][16j + li].  Only the blocks of A_t on
  // and below the diagonal are read (the statistics may leave the others
  // unwritten): for j >= i, A_t is symmetric, so the segment is read as the
  // contiguous row segment M[16j + li][16i + 4lg .. +3] of block (j, i) with
  // one 16-byte load (and the result is written back the same way); for
  // j < i, straight from block (i, j) as four scalars.
  // All blocks of this wave's rows of one partial are loaded in one memory
  // round trip: the first partial straight into the accumulators, each
  // further token range of a split frame into a staging set that is then
  // added in range order (one round trip per partial).
  auto load_block = [&](const float* m, int i, int j) -> floatx4 {
    if (j >= i)
      return *reinterpret_cast<const floatx4*>(m + (size_t)(16 * j + li) * DK + 16 * i + 4 * lg);
    const float* p = m + (size_t)(16 * i + 4 * lg) * DK + 16 * j + li;
    return floatx4{p[0], p[DK], p[2 * DK], p[3 * DK]};
  };
  floatx4 acc[RPW][NB];
  const float* a0 = A_part + base;
#pragma unroll
  for (int q = 0; q < RPW; ++q)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[q][j] = load_block(a0, WV + W * q, j);
  for (int s = 1; s < splits; ++s) {
    floatx4 x[RPW][NB];
#pragma unroll
    for (int q = 0; q < RPW; ++q)
#pragma unroll
      for (int j = 0; j < NB; ++j) x[q][j] = load_block(a0 + s * part_stride, WV + W * q, j);
#pragma unroll
    for (int q = 0; q < RPW; ++q)
#pragma unroll
      for (int j = 0; j < NB; ++j) acc[q][j] += x[q][j];
  }
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    const int i = WV + W * q;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (4 * lg + r == li) acc[q][i][r] += 1.0f;
  }

  // Step kb's pivot is published by the owner of row kb during step kb - 1
  // (step 0's before the loop): it applies step kb - 1 to row kb first,
  // inverts the new pivot block and publishes it, and defers step kb - 1 for
  // its other rows to the start of step kb.  So the serial pivot chain runs
  // while the other waves do their products, and the pivot buffers are
  // triple buffered (a deferred update still reads step kb - 1's).
  if (WV == 0) publish_pivot<NB>(acc[0], 0, &piv[0][0][0], li, lg, lane);
#pragma unroll
  for (int kb = 0; kb < NB; ++kb) {
    lds_barrier();
    if (kb >= 1 && kb % W == WV) {  // deferred: step kb - 1 for this wave's other rows
      const float* pp = &piv[(kb - 1) % 3][0][0];
      float dp[4];
      read_pivot_inverse(pp, kb - 1, lane, dp);
#pragma unroll
      for (int q = 0; q < RPW; ++q)
        if (WV + W * q != kb) update_row<NB>(acc[q], WV + W * q, kb - 1, pp, dp, lane);
    }
    const float* pb = &piv[kb % 3][0][0];
    float d[4];
    read_pivot_inverse(pb, kb, lane, d);
    if (kb + 1 < NB && (kb + 1) % W == WV) {
      const int qa = (kb + 1) / W;
      update_row<NB>(acc[qa], kb + 1, kb, pb, d, lane);
      publish_pivot<NB>(acc[qa], kb + 1, &piv[(kb + 1) % 3][0][0], li, lg, lane);
    } else {
#pragma unroll
      for (int q = 0; q < RPW; ++q) update_row<NB>(acc[q], WV + W * q, kb, pb, d, lane);
    }
  }

  if constexpr (TILED) {
    // Split-bf16 operand tiles (operand_tile_offset): block (i, j) at lane
    // (li, lg) holds X[16i + 4lg + r][16j + li], which is half i % 2 of that
    // lane's B-operand of tile (nb = j, ks = i / 2), so every lane writes
    // its own 8-byte halves with no exchange.
    char* t0 = reinterpret_cast<char*>(Inv + base);
#pragma unroll
    for (int q = 0; q < RPW; ++q) {
      const int i = WV + W * q;
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const floatx4 a = acc[q][j];
        const uint32_t h01 = pack_bf16x2(a[0], a[1]);
        const uint32_t h23 = pack_bf16x2(a[2], a[3]);
        const uint32_t l01 = pack_bf16x2(a[0] - bf16_lo(h01), a[1] - bf16_hi(h01));
        const uint32_t l23 = pack_bf16x2(a[2] - bf16_lo(h23), a[3] - bf16_hi(h23));
        char* t = t0 + operand_tile_offset(DK, 0, j, i / 2, lane) + (i & 1) * 8;
        *reinterpret_cast<uint2*>(t) = make_uint2(h01, h23);
        *reinterpret_cast<uint2*>(t + (size_t)DK * DK * 2) = make_uint2(l01, l23);
      }
    }
  } else {
#pragma unroll
    for (int q = 0; q < RPW; ++q) {
      const int i = WV + W * q;
#pragma unroll
      for (int j = 0; j < NB; ++j)
        *reinterpret_cast<float4*>(Inv + base + (size_t)(16 * j + li) * DK + 16 * i + 4 * lg) =
            make_float4(acc[q][j][0], acc[q][j][1], acc[q][j][2], acc[q][j][3]);
    }
  }
}

// Sum the token-split partials of B_t into the first one (in place, in
// partial order) over the element range [lo, hi) of the matrix; all threads
// of the workgroup take part.  Each thread holds up to four 16-byte pieces,
// and the pieces of every partial are loaded together, so the whole range
// takes one memory round trip (splits <= 4).
__device__ __forceinline__ void fold_b_partials(float* b0, int splits, size_t lo, size_t hi,
                                                size_t b_stride, int tid, int nthreads) {
  const size_t step = (size_t)nthreads * 4;
  for (size_t idx0 = lo + (size_t)tid * 4; idx0 < hi; idx0 += 4 * step) {
    floatx4 a[4][4];  // [partial][piece]
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const size_t idx = idx0 + e * step;
        a[s][e] = s < splits && idx < hi
                      ? *reinterpret_cast<const floatx4*>(b0 + s * b_stride + idx)
                      : floatx4{0.f, 0.f, 0.f, 0.f};
      }
    floatx4 sum[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) sum[e] = ((a[0][e] + a[1][e]) + a[2][e]) + a[3][e];
    for (int s = 4; s < splits; ++s)  // more than four ranges (stage entry point only)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const size_t idx = idx0 + e * step;
        if (idx < hi) sum[e] += *reinterpret_cast<const floatx4*>(b0 + s * b_stride + idx);
      }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const size_t idx = idx0 + e * step;
      if (idx < hi) *reinterpret_cast<floatx4*>(b0 + idx) = sum[e];
    }
  }
}

// Invert one matrix with the first min(4, d_k/16) waves of the workgroup
// (any further waves only take part in the barriers); `piv` is
// 3 * (d_k/16) * 256 floats of LDS.  The matrix is the sum of `splits`
// partials at A_part + s * part_stride + base; the result goes to Inv + base
// (which may alias the first partial): an fp32 d_k x d_k matrix, or with
// TILED the split-bf16 operand tiles of the same size in bytes.
template <int DK, bool TILED>
__device__ __forceinline__ void invert_matrix(const float* A_part, int splits, size_t part_stride,
                                              size_t base, float* Inv, float* piv_lds, int tid) {
  constexpr int NB = DK / 16;
  constexpr int W = NB < 4 ? NB : 4;
  auto piv = reinterpret_cast<float (*)[NB][64 * 4]>(piv_lds);
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  if (wave >= W) {  // a workgroup with more waves: the others only keep the barriers
    for (int kb = 0; kb < NB; ++kb) lds_barrier();
    return;
  }
  switch (wave) {
    case 0: invert_rows<DK, 0, TILED>(A_part, splits, part_stride, base, Inv, piv, lane); break;
    case 1: invert_rows<DK, 1 % W, TILED>(A_part, splits, part_stride, base, Inv, piv, lane); break;
    case 2: invert_rows<DK, 2 % W, TILED>(A_part, splits, part_stride, base, Inv, piv, lane); break;
    default: invert_rows<DK, 3 % W, TILED>(A_part, splits, part_stride, base, Inv, piv, lane); break;
  }
}

}  // namespace inv
}  // namespace vda
