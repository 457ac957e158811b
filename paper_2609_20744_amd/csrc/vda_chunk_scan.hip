// Chunk-wise scans (Section 4): the frames of each chunk of the local-window
// grid are composed into one affine map of Eq. A.1,
//     S_out = S_in M_c + J_c,
// and the short chunk sequence is then scanned in both directions.  With a
// chunked local window the readout reads the states only at chunk
// boundaries (Eq. A.4: P entering the window's first chunk, R leaving its
// last), so this gives the forward state entering every chunk and the
// reverse state entering it from the right, in F / chunk serial steps
// instead of F.
//
// Two launches:
//   compose     (compose_kernel, here) one workgroup per (head, chunk,
//               direction) for the whole stacked map Z = [M; J]
//               ((d_k + d_v) x d_k).  Z starts at [I; 0] and each frame of
//               the chunk, in scan order, applies
//               Z <- (Z Diag(alpha_t) + [0; B_t]) Inv_t.  M_c is written as
//               split-bf16 operand tiles (the layout of Inv_t), J_c as fp32.
//   chunk scan  (the tiled frame scan in its chunk mode) x <- x M_c + J_c
//               over the chunks in scan order from S_T / 2 (or zero),
//               storing the state entering each chunk at the chunk's first
//               frame (forward) or last frame (reverse).
//
// Compose work split: each of four waves owns up to four 16-row blocks of
// Z, for all d_k columns.  The product is formed as Inv^T Z^T with the
// Inv_t tiles as A operands and Z as B operands, so a lane receives four
// consecutive columns of one row of Z Inv, and the results of output slices
// 2 ks and 2 ks + 1 are exactly the B operand of k step ks of the next
// product: Z never leaves the registers.  Each frame's tiles (d_k * d_k * 4
// bytes) are copied into a two-slot LDS ring (buffer loads to LDS, a quarter
// per wave, with alpha_t) one frame ahead, during the previous frame's
// products, which read every tile once per wave for all of its row blocks;
// one barrier per frame hands the next slot over.  Every chunk is
// independent, so the launch fills the device where the frame scans run
// one workgroup per 16 rows of a chain.
//
// Products: split-bf16 (hi = bf16(x), lo = bf16(x - hi); hi*hi + hi*lo +
// lo*hi) on v_mfma_f32_16x16x32_bf16 with fp32 accumulation, as in the
// frame scans.
#include "vda_common.h"
#include "vda_launch.h"

namespace vda {
namespace {

constexpr int kComposeThreads = kThreads;  // four waves, one per SIMD

__device__ __forceinline__ int chunk_first(int c, int chunk, int offset) {
  return max(0, c * chunk - offset);
}
__device__ __forceinline__ int chunk_last(int c, int F, int chunk, int offset) {
  return min(F - 1, (c + 1) * chunk - offset - 1);
}

__device__ __forceinline__ u32x2 split_hi(const floatx4& v, u32x2& lo) {
  const uint32_t h01 = pack_bf16x2(v[0], v[1]);
  const uint32_t h23 = pack_bf16x2(v[2], v[3]);
  lo = u32x2{pack_bf16x2(v[0] - bf16_lo(h01), v[1] - bf16_hi(h01)),
             pack_bf16x2(v[2] - bf16_lo(h23), v[3] - bf16_hi(h23))};
  return u32x2{h01, h23};
}

struct ComposeArgs {
  const uint16_t* Invt;  // [H][F] frames of operand tiles
  const float* Bm;       // [H][F][d_v][d_k]
  const float* alpha;    // [H][F][d_k] or null
  uint16_t* Mt;          // [H][2][C] operand tiles of M_c
  float* Jc;             // [H][2][C][d_v][d_k]
  int F, chunk, offset, C;
  unsigned nwg;
};

// One workgroup per (head, chunk, direction) holds all of Z.  Wave w owns
// the M-row blocks w + 4 i (i < MW) and the J-row blocks w + 4 i (i < JW) of
// their halves, so which of its blocks take B is fixed at compile time.
template <int DK, int DV, bool DECAY>
__global__ __launch_bounds__(kComposeThreads)
void compose_kernel(ComposeArgs a) {
  constexpr int NB = DK / 16, KB = DK / 32;
  constexpr int MW = (DK / 16 + 3) / 4, JW = (DV / 16 + 3) / 4, R = MW + JW;
  constexpr int TB = DK * DK * 4;  // tile bytes of one matrix
  constexpr int PIECES = TB / 1024;  // 1 KB copies per frame, split over the waves
  __shared__ __align__(16) unsigned char tiles[2][TB];
  // alpha of a frame: one 16-byte piece per lane of wave 0, the first
  // d_k / 4 of them alpha_t.
  __shared__ __align__(16) float alds[DECAY ? 2 : 1][DECAY ? 256 : 4];

  const int F = a.F, C = a.C;
  // L = (h * C + c) * 2 + dir: both directions of a chunk, which read the
  // same frames, side by side (on one XCD).
  const unsigned L = xcd_grouped_id(blockIdx.x, a.nwg);
  const int dir = L & 1;
  const int c = (int)((L >> 1) % C);
  const unsigned hb = (L >> 1) / C;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int li = lane & 15, lg = lane >> 4;

  const int lo = chunk_first(c, a.chunk, a.offset);
  const int hi = chunk_last(c, F, a.chunk, a.offset);
  const int nsteps = hi - lo + 1;
  auto frame_of = [&](int j) { return dir == 0 ? lo + j : hi - j; };
  const size_t mc = ((size_t)hb * 2 + dir) * C + c;  // this map's index
  const size_t mat_b = (size_t)DV * DK;

  // Frame copies into LDS, shared by the four waves: this wave's quarter of
  // frame j's tiles into slot j % 2, and (wave 0, decay) alpha of frame j
  // into alpha slot j % 2.
  const __amdgpu_buffer_rsrc_t trsrc =
      make_rsrc(a.Invt + (size_t)hb * F * (TB / 2), (uint32_t)F * (uint32_t)TB);
  const __amdgpu_buffer_rsrc_t arsrc =
      make_rsrc(DECAY ? a.alpha + (size_t)hb * F * DK : a.Bm, DECAY ? (uint32_t)(F * DK * 4) : 0u);
  constexpr int WPIECES = (PIECES + 3) / 4;  // copies per wave and frame
  // Copy i of this wave's quarter of frame j's tiles into slot j % 2.
  auto copy_piece = [&](int j, int i) {
    const int piece = wave + 4 * i;
    if (PIECES % 4 == 0 || piece < PIECES)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          trsrc, (__attribute__((address_space(3))) void*)&tiles[j & 1][piece * 1024], 16,
          (uint32_t)frame_of(j) * (uint32_t)TB + (uint32_t)piece * 1024u + (uint32_t)lane * 16u, 0,
          0, 0);
  };
  auto copy_tiles = [&](int j) {
#pragma unroll
    for (int i = 0; i < WPIECES; ++i) copy_piece(j, i);
  };
  auto copy_alpha = [&](int j) {
    if constexpr (DECAY) {
      if (wave == 0 && j < nsteps)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            arsrc, (__attribute__((address_space(3))) void*)&alds[j & 1][0], 16,
            lane < DK / 4 ? (uint32_t)(frame_of(j) * DK * 4 + lane * 16) : kOutOfRange, 0, 0, 0);
    }
  };

  // Row block r of this wave: M rows for r < MW (Z row = M row), J rows
  // after (Z row d_k + J row); live if inside the matrix.
  int vrow[R];  // row within M or J
  bool live[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int blk = wave + 4 * (r < MW ? r : r - MW);
    vrow[r] = 16 * blk + li;
    live[r] = 16 * blk < (r < MW ? DK : DV);
  }
  const __amdgpu_buffer_rsrc_t brsrc =
      make_rsrc(a.Bm + (size_t)hb * F * mat_b, (uint32_t)(F * mat_b * 4));

  floatx4 acc[R][NB];
  u32x4 add[JW][NB];  // B of the next prepare (J rows)
  auto load_b = [&](int t) {
#pragma unroll
    for (int q = 0; q < JW; ++q)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        add[q][nb] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                       brsrc,
                       (int)(live[MW + q] ? (uint32_t)t * (uint32_t)(mat_b * 4) +
                                                (uint32_t)((vrow[MW + q] * DK + 16 * nb + 4 * lg) * 4)
                                          : kOutOfRange),
                       0, 0));
  };

  // The split Z of the next product (B operands per row block and k step).
  u32x4 xhi[R][KB], xlo[R][KB];
  // prepare j: decay (alpha of frame j; from memory for j = 0, else from LDS
  // slot j % 2), add B of frame j on J rows, split.
  auto prepare = [&](int j) {
    auto piece = [&](int r, int nb, u32x2& lw) -> u32x2 {
      floatx4 v = acc[r][nb];
      if constexpr (DECAY) {
        const floatx4 al =
            j == 0 ? *reinterpret_cast<const floatx4*>(a.alpha + ((size_t)hb * F + frame_of(0)) * DK +
                                                       16 * nb + 4 * lg)
                   : *reinterpret_cast<const floatx4*>(&alds[j & 1][16 * nb + 4 * lg]);
        v *= al;
      }
      if (r >= MW) {
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] += __uint_as_float(add[r - MW][nb][i]);
      }
      return split_hi(v, lw);
    };
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int ks = 0; ks < KB; ++ks) {
        u32x2 l0, l1;
        const u32x2 h0 = piece(r, 2 * ks, l0);
        const u32x2 h1 = piece(r, 2 * ks + 1, l1);
        xhi[r][ks] = u32x4{h0[0], h0[1], h1[0], h1[1]};
        xlo[r][ks] = u32x4{l0[0], l0[1], l1[0], l1[1]};
      }
  };

  // Z = [I; 0], frame 0's tiles (and alpha of frame 1) into LDS, frame 0's
  // operand.
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      floatx4 x = {0.f, 0.f, 0.f, 0.f};
      if (r < MW) {
#pragma unroll
        for (int i = 0; i < 4; ++i) x[i] = vrow[r] == 16 * nb + 4 * lg + i ? 1.0f : 0.0f;
      }
      acc[r][nb] = x;
    }
  copy_tiles(0);
  copy_alpha(1);
  load_b(frame_of(0));
  prepare(0);
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): this wave's copies are in LDS
  lds_barrier();

  for (int j = 0; j < nsteps; ++j) {
    // Slot (j + 1) % 2 was read last in step j - 1: copy the next frame's
    // tiles (and alpha two frames on) now, and B of the next frame, all in
    // flight during the products.
    // The next frame's tiles are copied a piece at a time between the
    // products below (a burst of copies would stall the issuing wave until
    // the memory pipeline had taken most of them); B of the next frame is
    // in flight during the products too.
    const bool more = j + 1 < nsteps;
    if (more) load_b(frame_of(j + 1));
    copy_alpha(j + 2);
    const unsigned char* tl = tiles[j & 1];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[r][nb] = floatx4{0.f, 0.f, 0.f, 0.f};
    // For each tile pair, the products of all row blocks: independent
    // accumulators rotate between dependent products.  The next pair's
    // tiles are read from LDS during this pair's products.
    auto read_pair = [&](int ks, int nb, bf16x8& th, bf16x8& tw) {
      th = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(tl + operand_tile_offset(DK, 0, nb, ks, lane)));
      tw = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(tl + operand_tile_offset(DK, 1, nb, ks, lane)));
    };
    bf16x8 nth, ntw;
    read_pair(0, 0, nth, ntw);
#pragma unroll
    for (int ks = 0; ks < KB; ++ks) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const bf16x8 th = nth, tw = ntw;
        const int q = ks * NB + nb;  // iteration index, 0 .. KB * NB - 1
        if (q + 1 < KB * NB) read_pair((q + 1) / NB, (q + 1) % NB, nth, ntw);
        // Copies spread evenly over the KB * NB iterations.
        if (more && (q * WPIECES) / (KB * NB) != ((q + 1) * WPIECES) / (KB * NB))
          copy_piece(j + 1, (q * WPIECES) / (KB * NB));
#pragma unroll
        for (int r = 0; r < R; ++r)
          acc[r][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              th, __builtin_bit_cast(bf16x8, xlo[r][ks]), acc[r][nb], 0, 0, 0);
#pragma unroll
        for (int r = 0; r < R; ++r)
          acc[r][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              tw, __builtin_bit_cast(bf16x8, xhi[r][ks]), acc[r][nb], 0, 0, 0);
#pragma unroll
        for (int r = 0; r < R; ++r)
          acc[r][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              th, __builtin_bit_cast(bf16x8, xhi[r][ks]), acc[r][nb], 0, 0, 0);
        // Keep the scheduler from hoisting further tile reads (it would
        // hold them all in registers at once).
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    if (j + 1 < nsteps) prepare(j + 1);
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): this wave's copies are in LDS
    lds_barrier();
  }

  // acc holds Z after the chunk.  J rows: fp32 to J_c.  M rows: through an
  // LDS transpose (the tile slots are free after the last barrier) into
  // operand tiles of M_c.
  float* jc = a.Jc + mc * mat_b;
  constexpr int TLD = DK + 8;  // bf16 row stride of the transposed planes
  uint16_t* mt = reinterpret_cast<uint16_t*>(&tiles[0][0]);  // [plane][n][k]
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (!live[r]) continue;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      if (r < MW) {
        u32x2 lw;
        const u32x2 hw = split_hi(acc[r][nb], lw);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int n = 16 * nb + 4 * lg + i;
          const uint32_t hv = i & 1 ? hw[i >> 1] >> 16 : hw[i >> 1] & 0xffffu;
          const uint32_t lv = i & 1 ? lw[i >> 1] >> 16 : lw[i >> 1] & 0xffffu;
          mt[n * TLD + vrow[r]] = (uint16_t)hv;
          mt[DK * TLD + n * TLD + vrow[r]] = (uint16_t)lv;
        }
      } else {
        *reinterpret_cast<floatx4*>(jc + (size_t)vrow[r] * DK + 16 * nb + 4 * lg) = acc[r][nb];
      }
    }
  }
  lds_barrier();
  unsigned char* dst = reinterpret_cast<unsigned char*>(a.Mt) + mc * TB;
  for (int tix = wave; tix < 2 * NB * KB; tix += 4) {
    const int p = tix / (NB * KB), nb = (tix / KB) % NB, ks = tix % KB;
    const uint16_t* srow = mt + p * DK * TLD + (16 * nb + li) * TLD + 32 * ks + 4 * lg;
    const u32x2 e0 = *reinterpret_cast<const u32x2*>(srow);
    const u32x2 e1 = *reinterpret_cast<const u32x2*>(srow + 16);
    *reinterpret_cast<u32x4*>(dst + operand_tile_offset(DK, p, nb, ks, lane)) =
        u32x4{e0[0], e0[1], e1[0], e1[1]};
  }
}

template <int DK, int DV>
hipError_t launch_compose_v(const ComposeArgs& a, bool decay, hipStream_t stream) {
  if (decay)
    hipLaunchKernelGGL((compose_kernel<DK, DV, true>), dim3(a.nwg), dim3(kComposeThreads), 0,
                       stream, a);
  else
    hipLaunchKernelGGL((compose_kernel<DK, DV, false>), dim3(a.nwg), dim3(kComposeThreads), 0,
                       stream, a);
  return hipGetLastError();
}

template <int DK>
hipError_t launch_compose_t(ComposeArgs a, int H, int d_v, bool decay, hipStream_t stream) {
  a.nwg = (unsigned)H * 2u * (unsigned)a.C;
  switch (d_v) {
    case 32: return launch_compose_v<DK, 32>(a, decay, stream);
    case 64: return launch_compose_v<DK, 64>(a, decay, stream);
    case 128: return launch_compose_v<DK, 128>(a, decay, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int chunk_count(int F, int chunk, int offset) { return (F - 1 + offset) / chunk + 1; }

size_t chunked_scan_workspace(int F, int H, int d_k, int d_v, int chunk, int offset) {
  const size_t per = (size_t)d_k * d_k * 4 + (size_t)d_v * d_k * 4;
  return (size_t)H * 2 * (size_t)chunk_count(F, chunk, offset) * per;
}

hipError_t launch_state_scan_chunked(const void* Inv_tiles, const float* Bm, const float* alpha,
                                     const float* text_state, int F, int H, int d_k, int d_v,
                                     int chunk, int offset, void* work, float* S_fwd,
                                     float* S_rev, hipStream_t stream) {
  ComposeArgs a{};
  a.Invt = static_cast<const uint16_t*>(Inv_tiles);
  a.Bm = Bm;
  a.alpha = alpha;
  a.F = F;
  a.chunk = chunk;
  a.offset = offset;
  a.C = chunk_count(F, chunk, offset);
  const size_t mt_bytes = (size_t)H * 2 * a.C * d_k * d_k * 4;
  a.Mt = static_cast<uint16_t*>(work);
  a.Jc = reinterpret_cast<float*>(static_cast<char*>(work) + mt_bytes);
  const bool decay = alpha != nullptr;
  hipError_t e;
  switch (d_k) {
    case 32: e = launch_compose_t<32>(a, H, d_v, decay, stream); break;
    case 64: e = launch_compose_t<64>(a, H, d_v, decay, stream); break;
    case 128: e = launch_compose_t<128>(a, H, d_v, decay, stream); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  return launch_chunk_sequence_scan(a.Mt, a.Jc, text_state, F, H, d_k, d_v, chunk, offset, a.C,
                                    S_fwd, S_rev, stream);
}

}  // namespace vda
