// Internal launchers of the four VDA kernels (arguments already validated).
#pragma once

#include <hip/hip_runtime.h>

namespace vda {

// Split plan of the statistics step: the last `tail` of the `count` frames
// are split into `splits` token ranges; every other frame is one range.
// Partial p of frame f sits at matrix index f + p * tail (p = 0: index f).
struct SplitPlan {
  int tail;
  int splits;
};

inline long long partial_count(long long count, SplitPlan plan) {
  return plan.splits > 1 ? count + (long long)plan.tail * (plan.splits - 1) : count;
}

// Workgroups of the statistics step under `plan`.
inline long long stats_workgroups(long long count, SplitPlan plan) {
  return plan.splits > 1 ? count - plan.tail + (long long)plan.tail * plan.splits : count;
}

// Statistics workgroups one compute unit holds at once (occupancy query).
int stats_blocks_per_cu(bool is_f32, int d_k, int d_v);

// Step a1, Eq. 3b: partial frame statistics per token range.  lower_only
// (bf16 storage): A_t's blocks above the diagonal are left unwritten, for a
// caller whose only reader of A_t is launch_frame_inverse.
hipError_t launch_frame_stats(bool is_f32, const void* k, const void* v, const float* beta,
                              int F, int N, int H, int d_k, int d_v, SplitPlan plan,
                              float* A_part, float* B_part, hipStream_t stream,
                              bool lower_only = false);

// Step a2, Eq. 5: Inv = (I + sum of A partials)^{-1} (fp32 matrices, or
// split-bf16 operand tiles when `tiled`); also folds the B partials of every
// split frame into its first partial.  It reads only A_t's blocks on and
// below the diagonal.
hipError_t launch_frame_inverse(const float* A_part, float* B_part, SplitPlan plan,
                                long long count, int d_k, int d_v, bool tiled, float* Inv,
                                hipStream_t stream);

// Options of the scans beyond the core (defaults: the core scan).
struct ScanOptions {
  bool frozen = false;                // Eq. 3c with 1/sqrt(U) scaling; Mat holds A_t
  const float* alpha = nullptr;       // [H][F][d_k] channel decay, or null (1)
  const float* text_state = nullptr;  // [H][d_v][d_k] S_T (both scans start at S_T/2), or null
  int tokens = 0;                     // U, tokens per frame (frozen rule)
};

// Steps a3/a4, Eq. A.1: forward and reverse state scans (exact fp32 products,
// or split-bf16 products with fp32 accumulation).  Mat is Inv_t (joint rule)
// or A_t (frozen rule), symmetric.
hipError_t launch_state_scan(bool exact_f32, const float* Mat, const float* Bm, int F, int H,
                             int d_k, int d_v, const ScanOptions& o, float* S_fwd, float* S_rev,
                             hipStream_t stream);

// The frozen rule (Eq. 3c with the 1/sqrt(U) scaling) on the tiled scan:
// launch_frozen_tiles overwrites each A_t [H][F][d_k][d_k] in place with the
// operand tiles of M_t = Diag(alpha_t)(I - A_t / U) (alpha null: 1), summing
// the token-range partials of split frames (and folding their B_t partials
// into B_part[frame]) under the plan the statistics used, and
// launch_frozen_scan_tiled runs x <- x M_t + B_t / sqrt(U) in both
// directions from S_T / 2 (or zero), storing every frame's entering state.
hipError_t launch_frozen_tiles(float* A, float* B_part, SplitPlan plan, const float* alpha, int F,
                               int H, int d_k, int d_v, int tokens, hipStream_t stream);
hipError_t launch_frozen_scan_tiled(const void* M_tiles, const float* Bm, const float* text_state,
                                    int F, int H, int d_k, int d_v, int tokens, float* S_fwd,
                                    float* S_rev, hipStream_t stream);

// Steps a3/a4 for the joint rule on the bf16 storage path, with Inv_t given
// as split-bf16 operand tiles (operand_tile_offset); alpha and the text
// state of `o` apply, `o.frozen` must be false.
hipError_t launch_state_scan_tiled(const void* Inv_tiles, const float* Bm, int F, int H, int d_k,
                                   int d_v, const ScanOptions& o, float* S_fwd, float* S_rev,
                                   hipStream_t stream);

// Chunk-wise scans (joint rule, bf16 storage path): the chunks of the
// window grid (`chunk` frames counted from `offset` before frame 0) are
// composed into affine maps (M_c as operand tiles, J_c fp32, in `work`),
// then scanned; writes the state entering each chunk, forward at its first
// frame of S_fwd and reverse at its last frame of S_rev.
int chunk_count(int F, int chunk, int offset);
// The chunk-sequence scan alone: x <- x M_c + J_c over the C chunks (M_c as
// operand tiles [H][2][C], J_c [H][2][C][d_v][d_k]), storing the boundary
// states as above.
hipError_t launch_chunk_sequence_scan(const void* Mt, const float* Jc, const float* text_state,
                                      int F, int H, int d_k, int d_v, int chunk, int offset,
                                      int C, float* S_fwd, float* S_rev, hipStream_t stream);
size_t chunked_scan_workspace(int F, int H, int d_k, int d_v, int chunk, int offset);
hipError_t launch_state_scan_chunked(const void* Inv_tiles, const float* Bm, const float* alpha,
                                     const float* text_state, int F, int H, int d_k, int d_v,
                                     int chunk, int offset, void* work, float* S_fwd,
                                     float* S_rev, hipStream_t stream);

// VDA-Prep: Q' = L2(Q), K' = L2(SiLU(conv_k(K))), V' = SiLU(conv_v(V)) from
// token-major projections [B][F][gh*gw][H*d] to [B*H][F][gh*gw][d] (bf16;
// d_k, d_v in {64, 128}).
hipError_t launch_prep(const void* q, const void* k, const void* v, const float* wks,
                       const float* wkt, const float* wvs, const float* wvt, int B, int F, int gh,
                       int gw, int H, int d_k, int d_v, void* q_out, void* k_out, void* v_out,
                       hipStream_t stream);

// Options of the gather beyond the core (defaults: own frame, no decay).
struct GatherOptions {
  const float* alpha = nullptr;  // [H][F][d_k] channel decay, or null (1)
  int chunk = 1;                 // local window: frames per chunk,
  int radius = 0;                // chunks on each side,
  int offset = 0;                // and chunk position of frame 0
  // [H][F][N][d_v] output gate G^L per token and channel (the storage type
  // of q and out), or null: the per-head gate applies.
  const void* gate_tokens = nullptr;
  // Output layout: head problems per clip of a token-major output
  // [H / out_heads][F][N][out_heads * d_v_norm] (head problem b * out_heads
  // + h writes channels h * d_v_norm ..); 1 is frame-major per head,
  // [H][F][N][d_v_norm].
  int out_heads = 1;
  // Query layout, likewise: q_heads > 1 reads q token-major,
  // [H / q_heads][F][N][q_heads * d_k]; 1 is frame-major per head.
  int q_heads = 1;
  // Whether q is the raw projection: the readout then applies the feature
  // map's L2 normalisation to each token's query (Sec. 2.3) itself.
  bool q_l2 = false;
};

// Steps a5-a7, Eq. A.4 / 1a / 1c: gather, readout, RMSNorm and gate.
// d_v_norm: the true number of value channels, which RMSNorm averages over
// and out holds per head (d_v, or fewer when the trailing value channels of
// the padded heads are zero padding: only the first d_v_norm are written).
hipError_t launch_readout(bool is_f32, const void* q, const float* S_fwd, const float* S_rev,
                          const float* gate, int F, int N, int H, int d_k, int d_v,
                          int d_v_norm, const GatherOptions& g, void* out, hipStream_t stream);

// The prompt state from its frame's reduced statistics: S = B Inv (joint
// rule; Inv != null) or S = B * scale (frozen rule).  B [H][pv][pk], Inv
// [H][pk][pk], S [H][d_v][d_k] (pk >= d_k, pv >= d_v).
hipError_t launch_text_state(const float* B, const float* Inv, int H, int pk, int pv, int d_k,
                             int d_v, float scale, float* S, hipStream_t stream);

// Row-wise channel padding (zero fill), in 16-byte pieces.
hipError_t launch_pad_rows(const void* src, void* dst, long long rows, int src_bytes,
                           int dst_bytes, hipStream_t stream);

// Token count of each statistics split (a multiple of the 64-token tile).
inline int stats_tokens_per_split(int N, int splits) {
  const int per = (N + splits - 1) / splits;
  return ((per + 63) / 64) * 64;
}

}  // namespace vda
