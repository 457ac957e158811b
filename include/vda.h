/*
 * vda.h -- Video Delta Attention (VDA) forward pass on AMD Instinct MI355X (gfx950).
 *
 * VDA is the linear branch of Video DeltaNet (arXiv 2609.20744).  For every
 * independent head problem h and every frame t (U = N tokens per frame) it
 * forms the frame statistics (Eq. 3b)
 *     A_t = K_t^T Diag(beta_t) K_t            (d_k x d_k)
 *     B_t = V_t^T Diag(beta_t) K_t            (d_v x d_k)
 * and updates a d_v x d_k state once per frame with the joint solve (Eq. 5,
 * no decay, so Sbar_t = S_{t-1})
 *     S_t = (S_{t-1} + B_t) (I + A_t)^{-1},
 * scanned forward (P) and backward (R) over the frames from a zero state
 * (Eq. A.1; Algorithm 1, step 5).  Frame t reads the states outside itself
 * (Eq. A.4 with the local window reduced to the own frame, Eq. 1a)
 *     o_{t,u} = (P_{t-1} + R_{t+1}) q_{t,u}
 * and the branch epilogue (Eq. 1c) gives
 *     y_{t,u} = gate_h * o_{t,u} / sqrt(mean_j o_{t,u,j}^2 + 1e-6).
 * Frame 1 reads only R_2, frame F only P_{F-1}; a one-frame clip gives y = 0.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All tensor pointers are DEVICE pointers owned by the caller; the library
 *    never frees or retains them.  Tensors are dense, row-major, frame-major:
 *        q, k      [H][F][N][d_k]
 *        v, out    [H][F][N][d_v]
 *        beta      [H][F][N]     fp32, per-token write strength, >= 0
 *                                 (0 allowed; negative values are not checked
 *                                 and give undefined results)
 *        gate      [H]           fp32, per-head output gate (already squashed)
 *    H counts independent head problems (batch folded in: H = B * heads).
 *  - Supported head dimensions: d_k, d_v in {32, 64, 128} for every entry
 *    point, and also 16 for vda_forward / vda_forward_f32.  F, N, H >= 1.
 *    Offsets are 32-bit: H*F*64, N*d*4 and F*d*d*4 (d the larger of d_k and
 *    d_v, at least 32) must each stay below 2^31 (else VDA_ERR_SIZE).
 *  - q, k, v, out and the fp32 work buffers must be 16-byte aligned; beta and
 *    gate 4-byte aligned.  out must not overlap any input.
 *  - Every call is asynchronous on `stream` (0 = the null stream): it
 *    validates its arguments on the host, enqueues kernels and returns.  It
 *    never synchronises.  Invalid arguments are reported before anything is
 *    enqueued.  A device fault surfaces at the caller's next synchronisation.
 *  - Calls keep no state between them except per-device cached properties
 *    and cached workspace buffers; they may be issued concurrently from
 *    several threads on different streams.
 *  - Results are deterministic: no floating-point atomics are used.
 *  - No C++ exception crosses this interface.
 */
#ifndef VDA_H
#define VDA_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes returned by every entry point. */
typedef enum {
  VDA_OK = 0,
  VDA_ERR_NULL = 1,        /* a required pointer is NULL                      */
  VDA_ERR_SIZE = 2,        /* F, N, H or splits < 1, or sizes overflow limits */
  VDA_ERR_UNSUPPORTED = 3, /* d_k or d_v not a supported head dimension      */
  VDA_ERR_ALIGN = 4,       /* a pointer is not aligned as required            */
  VDA_ERR_OVERLAP = 5,     /* the output overlaps an input                    */
  VDA_ERR_HIP = 6,         /* the HIP runtime reported an error               */
  VDA_ERR_NOMEM = 7,       /* workspace allocation failed                     */
  VDA_ERR_SCRATCH = 8      /* vda_forward_noalloc: one head's workspace is
                              larger than VDA_NOALLOC_SCRATCH_BYTES           */
} vda_status;

/* Human-readable name of a status code (static storage; never NULL). */
const char* vda_status_string(int status);

/* ------------------------------------------------------------------------- */
/* Whole operator                                                             */
/* ------------------------------------------------------------------------- */

/*
 * vda_forward -- the whole forward pass (Eq. 3b, 5, A.1, A.4, 1a, 1c) with
 * bf16 storage for q, k, v (inputs) and out (output, round-to-nearest-even).
 * Frame statistics and the readout run on bf16 matrix cores with fp32
 * accumulation; (I + A_t)^{-1}, the recurrent states and the epilogue are
 * fp32, and the state products use split-bf16 operands (vda_frame_inverse_tiles
 * and vda_state_scan_tiles are its steps a2-a4).
 * Workspace of (P*(d_k*d_k + d_v*d_k) + 2*H*F*d_v*d_k)*4 bytes, with
 * P = H*F + T*(S-1) partials of the plan (T, S) = vda_default_split_plan(F,
 * N, H, d_k, d_v, is_f32) (P = H*F when S == 1), comes from a per-device cache of
 * library-owned device buffers: a buffer is reused by later calls on the
 * same stream, or on another stream once the work of its last call has
 * finished, and otherwise a new one is allocated (hipMalloc; VDA_ERR_NOMEM
 * on failure).  Cached buffers are kept until vda_release_workspace frees
 * them or the process ends.
 * A 16-channel d_k or d_v is run as a 32-channel head whose extra channels
 * are zero: q, k (and v) are copied into padded workspace buffers, zero
 * channels leave A_t, B_t, the states and the readout unchanged, RMSNorm
 * averages over the true d_v, and the padded output is copied back into
 * out.  The workspace then also holds those padded copies (the formula above
 * with 32 for the padded dimension, plus 2*H*F*N*32 elements of the storage
 * type per padded dimension).
 */
int vda_forward(const void* q, const void* k, const void* v,
                const float* beta, const float* gate,
                int F, int N, int H, int d_k, int d_v,
                void* out, hipStream_t stream);

/* Bytes of the fixed device scratch array of vda_forward_noalloc. */
#define VDA_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)

/*
 * vda_forward_noalloc -- vda_forward for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Same arguments, semantics, argument checks and kernels
 * as vda_forward; the call allocates and frees nothing.  Its workspace is a
 * fixed array of VDA_NOALLOC_SCRATCH_BYTES (256 MiB) of device memory that
 * the library's code object holds on every device the library runs on,
 * until the process ends.  The caller still passes all inputs and out.
 * When vda_forward's workspace for all H heads is larger than the array,
 * the heads run in consecutive groups, each as one forward pass over its
 * heads (the largest groups that fit); head problems are independent, so
 * the results are vda_forward's up to the summation order of the split
 * statistics.  Every call on a device shares that device's one array, and
 * the array keeps the last call's contents (nothing in it needs to start at
 * zero): calls that overlap in time on one device, on different streams or
 * from different threads, race and give undefined results; order them on
 * one stream or with events.
 * Errors: as vda_forward; VDA_ERR_SCRATCH (nothing enqueued) when a single
 * head's workspace is larger than the array, e.g. more than about 1000
 * frames at d_k = d_v = 128; VDA_ERR_HIP if the array's device address
 * cannot be obtained or a launch fails.
 */
int vda_forward_noalloc(const void* q, const void* k, const void* v,
                        const float* beta, const float* gate,
                        int F, int N, int H, int d_k, int d_v,
                        void* out, hipStream_t stream);

/*
 * vda_forward_f32 -- identical semantics and arguments with fp32 storage for
 * q, k, v and out; every product and sum is computed in fp32.
 */
int vda_forward_f32(const float* q, const float* k, const float* v,
                    const float* beta, const float* gate,
                    int F, int N, int H, int d_k, int d_v,
                    float* out, hipStream_t stream);

/* ------------------------------------------------------------------------- */
/* The full operator: decay, local window, text state, and the frozen rule    */
/* ------------------------------------------------------------------------- */

/* Frame update rule. */
typedef enum {
  /* Eq. 5 (Sec. 3.2): S_t = (Sbar_t + B_t)(I + A_t)^{-1}, the VDA joint solve. */
  VDA_RULE_JOINT = 0,
  /* Eq. 3c (Sec. 3.1) with every key scaled by 1/sqrt(U), U = N tokens per
   * frame (Sec. 3.2, App. A.2): S_t = Sbar_t (I - A_t / U) + B_t / sqrt(U),
   * the frozen-state additive update the paper compares against. */
  VDA_RULE_FROZEN_SCALED = 1
} vda_rule;

/*
 * Options of vda_forward_ex.  A NULL pointer to this struct, or all fields at
 * their defaults (rule 0, NULL pointers, chunk 1, radius 0, offset 0,
 * out_heads 0, q_heads 0), give exactly vda_forward.
 *  - rule: a vda_rule.
 *  - alpha: NULL (alpha = 1) or a DEVICE pointer to [H][F][d_k] fp32 channel
 *    decays in [0, 1] (16-byte aligned), one per frame and key channel:
 *    Sbar_t = S_{t-1} Diag(alpha_t) (Eq. 5, A.1; Eq. 3a for the frozen rule),
 *    and the decay bridge of Eq. A.4.  Values outside [0, 1] are not checked.
 *  - text_state: NULL (zero) or a DEVICE pointer to [H][d_v][d_k] fp32 S_T
 *    (16-byte aligned): both scans start from S_T / 2 (Eq. 1b).
 *  - window_chunk, window_radius, window_offset: the local Softmax window of
 *    each frame (Sec. 2.1; App. A.3).  Frames are grouped into chunks of
 *    window_chunk >= 1 consecutive frames, counted from window_offset
 *    (0 <= offset < chunk) positions before frame 0 (for example a leading
 *    anchor frame).  Frame t's window [l_t, h_t] is its own chunk and
 *    window_radius >= 0 chunks on each side, clipped to [0, F).  The paper's
 *    setting is chunk 5, radius 1 (offset 1 with one leading anchor).
 *  - gate_tokens: NULL (the per-head gate applies) or a DEVICE pointer to
 *    [H][F][N][d_v] output gates G^L in the storage type of q and out (bf16
 *    for vda_forward_ex, fp32 for vda_forward_ex_f32; 16-byte aligned): the
 *    content-dependent sigmoid gate of Eq. 1c, one value per token and value
 *    channel, computed upstream and applied after RMSNorm,
 *    out[t][u][c] = G^L[t][u][c] * RMSNorm(S~_t q[t][u])[c].  It replaces
 *    the per-head gate, whose pointer may then be NULL.
 *  - out_heads: the layout of out.  0: frame-major per head, [H][F][N][d_v]
 *    (as vda_forward).  out_heads > 0: token-major, the layout of the
 *    attention output that the model's output projection reads (the final
 *    layout conversion of the epilogue, Sec. 4): the H head problems are
 *    H / out_heads clips of out_heads heads each, and out is
 *    [H / out_heads][F][N][out_heads * d_v], head problem b * out_heads + h
 *    writing channels h * d_v .. h * d_v + d_v - 1 of its clip's rows.  The
 *    inputs and gate_tokens keep their per-head layouts.  VDA_ERR_SIZE if
 *    out_heads < 0, if it does not divide H, or if (N + 64) * out_heads * d_v
 *    elements of one frame exceed 2^31 bytes.
 *  - q_heads: the form of q.  0: q is the feature-mapped query phi(q) in the
 *    frame-major per-head layout [H][F][N][d_k] (as vda_forward).  q_heads
 *    > 0: q is the raw query projection in its token-major layout
 *    [H / q_heads][F][N][q_heads * d_k] (head problem b * q_heads + h reads
 *    channels h * d_k .. h * d_k + d_k - 1 of its clip's rows), and the
 *    readout applies the query's L2 feature map itself (Sec. 2.3: each token
 *    of each head divided by sqrt(sum of its squared channels + 1e-6), the
 *    map vda_prep applies).  RMSNorm is invariant to a positive per-token
 *    scale up to its epsilon, so the readout folds the division into the
 *    norm: with o = S~_t q the raw product and n = |q|^2 + 1e-6,
 *    RMSNorm(o / sqrt(n)) = o / sqrt(mean(o^2) + eps * n) times the norm
 *    weight, which is what is computed (no normalised copy of q is rounded
 *    to the storage type).  k and v keep the per-head layout (vda_prep
 *    writes it; its query output can then be skipped).  VDA_ERR_SIZE if
 *    q_heads < 0, if it does not divide H, or if (N + 64) * q_heads * d_k
 *    elements of one frame exceed 2^31 bytes; VDA_ERR_UNSUPPORTED if d_k is
 *    not one of the kernels' key widths (32, 64, 128; a narrower key is
 *    zero-padded, which needs the per-head query layout).
 */
typedef struct vda_options {
  int rule;
  const float* alpha;
  const float* text_state;
  int window_chunk;
  int window_radius;
  int window_offset;
  const void* gate_tokens;
  int out_heads;
  int q_heads;
} vda_options;

/*
 * vda_forward_ex -- the linear branch of Algorithm 1, steps 3-7, with the
 * options above (bf16 storage; otherwise as vda_forward).  Per head, with
 * frames numbered 0..F-1 here:
 *     P_0 = R_F = S_T / 2,
 *     P_{j+1} = update(P_j, frame j),   R_j = update(R_{j+1}, frame j),
 * where update applies the rule to Sbar = S Diag(alpha_j) with A_j, B_j (so
 * P_j is the forward state after frames 0..j-1 and R_j the reverse state
 * after frames F-1..j), and the gather of Eq. A.4 reads
 *     S~_t = P_{l_t} Diag(prod_{r=l_t..t} alpha_r)
 *          + R_{h_t+1} Diag(prod_{r=t..h_t} alpha_r),
 *     out[t][u] = gate * RMSNorm(S~_t q[t][u])  (G^L elementwise in place of
 * gate with gate_tokens).  A window
 * that covers the whole clip is evaluated as written (both sides read the
 * decayed initial state); callers that bypass the linear branch in that case
 * do so themselves.  With fp32 storage the frozen rule never splits frames
 * (its scan reads the statistics directly); with bf16 storage it splits them
 * as vda_forward does (its map step sums the partials).  Errors: VDA_ERR_UNSUPPORTED
 * for an unknown rule, VDA_ERR_SIZE for invalid window fields, VDA_ERR_ALIGN,
 * VDA_ERR_OVERLAP if out overlaps alpha, text_state or gate_tokens,
 * VDA_ERR_NULL if both gate and gate_tokens are NULL.
 */
int vda_forward_ex(const void* q, const void* k, const void* v,
                   const float* beta, const float* gate,
                   int F, int N, int H, int d_k, int d_v,
                   const vda_options* opts, void* out, hipStream_t stream);

/* vda_forward_ex_f32 -- the same with fp32 storage (as vda_forward_f32). */
int vda_forward_ex_f32(const float* q, const float* k, const float* v,
                       const float* beta, const float* gate,
                       int F, int N, int H, int d_k, int d_v,
                       const vda_options* opts, float* out, hipStream_t stream);

/* ------------------------------------------------------------------------- */
/* VDA-Prep: the linear branch's feature map before the operator              */
/* ------------------------------------------------------------------------- */

/*
 * vda_prep -- the feature map of the linear branch (Sec. 2.3; the VDA-Prep
 * step of Sec. 4) from the QKV projections to the operator's inputs:
 *     q_out = L2(q),  k_out = L2(SiLU(T_k * S_k * k)),  v_out = SiLU(T_v * S_v * v)
 * S is a depthwise 5 x 5 spatial filter over each frame's latent grid and T
 * a depthwise five-tap temporal filter over the frames, both centred
 * cross-correlations with zero padding at the grid and clip borders:
 *     (S x)[f][y][x][c] = sum_{i,j<5} w_spatial[c][i*5+j] x[f][y+i-2][x+j-2][c]
 *     (T s)[f][y][x][c] = sum_{i<5}   w_temporal[c][i]    s[f+i-2][y][x][c]
 * SiLU(x) = x / (1 + exp(-x)); L2 divides one token of one head by
 * sqrt(sum of its d squared channels + 1e-6).  The F frames are the clip's
 * interior frames (anchor rows already removed, Algorithm 1 step 2).
 *  - q, k [B][F][grid_h*grid_w][H*d_k], v [B][F][grid_h*grid_w][H*d_v]:
 *    bf16 DEVICE pointers, tokens of a frame in row-major grid order, head h
 *    owning channels h*d .. h*d+d-1 (the projections' token-major layout).
 *  - wk_spatial [H*d_k][25], wk_temporal [H*d_k][5], wv_spatial [H*d_v][25],
 *    wv_temporal [H*d_v][5]: fp32 DEVICE pointers, one filter per channel.
 *  - q_out, k_out [B*H][F][grid_h*grid_w][d_k], v_out [..][d_v]: bf16 DEVICE
 *    pointers, the frame-major per-head layout of vda_forward (index b*H+h).
 *  - q and q_out may both be NULL: the query map is then not computed here
 *    (vda_forward_ex with q_heads = H reads the raw token-major query and
 *    applies the L2 map in its readout); one of the two NULL alone is
 *    VDA_ERR_NULL.
 * The filters accumulate in fp32; results are rounded to bf16 once.
 * d_k, d_v in {64, 128}; B, F, grid_h, grid_w, H >= 1.  Tensors 16-byte
 * aligned, filters 4-byte aligned; no output may overlap an input or
 * another output.  Errors: VDA_ERR_NULL, VDA_ERR_SIZE, VDA_ERR_UNSUPPORTED,
 * VDA_ERR_ALIGN, VDA_ERR_OVERLAP, VDA_ERR_HIP.
 */
int vda_prep(const void* q, const void* k, const void* v,
             const float* wk_spatial, const float* wk_temporal,
             const float* wv_spatial, const float* wv_temporal,
             int B, int F, int grid_h, int grid_w, int H, int d_k, int d_v,
             void* q_out, void* k_out, void* v_out, hipStream_t stream);

/*
 * vda_text_state -- the prompt state S_T of Eq. 1b (Sec. 2.2), formed as the
 * paper does: the prompt is a leading virtual frame updated from the zero
 * state (Sec. 4).  Per head h, over its L prompt tokens, with
 * A_T = sum_u beta k k^T and B_T = sum_u beta v k^T (Eq. 3b):
 *     rule VDA_RULE_JOINT           S_T[h] = B_T (I + A_T)^{-1}   (Eq. 5)
 *     rule VDA_RULE_FROZEN_SCALED   S_T[h] = B_T / sqrt(L)        (Eq. 3c, U = L)
 * The result is the text_state of vda_options (the scans then start from
 * S_T / 2).
 *  - k [H][L][d_k], v [H][L][d_v]: DEVICE, bf16 (is_f32 == 0) or fp32
 *    (is_f32 != 0), 16-byte aligned; beta [H][L] fp32 >= 0, 4-byte aligned.
 *  - S_T [H][d_v][d_k] fp32, DEVICE, 16-byte aligned, written entirely; it
 *    must not overlap the inputs.
 *  - d_k, d_v in {16, 32, 64, 128}; L, H >= 1, with the limits of the
 *    frame shape (N = L, F = 1).
 * The statistics, inverse and precision are those of vda_forward's frames
 * (bf16 storage rounds beta * k to bf16; the inverse is fp32); the final
 * product is an fp32 loop.  Work memory comes from the library's per-device
 * cache, as for vda_forward.  Errors: VDA_ERR_NULL, VDA_ERR_SIZE,
 * VDA_ERR_UNSUPPORTED (dimension or rule), VDA_ERR_ALIGN, VDA_ERR_OVERLAP,
 * VDA_ERR_NOMEM, VDA_ERR_HIP.  Asynchronous on `stream`.
 */
int vda_text_state(const void* k, const void* v, const float* beta, int L, int H,
                   int d_k, int d_v, int rule, int is_f32, float* S_T, hipStream_t stream);

/*
 * vda_release_workspace -- frees the workspace buffers that the library has
 * cached on `device` (-1: the current device) for vda_forward,
 * vda_forward_ex(_f32), vda_forward_f32 and vda_text_state, except buffers
 * that a call on another host thread is using at that moment (they stay
 * cached).  Before freeing a buffer it waits on the host until the work of
 * the buffer's last call has finished, so it blocks the calling thread and
 * must not be called while a stream is being captured.  Later calls
 * allocate again as they need.  *bytes_freed (may be NULL) receives the
 * bytes freed.  The current device is left as it was.
 * Errors: VDA_ERR_SIZE if device < -1 or device is not a device index;
 * VDA_ERR_HIP if the runtime fails (buffers freed before the failure stay
 * freed).
 */
int vda_release_workspace(int device, size_t* bytes_freed);

/*
 * vda_workspace_bytes -- bytes of workspace the library currently holds
 * cached on `device` (-1: the current device), in use or idle.
 * Errors: VDA_ERR_NULL if bytes is NULL; VDA_ERR_SIZE, VDA_ERR_HIP as for
 * vda_release_workspace.
 */
int vda_workspace_bytes(int device, size_t* bytes);

/* ------------------------------------------------------------------------- */
/* Stage interface: the same kernels as vda_forward, one step per call, with  */
/* caller-owned fp32 work buffers (all device pointers, 16-byte aligned).     */
/* ------------------------------------------------------------------------- */

/*
 * Split plans.  The frame-statistics step may split frames into token
 * ranges; each range yields one partial A and B, which the later steps add in
 * range order.  A plan (tail_frames T, splits S) splits the last T of the
 * count = H*F frames (frame index i = h*F + t) into S ranges each and leaves
 * the others whole (S == 1: no frame is split; T is then ignored).  Range s of
 * a split frame covers tokens [s*R, min(N, (s+1)*R)) with
 * R = 64 * ceil(ceil(N / S) / 64).  Partials are stored as one array of
 * count + T*(S-1) matrices (count when S == 1): matrix i holds frame i's
 * first (or only) range, and range s >= 1 of split frame i is matrix
 * i + s*T.
 */

/*
 * vda_default_split_plan -- the plan vda_forward uses on the current device
 * for these sizes and storage type (is_f32 != 0: fp32).  Whole frames occupy
 * the device in rounds; when the last round is partial its frames are split
 * (at most 4 ranges of at least 256 tokens).  Writes *tail_frames and
 * *splits.
 */
int vda_default_split_plan(int F, int N, int H, int d_k, int d_v, int is_f32,
                           int* tail_frames, int* splits);

/*
 * vda_frame_stats -- step a1, Eq. 3b, under the split plan (tail_frames,
 * splits).  For the token range of partial matrix m of frame i = h*F + t:
 *     A_part[m] = sum_u beta k k^T   (d_k x d_k, fp32)
 *     B_part[m] = sum_u beta v k^T   (d_v x d_k, fp32)
 * A_part is [P][d_k][d_k] and B_part is [P][d_v][d_k] with
 * P = H*F + tail_frames*(splits-1) (H*F when splits == 1).
 * k, v are bf16 (is_f32 == 0) or fp32 (is_f32 != 0).  With bf16 storage the
 * products beta * k are rounded to bf16 before the fp32-accumulated matrix
 * product, and only A's 16 x 16 blocks on and above the diagonal are
 * computed (the blocks below are their transposes); with fp32 storage
 * everything is fp32.  splits must not
 * exceed ceil(N / 64); with splits > 1, 1 <= tail_frames <= H*F.
 */
int vda_frame_stats(const void* k, const void* v, const float* beta,
                    int F, int N, int H, int d_k, int d_v, int tail_frames, int splits,
                    int is_f32, float* A_part, float* B_part, hipStream_t stream);

/*
 * vda_frame_inverse -- step a2, Eq. 5: Inv[i] = (I + sum of frame i's A
 * partials)^{-1} for i < count, under the split plan (tail_frames, splits)
 * that produced the partials, in fp32 by blocked Gauss-Jordan elimination
 * without pivoting (I + A is symmetric positive definite with eigenvalues
 * >= 1 when beta >= 0).  A_t is symmetric, and only its 16 x 16 blocks on
 * and below the diagonal are read (the others are taken as their transposes;
 * vda_frame_stats writes the whole matrix).  Inv is [count][d_k][d_k].  Inv may alias A_part
 * (in place onto the first count matrices); it must not overlap any other
 * partial.  When splits > 1 the call also folds the partials of B in place
 * (B_part[i] = sum of frame i's B partials; B_part as in vda_frame_stats;
 * d_v and B_part are ignored when splits == 1), so the state scan reads B_part
 * as [count][d_v][d_k].
 */
int vda_frame_inverse(const float* A_part, float* B_part, int tail_frames, int splits,
                      int count, int d_k, int d_v, float* Inv, hipStream_t stream);

/*
 * vda_state_scan -- steps a3 and a4, Eq. A.1 and Algorithm 1 step 5 with a
 * zero initial state.  With B_t = B[h][t] ([H][F][d_v][d_k] fp32, the reduced
 * frame statistic; after vda_frame_inverse it is B_part[0]):
 *     forward  P_0 = 0,     P_t = (P_{t-1} + B_t) Inv_t,  S_fwd[h][t] = P_{t-1}
 *     reverse  R_{F+1} = 0, R_t = (R_{t+1} + B_t) Inv_t,  S_rev[h][t] = R_{t+1}
 * (frames numbered 1..F here; array index t-1).  S_fwd, S_rev are
 * [H][F][d_v][d_k] fp32; Inv is [H][F][d_k][d_k] and must be symmetric (as
 * (I + A_t)^{-1} is): with is_f32 != 0 element Inv[k][j] is read from
 * Inv[j][k]; with is_f32 == 0 only the 16 x 16 blocks on and above the
 * diagonal are read and each block below is taken as the transpose of its
 * mirror.
 * The state is fp32.  is_f32 != 0: fp32 matrix products.  is_f32 == 0 (the
 * bf16 storage path): each product operand is split into two bf16 parts
 * (hi + lo) and three bf16 matrix products are accumulated in fp32, about
 * 16 mantissa bits per operand.
 */
int vda_state_scan(const float* Inv, const float* B,
                   int F, int H, int d_k, int d_v, int is_f32,
                   float* S_fwd, float* S_rev, hipStream_t stream);

/*
 * Split-bf16 operand tiles.  The bf16 storage path passes each inverse
 * Inv_t (d_k x d_k, symmetric) from step a2 to the state scan pre-split for
 * the scan's bf16 matrix products: every element x is stored as
 * hi = bf16(x) and lo = bf16(x - hi) (round-to-nearest-even), in the order
 * in which the scan's matrix instructions take them.  One frame's tiles fill
 * d_k*d_k*4 bytes (the size of the fp32 matrix): two planes (p = 0: hi,
 * p = 1: lo) of d_k*d_k bf16 values, plane p at byte p*d_k*d_k*2.  Within a
 * plane, for nb < d_k/16, ks < d_k/32, lane < 64 and e < 8, the value at
 * bf16 index ((nb*(d_k/32) + ks)*64 + lane)*8 + e is element [k][n] of
 * Inv_t with
 *     n = 16*nb + lane % 16,
 *     k = 32*ks + 4*(lane / 16) + e        for e < 4,
 *     k = 32*ks + 16 + 4*(lane / 16) + e - 4  for e >= 4.
 */

/*
 * vda_frame_inverse_tiles -- step a2 as vda_frame_inverse (same arguments,
 * checks, split plan, in-place rule and B folding), with each inverse written
 * as split-bf16 operand tiles (above) instead of an fp32 matrix.  Inv_tiles
 * is count * d_k*d_k*4 bytes.  This is the inverse vda_forward runs with
 * bf16 storage (joint rule).
 */
int vda_frame_inverse_tiles(const float* A_part, float* B_part, int tail_frames, int splits,
                            int count, int d_k, int d_v, void* Inv_tiles, hipStream_t stream);

/*
 * vda_state_scan_tiles -- steps a3 and a4 as vda_state_scan with
 * is_f32 == 0 (same recurrence, zero initial state, outputs and split-bf16
 * products with fp32 accumulation and fp32 state), reading each Inv_t from
 * split-bf16 operand tiles: Inv_tiles is [H][F] frames of d_k*d_k*4 bytes
 * (vda_frame_inverse_tiles writes them).  Element [k][n] of each tile set is
 * used as Inv_t[k][n] (no symmetry is assumed).  This is the scan
 * vda_forward runs with bf16 storage (joint rule).  Errors as
 * vda_state_scan.
 */
int vda_state_scan_tiles(const void* Inv_tiles, const float* B,
                         int F, int H, int d_k, int d_v,
                         float* S_fwd, float* S_rev, hipStream_t stream);

/*
 * vda_state_scan_chunked -- steps a3 and a4 for a chunked local window, by
 * chunk-wise scans (Sec. 4): the frames of each chunk of the window grid
 * (chunks of `chunk` >= 1 frames counted from `offset` positions before frame
 * 0, 0 <= offset < chunk, clipped to [0, F); the grid of vda_options) are
 * composed into one affine map of Eq. A.1, S_out = S_in M_c + J_c, in each
 * direction, and the chunk sequence is scanned:
 *     forward  P = S_T/2 (or 0); for chunks c in order: S_fwd[h][first(c)] = P,
 *              P = P M_c + J_c
 *     reverse  R = S_T/2 (or 0); for chunks c in reverse order:
 *              S_rev[h][last(c)] = R, R = R M_c + J_c
 * with the frame maps of vda_forward_ex (joint rule, decay alpha if not NULL;
 * Inv_tiles and B as for vda_state_scan_tiles).  These are the states the
 * windowed readout reads (Eq. A.4); all other frames of S_fwd and S_rev are
 * left untouched.  alpha [H][F][d_k] and text_state [H][d_v][d_k] (both
 * 16-byte aligned) are DEVICE pointers or NULL.  `work` is a
 * caller-owned device buffer (16-byte aligned) of
 * vda_state_scan_chunked_workspace(...) bytes for M_c (split-bf16 operand
 * tiles) and J_c (fp32).  Products are split-bf16 with fp32 accumulation.
 * Errors: VDA_ERR_SIZE for invalid chunk / offset, else as
 * vda_state_scan_tiles.  This is the scan vda_forward_ex runs with bf16
 * storage, the joint rule and window_chunk >= 2 (when the clip has at least
 * two chunks).
 */
int vda_state_scan_chunked(const void* Inv_tiles, const float* B, const float* alpha,
                           const float* text_state, int F, int H, int d_k, int d_v,
                           int chunk, int offset, void* work,
                           float* S_fwd, float* S_rev, hipStream_t stream);

/* Bytes of the work buffer of vda_state_scan_chunked (0 for invalid sizes). */
size_t vda_state_scan_chunked_workspace(int F, int H, int d_k, int d_v, int chunk, int offset);

/*
 * vda_readout -- steps a5-a7, Eq. A.4 (own-frame window), Eq. 1a and Eq. 1c:
 *     out[h][t][u] = gate[h] * RMSNorm((S_fwd[h][t] + S_rev[h][t]) q[h][t][u]).
 * q and out are bf16 (is_f32 == 0; the summed state is rounded to bf16 for
 * the fp32-accumulated matrix product) or fp32 (is_f32 != 0).
 */
int vda_readout(const void* q, const float* S_fwd, const float* S_rev,
                const float* gate, int F, int N, int H, int d_k, int d_v,
                int is_f32, void* out, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* VDA_H */
