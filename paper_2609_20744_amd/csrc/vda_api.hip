// C ABI of the VDA library: argument validation, workspace, launch order.
// Declarations and contracts are in include/vda.h.
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <atomic>
#include <mutex>
#include <vector>

#include "../../include/vda.h"
#include "vda_common.h"
#include "vda_launch.h"

namespace {

constexpr int kMaxDevices = 64;

bool supported_dim(int d) { return d == 32 || d == 64 || d == 128; }

// The whole forward also takes 16-channel heads, run as zero-padded 32-channel
// heads (the stage entry points take only the kernels' own widths).
bool forward_dim(int d) { return d == 16 || supported_dim(d); }

int padded_dim(int d) { return d < 32 ? 32 : d; }

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

struct Range {
  uintptr_t lo, hi;  // [lo, hi)
};

Range range_of(const void* p, size_t bytes) {
  const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
  return Range{lo, lo + bytes};
}

bool overlaps(Range a, Range b) { return a.lo < b.hi && b.lo < a.hi; }

// Shape checks shared by every entry point.  Grids are one-dimensional with
// one workgroup per (frame, head, split/chunk), so H*F*64 must fit 31 bits.
int check_shape(int F, int N, int H, int d_k, int d_v, bool forward = false) {
  if (F < 1 || N < 1 || H < 1) return VDA_ERR_SIZE;
  if (forward ? !(forward_dim(d_k) && forward_dim(d_v))
              : !(supported_dim(d_k) && supported_dim(d_v)))
    return VDA_ERR_UNSUPPORTED;
  if ((long long)H * F * 64 > 0x7fffffffLL) return VDA_ERR_SIZE;
  // Byte offsets within one frame of one head, and within one head's
  // per-frame matrices, are 32-bit.
  const int dmax = padded_dim(d_k > d_v ? d_k : d_v);
  if ((long long)N * dmax * 4 > 0x7fffffffLL) return VDA_ERR_SIZE;
  if ((long long)F * dmax * dmax * 4 > 0x7fffffffLL) return VDA_ERR_SIZE;
  return VDA_OK;
}

int hip_status(hipError_t e) { return e == hipSuccess ? VDA_OK : VDA_ERR_HIP; }

int current_device_cus() {
  static int cus[kMaxDevices] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
  if (cus[dev] == 0) {
    int c = 0;
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || c <= 0)
      c = 256;
    cus[dev] = c;
  }
  return cus[dev];
}

// Library-owned workspace cache per device.  Buffers come from hipMalloc
// and stay cached until vda_release_workspace or the end of the process (a
// free synchronises the device, so calls never free).  A buffer is reused by a later call on the same stream (stream
// order makes that safe) or, on another stream, once the event recorded after
// its last use has completed; between acquire and release it is marked busy
// so concurrent host threads never share it.  (Stream-ordered pool
// allocations were measured slower: a gap before every call and slower
// kernels on the pool's memory.)
struct WsEntry {
  void* ptr = nullptr;
  size_t bytes = 0;
  hipStream_t stream = nullptr;
  hipEvent_t done = nullptr;
  bool busy = false;
};

struct WsCache {
  std::mutex mu;
  std::vector<WsEntry> entries;
};

WsCache& ws_cache(int dev) {
  static WsCache caches[kMaxDevices];
  return caches[dev];
}

// Returns the entry index, or -1 (allocation failure).
int acquire_workspace(int dev, size_t bytes, hipStream_t stream) {
  WsCache& c = ws_cache(dev);
  std::lock_guard<std::mutex> lock(c.mu);
  int pick = -1;
  for (int pass = 0; pass < 2 && pick < 0; ++pass) {
    for (size_t i = 0; i < c.entries.size(); ++i) {
      WsEntry& e = c.entries[i];
      if (e.busy || e.bytes < bytes) continue;
      if (pass == 0 ? e.stream == stream : hipEventQuery(e.done) == hipSuccess) {
        pick = (int)i;
        break;
      }
    }
  }
  if (pick < 0) {
    WsEntry e;
    if (hipMalloc(&e.ptr, bytes) != hipSuccess) return -1;
    if (hipEventCreateWithFlags(&e.done, hipEventDisableTiming) != hipSuccess) {
      (void)hipFree(e.ptr);
      return -1;
    }
    e.bytes = bytes;
    // An empty slot left by vda_release_workspace is reused.
    for (size_t i = 0; i < c.entries.size() && pick < 0; ++i)
      if (!c.entries[i].ptr && !c.entries[i].busy) pick = (int)i;
    if (pick < 0) {
      c.entries.push_back(e);
      pick = (int)c.entries.size() - 1;
    } else {
      c.entries[pick] = e;
    }
  }
  c.entries[pick].busy = true;
  c.entries[pick].stream = stream;
  return pick;
}

void* workspace_ptr(int dev, int idx) {
  WsCache& c = ws_cache(dev);
  std::lock_guard<std::mutex> lock(c.mu);
  return c.entries[idx].ptr;
}

hipError_t release_workspace(int dev, int idx, hipStream_t stream) {
  WsCache& c = ws_cache(dev);
  std::lock_guard<std::mutex> lock(c.mu);
  WsEntry& e = c.entries[idx];
  const hipError_t r = hipEventRecord(e.done, stream);
  e.busy = false;
  return r;
}

// Resolves `device` (-1: the current device) for the workspace entry points.
int workspace_device(int device, int* dev) {
  if (device < -1 || device >= kMaxDevices) return VDA_ERR_SIZE;
  int count = 0;
  if (hipGetDeviceCount(&count) != hipSuccess) return VDA_ERR_HIP;
  if (device >= count) return VDA_ERR_SIZE;
  if (device == -1 && (hipGetDevice(&device) != hipSuccess || device < 0 || device >= kMaxDevices))
    return VDA_ERR_HIP;
  *dev = device;
  return VDA_OK;
}

// Frees the cached buffers of `dev` that no call holds, after the work of
// each one's last call has finished, and returns the bytes freed in *freed.
// A freed entry stays in the list as an empty slot (calls hold entries by
// index) and is reused by the next allocation.
int release_cached_workspace(int dev, size_t* freed) {
  WsCache& c = ws_cache(dev);
  std::lock_guard<std::mutex> lock(c.mu);
  int cur = 0;
  if (hipGetDevice(&cur) != hipSuccess) return VDA_ERR_HIP;
  if (cur != dev && hipSetDevice(dev) != hipSuccess) return VDA_ERR_HIP;
  int st = VDA_OK;
  size_t bytes = 0;
  for (WsEntry& e : c.entries) {
    if (e.busy || !e.ptr) continue;
    if (hipEventSynchronize(e.done) != hipSuccess || hipFree(e.ptr) != hipSuccess) {
      st = VDA_ERR_HIP;
      break;
    }
    (void)hipEventDestroy(e.done);
    bytes += e.bytes;
    e = WsEntry();
  }
  if (cur != dev && hipSetDevice(cur) != hipSuccess && st == VDA_OK) st = VDA_ERR_HIP;
  if (freed) *freed = bytes;
  return st;
}

size_t cached_workspace_bytes(int dev) {
  WsCache& c = ws_cache(dev);
  std::lock_guard<std::mutex> lock(c.mu);
  size_t bytes = 0;
  for (const WsEntry& e : c.entries) bytes += e.bytes;
  return bytes;
}

// Workgroups of the statistics kernel one compute unit holds at once, per
// device, storage type and head dimensions (cached; 0 = not yet known).
int stats_blocks_per_cu(int dev, bool is_f32, int d_k, int d_v) {
  static std::atomic<int> cache[kMaxDevices][2][3][3];
  auto idx = [](int d) { return d == 32 ? 0 : d == 64 ? 1 : 2; };
  std::atomic<int>& c = cache[dev][is_f32 ? 1 : 0][idx(d_k)][idx(d_v)];
  int n = c.load(std::memory_order_relaxed);
  if (n == 0) {
    n = vda::stats_blocks_per_cu(is_f32, d_k, d_v);
    if (n < 1) n = 1;
    c.store(n, std::memory_order_relaxed);
  }
  return n;
}

// Split plan of the statistics step.  Whole frames fill the device in
// rounds of (resident workgroups) frames; when the last round is partial,
// its frames are split into up to four token ranges (at least 256 tokens
// each) so that the end of the launch keeps more compute units streaming.
// Each extra range costs one partial A_t, B_t written here and read back by
// the inverse step, which is why the split is kept small and limited to
// the partial round.
vda::SplitPlan default_plan(int dev, int F, int N, int H, int d_k, int d_v, bool is_f32) {
  constexpr int kMaxSplits = 4;
  const long long count = (long long)H * F;
  const long long slots = (long long)stats_blocks_per_cu(dev, is_f32, d_k, d_v) * current_device_cus();
  const long long rem = count % slots;
  if (rem == 0) return vda::SplitPlan{0, 1};
  long long k = slots / rem;
  if (k > kMaxSplits) k = kMaxSplits;
  if (k > N / 256) k = N / 256;
  if (k < 2) return vda::SplitPlan{0, 1};
  return vda::SplitPlan{(int)rem, (int)k};
}

struct Workspace {
  size_t a_part, b_part, s_fwd, s_rev, total;  // byte offsets / total
};

Workspace workspace_layout(int F, int H, int d_k, int d_v, vda::SplitPlan plan) {
  const size_t fh = (size_t)H * F;
  const size_t parts = (size_t)vda::partial_count((long long)fh, plan);
  const size_t a = parts * d_k * d_k * sizeof(float);
  const size_t b = parts * d_v * d_k * sizeof(float);
  const size_t s = fh * d_v * d_k * sizeof(float);
  Workspace w;
  w.a_part = 0;
  w.b_part = a;
  w.s_fwd = a + b;
  w.s_rev = a + b + s;
  w.total = a + b + 2 * s;
  return w;
}

// Whether the chunk-wise scans beat the frame-by-frame scan for a chunked
// window, by a cost model fitted per key width to measurements on MI355X
// (both scans alone, d_v = d_k, chunks of five after one anchor, at 16 heads
// x 36 frames and 7 heads x 100 frames).  The frame scan costs about
// a * F + b us; the chunk-wise scans s * (5 * chunk + 13) us per round of
// 2 * H * C compose workgroups over the compute units plus g us per chunk.
//   d_k = 128: frame 43.4 / 97.6 us, chunk-wise 56.6 / 90.1 us
//   d_k =  64: frame 18.5 / 46.4 us, chunk-wise 15.1 / 24.3 us
//   d_k =  32: frame 13.6 / 33.7 us, chunk-wise 10.8 / 14.5 us
bool chunked_scan_pays(int F, int H, int d_k, int chunk, int offset) {
  const int C = vda::chunk_count(F, chunk, offset);
  if (C < 2) return false;
  struct Fit { double a, b, s, g; };
  const Fit fit = d_k >= 128 ? Fit{0.847, 12.9, 1.042, 2.12}
                  : d_k >= 64 ? Fit{0.436, 2.8, 0.274, 0.587}
                              : Fit{0.314, 2.3, 0.247, 0.176};
  const double rounds = std::max(1.0, 2.0 * H * C / (double)current_device_cus());
  const double chunked_us = rounds * fit.s * (5.0 * chunk + 13.0) + fit.g * C;
  const double frame_us = fit.a * F + fit.b;
  return chunked_us < frame_us;
}

// Options of the full operator, validated into *out; a null vda_options is
// the core operator.
int check_options(const vda_options* o, vda_options* out) {
  vda_options d;
  d.rule = VDA_RULE_JOINT;
  d.alpha = nullptr;
  d.text_state = nullptr;
  d.window_chunk = 1;
  d.window_radius = 0;
  d.window_offset = 0;
  d.gate_tokens = nullptr;
  d.out_heads = 0;
  d.q_heads = 0;
  if (o) d = *o;
  if (d.rule != VDA_RULE_JOINT && d.rule != VDA_RULE_FROZEN_SCALED) return VDA_ERR_UNSUPPORTED;
  if (d.window_chunk < 1 || d.window_radius < 0 || d.window_offset < 0 ||
      d.window_offset >= d.window_chunk || d.out_heads < 0 || d.q_heads < 0)
    return VDA_ERR_SIZE;
  if (!aligned(d.alpha, 16) || !aligned(d.text_state, 16) || !aligned(d.gate_tokens, 16))
    return VDA_ERR_ALIGN;
  *out = d;
  return VDA_OK;
}

// Everything a forward call decides on the host before it launches: the
// validated arguments, the padded widths, the split plan, the scan path and
// the workspace layout (offsets from the workspace base).
struct ForwardCall {
  bool is_f32 = false, frozen = false, chunked = false, tiled = false;
  const void *q = nullptr, *k = nullptr, *v = nullptr;
  const float *beta = nullptr, *gate = nullptr;
  int F = 0, N = 0, H = 0, d_k = 0, d_v = 0, pk = 0, pv = 0;
  vda_options o;
  void* out = nullptr;
  size_t es = 0, tok = 0;
  vda::SplitPlan plan{0, 1};
  Workspace w;
  size_t qk_pad = 0, v_pad = 0, a_pad = 0, t_pad = 0, t_tmp = 0, g_pad = 0, c_ws = 0;
  size_t ws_bytes = 0;
};

// Every argument check of a forward call, on the host, before anything is
// enqueued; the validated options go to *o.
int check_forward(bool is_f32, const void* q, const void* k, const void* v, const float* beta,
                  const float* gate, int F, int N, int H, int d_k, int d_v,
                  const vda_options* opts, const void* out, vda_options* o_out) {
  if (!q || !k || !v || !beta || !out) return VDA_ERR_NULL;
  int st = check_shape(F, N, H, d_k, d_v, true);
  if (st != VDA_OK) return st;
  vda_options o;
  st = check_options(opts, &o);
  if (st != VDA_OK) return st;
  // The per-head gate may be absent only when the output gate per token
  // replaces it.
  if (!gate && !o.gate_tokens) return VDA_ERR_NULL;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
      !aligned(beta, 4) || !aligned(gate, 4))
    return VDA_ERR_ALIGN;
  // The window arithmetic stays within 32 bits.
  if ((long long)F + 2LL * (o.window_radius + 1) * o.window_chunk > 0x3fffffffLL) return VDA_ERR_SIZE;
  // A token-major output holds whole clips of out_heads heads, and one
  // frame's rows of it stay within 32-bit byte offsets.
  if (o.out_heads > 0 &&
      (H % o.out_heads != 0 ||
       (long long)(N + 64) * o.out_heads * d_v * (is_f32 ? 4 : 2) > 0x7fffffffLL))
    return VDA_ERR_SIZE;
  // A raw token-major query: whole clips, 32-bit row offsets, and the
  // kernels' own key widths (no padded copy of it is made).
  if (o.q_heads > 0) {
    if (H % o.q_heads != 0 ||
        (long long)(N + 64) * o.q_heads * d_k * (is_f32 ? 4 : 2) > 0x7fffffffLL)
      return VDA_ERR_SIZE;
    if (padded_dim(d_k) != d_k) return VDA_ERR_UNSUPPORTED;
  }
  const size_t es = is_f32 ? 4 : 2;
  const size_t tok = (size_t)H * F * N;
  const Range ro = range_of(out, tok * d_v * es);
  if (overlaps(ro, range_of(q, tok * d_k * es)) || overlaps(ro, range_of(k, tok * d_k * es)) ||
      overlaps(ro, range_of(v, tok * d_v * es)) || overlaps(ro, range_of(beta, tok * 4)) ||
      (gate && overlaps(ro, range_of(gate, (size_t)H * 4))) ||
      (o.gate_tokens && overlaps(ro, range_of(o.gate_tokens, tok * d_v * es))) ||
      (o.alpha && overlaps(ro, range_of(o.alpha, (size_t)H * F * d_k * 4))) ||
      (o.text_state && overlaps(ro, range_of(o.text_state, (size_t)H * d_v * d_k * 4))))
    return VDA_ERR_OVERLAP;
  *o_out = o;
  return VDA_OK;
}

// Lays out a checked forward call on device `dev`.
void plan_forward(bool is_f32, const void* q, const void* k, const void* v, const float* beta,
                  const float* gate, int F, int N, int H, int d_k, int d_v,
                  const vda_options& o, void* out, int dev, ForwardCall* c) {
  const size_t es = is_f32 ? 4 : 2;
  const size_t tok = (size_t)H * F * N;
  ForwardCall& C = *c;
  C = ForwardCall();
  C.is_f32 = is_f32;
  C.frozen = o.rule == VDA_RULE_FROZEN_SCALED;
  C.q = q, C.k = k, C.v = v, C.beta = beta, C.gate = gate, C.out = out, C.o = o;
  C.F = F, C.N = N, C.H = H, C.d_k = d_k, C.d_v = d_v;
  C.es = es, C.tok = tok;
  // Heads narrower than 32 channels run as zero-padded 32-channel heads; the
  // padded q, k, v, output, alpha and text state live after the state buffers.
  const int pk = padded_dim(d_k), pv = padded_dim(d_v);
  C.pk = pk, C.pv = pv;
  // The fp32 frozen rule's scan reads the statistics directly, so its frames
  // are not split; the bf16 frozen rule's map tiles sum the partials.
  C.plan = C.frozen && is_f32 ? vda::SplitPlan{0, 1} : default_plan(dev, F, N, H, pk, pv, is_f32);
  C.w = workspace_layout(F, H, pk, pv, C.plan);
  // With a chunked local window (bf16 storage, joint rule) the readout reads
  // the states at chunk boundaries only: chunk-wise scans compute just those,
  // where they are the faster path.
  C.chunked = !is_f32 && !C.frozen && o.window_chunk >= 2 &&
              chunked_scan_pays(F, H, pk, o.window_chunk, o.window_offset);
  C.tiled = !is_f32 && !C.frozen;
  C.c_ws = C.chunked ? round_up(vda::chunked_scan_workspace(F, H, pk, pv, o.window_chunk,
                                                            o.window_offset),
                                256)
                     : 0;
  C.qk_pad = pk != d_k ? round_up(tok * pk * es, 256) : 0;  // (never with a raw query)
  C.v_pad = pv != d_v ? round_up(tok * pv * es, 256) : 0;
  const bool pad_any = pk != d_k || pv != d_v;
  C.a_pad = pk != d_k && o.alpha ? round_up((size_t)H * F * pk * 4, 256) : 0;
  C.t_pad = pad_any && o.text_state ? round_up((size_t)H * pv * pk * 4, 256) : 0;
  C.t_tmp = pad_any && o.text_state ? round_up((size_t)H * d_v * pk * 4, 256) : 0;
  C.g_pad = o.gate_tokens && pv != d_v ? round_up(tok * pv * es, 256) : 0;
  C.ws_bytes = round_up(C.w.total, 256) + 2 * C.qk_pad + C.v_pad + C.a_pad + C.t_pad +
               C.t_tmp + C.g_pad + C.c_ws;
}

// Enqueues a planned forward call with its workspace at `base` (at least
// C.ws_bytes bytes, 256-byte aligned).
hipError_t launch_forward(const ForwardCall& C, char* base, hipStream_t stream) {
  const vda_options& o = C.o;
  const int F = C.F, N = C.N, H = C.H, d_k = C.d_k, d_v = C.d_v, pk = C.pk, pv = C.pv;
  const size_t es = C.es, tok = C.tok;
  float* A_part = reinterpret_cast<float*>(base + C.w.a_part);
  float* B_part = reinterpret_cast<float*>(base + C.w.b_part);
  float* S_fwd = reinterpret_cast<float*>(base + C.w.s_fwd);
  float* S_rev = reinterpret_cast<float*>(base + C.w.s_rev);
  float* Inv = A_part;  // the inverse overwrites the first partial
  char* pad_base = base + round_up(C.w.total, 256);
  const void* qx = C.q;
  const void* kx = C.k;
  const void* vx = C.v;

  const float* alpha_x = o.alpha;
  const float* ts_x = o.text_state;

  hipError_t e = hipSuccess;
  if (C.qk_pad) {
    void* qp = pad_base;
    void* kp = pad_base + C.qk_pad;
    e = vda::launch_pad_rows(C.q, qp, (long long)tok, (int)(d_k * es), (int)(pk * es), stream);
    if (e == hipSuccess)
      e = vda::launch_pad_rows(C.k, kp, (long long)tok, (int)(d_k * es), (int)(pk * es), stream);
    qx = qp;
    kx = kp;
  }
  if (C.v_pad && e == hipSuccess) {
    void* vp = pad_base + 2 * C.qk_pad;
    e = vda::launch_pad_rows(C.v, vp, (long long)tok, (int)(d_v * es), (int)(pv * es), stream);
    vx = vp;
  }
  char* opt_base = pad_base + 2 * C.qk_pad + C.v_pad;
  void* chunk_work = opt_base + C.a_pad + C.t_pad + C.t_tmp + C.g_pad;
  const void* gt_x = o.gate_tokens;
  if (C.g_pad && e == hipSuccess) {  // output gates [tok][d_v] -> [tok][32], zero channels added
    void* gp = opt_base + C.a_pad + C.t_pad + C.t_tmp;
    e = vda::launch_pad_rows(o.gate_tokens, gp, (long long)tok, (int)(d_v * es), (int)(pv * es),
                             stream);
    gt_x = gp;
  }
  if (C.a_pad && e == hipSuccess) {  // alpha [H][F][d_k] -> [H][F][32]
    float* ap = reinterpret_cast<float*>(opt_base);
    e = vda::launch_pad_rows(o.alpha, ap, (long long)H * F, d_k * 4, pk * 4, stream);
    alpha_x = ap;
  }
  if (C.t_pad && e == hipSuccess) {  // S_T [H][d_v][d_k] -> [H][d_v][pk] -> [H][pv][pk]
    float* tt = reinterpret_cast<float*>(opt_base + C.a_pad);
    float* tp = reinterpret_cast<float*>(opt_base + C.a_pad + C.t_tmp);
    e = vda::launch_pad_rows(o.text_state, tt, (long long)H * d_v, d_k * 4, pk * 4, stream);
    if (e == hipSuccess)
      e = vda::launch_pad_rows(tt, tp, (long long)H, d_v * pk * 4, pv * pk * 4, stream);
    ts_x = tp;
  }
  if (e == hipSuccess)
    e = vda::launch_frame_stats(C.is_f32, kx, vx, C.beta, F, N, H, pk, pv, C.plan, A_part, B_part,
                                stream, /*lower_only=*/!C.frozen);
  // With bf16 storage the joint rule's inverse is written as split-bf16
  // operand tiles for the state scan.
  if (e == hipSuccess && !C.frozen)
    e = vda::launch_frame_inverse(A_part, B_part, C.plan, (long long)H * F, pk, pv, C.tiled, Inv,
                                  stream);
  vda::ScanOptions so;
  so.frozen = C.frozen;
  so.alpha = alpha_x;
  so.text_state = ts_x;
  so.tokens = N;
  if (e == hipSuccess) {
    if (C.frozen && !C.is_f32) {
      // bf16 storage: the frozen maps as operand tiles (in place over A_t),
      // then the tiled scan in its map form.
      e = vda::launch_frozen_tiles(A_part, B_part, C.plan, alpha_x, F, H, pk, pv, N, stream);
      if (e == hipSuccess)
        e = vda::launch_frozen_scan_tiled(A_part, B_part, ts_x, F, H, pk, pv, N, S_fwd, S_rev,
                                          stream);
    } else if (C.chunked)
      e = vda::launch_state_scan_chunked(Inv, B_part, alpha_x, ts_x, F, H, pk, pv, o.window_chunk,
                                         o.window_offset, chunk_work, S_fwd, S_rev, stream);
    else if (C.tiled)
      e = vda::launch_state_scan_tiled(Inv, B_part, F, H, pk, pv, so, S_fwd, S_rev, stream);
    else
      e = vda::launch_state_scan(C.is_f32, C.frozen ? A_part : Inv, B_part, F, H, pk, pv, so,
                                 S_fwd, S_rev, stream);
  }
  vda::GatherOptions go;
  go.alpha = alpha_x;
  go.chunk = o.window_chunk;
  go.radius = o.window_radius;
  go.offset = o.window_offset;
  go.gate_tokens = gt_x;
  go.out_heads = o.out_heads > 0 ? o.out_heads : 1;
  go.q_heads = o.q_heads > 0 ? o.q_heads : 1;
  go.q_l2 = o.q_heads > 0;
  // The readout writes the true d_v channels of each head straight into out
  // (a padded head's zero channels are not stored).
  if (e == hipSuccess)
    e = vda::launch_readout(C.is_f32, qx, S_fwd, S_rev, C.gate, F, N, H, pk, pv, d_v, go, C.out,
                            stream);
  return e;
}

int forward_impl(bool is_f32, const void* q, const void* k, const void* v, const float* beta,
                 const float* gate, int F, int N, int H, int d_k, int d_v,
                 const vda_options* opts, void* out, hipStream_t stream) {
  vda_options o;
  const int st = check_forward(is_f32, q, k, v, beta, gate, F, N, H, d_k, d_v, opts, out, &o);
  if (st != VDA_OK) return st;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return VDA_ERR_HIP;
  ForwardCall C;
  plan_forward(is_f32, q, k, v, beta, gate, F, N, H, d_k, d_v, o, out, dev, &C);
  const int wsi = acquire_workspace(dev, C.ws_bytes, stream);
  if (wsi < 0) return VDA_ERR_NOMEM;
  const hipError_t e = launch_forward(C, static_cast<char*>(workspace_ptr(dev, wsi)), stream);
  const hipError_t ef = release_workspace(dev, wsi, stream);
  if (e != hipSuccess) return VDA_ERR_HIP;
  return hip_status(ef);
}

// Fixed device scratch of vda_forward_noalloc: the code object holds it on
// every device the library runs on, until the process ends.  Host code never
// passes this name to a kernel (on the host it is only a stand-in for the
// device array); it uses the address that hipGetSymbolAddress returns for
// the current device.
static __device__ __align__(256) unsigned char scratch[VDA_NOALLOC_SCRATCH_BYTES];

// Device address of `scratch` on device `dev` (the current device), looked up
// once per device; nullptr if the runtime cannot resolve it.
char* scratch_ptr(int dev) {
  static std::mutex mu;
  static char* ptrs[kMaxDevices] = {};
  std::lock_guard<std::mutex> lock(mu);
  if (!ptrs[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    ptrs[dev] = static_cast<char*>(p);
  }
  return ptrs[dev];
}

// Workspace bytes of vda_forward over `heads` heads starting at head h0.
size_t group_workspace(const void* q, const void* k, const void* v, const float* beta,
                       const float* gate, int F, int N, int h0, int heads, int d_k, int d_v,
                       const vda_options& o, void* out, int dev) {
  const size_t tokh = (size_t)F * N;  // tokens per head
  ForwardCall C;
  plan_forward(false, static_cast<const char*>(q) + h0 * tokh * d_k * 2,
               static_cast<const char*>(k) + h0 * tokh * d_k * 2,
               static_cast<const char*>(v) + h0 * tokh * d_v * 2, beta + h0 * tokh, gate + h0, F,
               N, heads, d_k, d_v, o, static_cast<char*>(out) + h0 * tokh * d_v * 2, dev, &C);
  return C.ws_bytes;
}

// vda_forward with its workspace in `scratch`: the heads run in consecutive
// groups, each as one forward over its heads, as many heads per group as fit.
int forward_noalloc_impl(const void* q, const void* k, const void* v, const float* beta,
                         const float* gate, int F, int N, int H, int d_k, int d_v, void* out,
                         hipStream_t stream) {
  vda_options o;
  int st = check_forward(false, q, k, v, beta, gate, F, N, H, d_k, d_v, nullptr, out, &o);
  if (st != VDA_OK) return st;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return VDA_ERR_HIP;
  char* base = scratch_ptr(dev);
  if (!base) return VDA_ERR_HIP;
  constexpr size_t cap = VDA_NOALLOC_SCRATCH_BYTES;
  auto fits = [&](int h0, int n) {
    return group_workspace(q, k, v, beta, gate, F, N, h0, n, d_k, d_v, o, out, dev) <= cap;
  };
  // Nothing is enqueued unless every head fits on its own.
  if (!fits(0, 1)) return VDA_ERR_SCRATCH;
  // Largest group size that fits, by bisection on the workspace of a group
  // at the first head (the workspace grows with the heads up to the
  // statistics' split partials; each group is re-checked below).
  int g = H;
  if (!fits(0, H)) {
    int lo = 1, hi = H;  // fits(lo), !fits(hi)
    while (hi - lo > 1) {
      const int mid = lo + (hi - lo) / 2;
      if (fits(0, mid)) lo = mid;
      else hi = mid;
    }
    g = lo;
  }
  const size_t tokh = (size_t)F * N;
  for (int h0 = 0; h0 < H;) {
    int n = std::min(g, H - h0);
    while (n > 1 && !fits(h0, n)) --n;
    ForwardCall C;
    plan_forward(false, static_cast<const char*>(q) + h0 * tokh * d_k * 2,
                 static_cast<const char*>(k) + h0 * tokh * d_k * 2,
                 static_cast<const char*>(v) + h0 * tokh * d_v * 2, beta + h0 * tokh, gate + h0,
                 F, N, n, d_k, d_v, o, static_cast<char*>(out) + h0 * tokh * d_v * 2, dev, &C);
    if (C.ws_bytes > cap) return VDA_ERR_SCRATCH;  // cannot happen: one head fits
    if (launch_forward(C, base, stream) != hipSuccess) return VDA_ERR_HIP;
    h0 += n;
  }
  return VDA_OK;
}

// The prompt state: one frame of L tokens per head from the zero state.
int text_state_impl(const void* k, const void* v, const float* beta, int L, int H, int d_k,
                    int d_v, int rule, int is_f32, float* S_T, hipStream_t stream) {
  if (!k || !v || !beta || !S_T) return VDA_ERR_NULL;
  int st = check_shape(1, L, H, d_k, d_v, true);
  if (st != VDA_OK) return st;
  if (rule != VDA_RULE_JOINT && rule != VDA_RULE_FROZEN_SCALED) return VDA_ERR_UNSUPPORTED;
  if (!aligned(k, 16) || !aligned(v, 16) || !aligned(beta, 4) || !aligned(S_T, 16))
    return VDA_ERR_ALIGN;
  const size_t es = is_f32 ? 4 : 2;
  const size_t tok = (size_t)H * L;
  const Range rs = range_of(S_T, (size_t)H * d_v * d_k * 4);
  if (overlaps(rs, range_of(k, tok * d_k * es)) || overlaps(rs, range_of(v, tok * d_v * es)) ||
      overlaps(rs, range_of(beta, tok * 4)))
    return VDA_ERR_OVERLAP;
  const bool frozen = rule == VDA_RULE_FROZEN_SCALED;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return VDA_ERR_HIP;
  const int pk = padded_dim(d_k), pv = padded_dim(d_v);
  // The frozen rule reads B directly, so its frame is not split; the joint
  // rule's inverse folds the partials of a split frame.
  const vda::SplitPlan plan =
      frozen ? vda::SplitPlan{0, 1} : default_plan(dev, 1, L, H, pk, pv, is_f32 != 0);
  const Workspace w = workspace_layout(1, H, pk, pv, plan);
  const size_t k_pad = pk != d_k ? round_up(tok * pk * es, 256) : 0;
  const size_t v_pad = pv != d_v ? round_up(tok * pv * es, 256) : 0;
  const size_t stats_bytes = round_up(w.s_fwd, 256);  // the A and B partials
  const int wsi = acquire_workspace(dev, stats_bytes + k_pad + v_pad, stream);
  if (wsi < 0) return VDA_ERR_NOMEM;
  char* base = static_cast<char*>(workspace_ptr(dev, wsi));
  float* A_part = reinterpret_cast<float*>(base + w.a_part);
  float* B_part = reinterpret_cast<float*>(base + w.b_part);
  char* pad_base = base + stats_bytes;
  const void* kx = k;
  const void* vx = v;
  hipError_t e = hipSuccess;
  if (k_pad) {
    e = vda::launch_pad_rows(k, pad_base, (long long)tok, (int)(d_k * es), (int)(pk * es), stream);
    kx = pad_base;
  }
  if (v_pad && e == hipSuccess) {
    e = vda::launch_pad_rows(v, pad_base + k_pad, (long long)tok, (int)(d_v * es), (int)(pv * es),
                             stream);
    vx = pad_base + k_pad;
  }
  if (e == hipSuccess)
    e = vda::launch_frame_stats(is_f32 != 0, kx, vx, beta, 1, L, H, pk, pv, plan, A_part, B_part,
                                stream);
  if (e == hipSuccess && !frozen)
    e = vda::launch_frame_inverse(A_part, B_part, plan, H, pk, pv, false, A_part, stream);
  if (e == hipSuccess)
    e = vda::launch_text_state(B_part, frozen ? nullptr : A_part, H, pk, pv, d_k, d_v,
                               (float)(1.0 / std::sqrt((double)L)), S_T, stream);
  const hipError_t ef = release_workspace(dev, wsi, stream);
  if (e != hipSuccess) return VDA_ERR_HIP;
  return hip_status(ef);
}

}  // namespace

extern "C" {

const char* vda_status_string(int status) {
  switch (status) {
    case VDA_OK: return "VDA_OK";
    case VDA_ERR_NULL: return "VDA_ERR_NULL: a required pointer is NULL";
    case VDA_ERR_SIZE: return "VDA_ERR_SIZE: a size is out of range";
    case VDA_ERR_UNSUPPORTED:
      return "VDA_ERR_UNSUPPORTED: d_k and d_v must be 32, 64 or 128 (16 too for the forward)";
    case VDA_ERR_ALIGN: return "VDA_ERR_ALIGN: a pointer is misaligned";
    case VDA_ERR_OVERLAP: return "VDA_ERR_OVERLAP: the output overlaps an input";
    case VDA_ERR_HIP: return "VDA_ERR_HIP: the HIP runtime reported an error";
    case VDA_ERR_NOMEM: return "VDA_ERR_NOMEM: workspace allocation failed";
    case VDA_ERR_SCRATCH:
      return "VDA_ERR_SCRATCH: one head needs more workspace than the fixed scratch array holds";
    default: return "VDA: unknown status";
  }
}

int vda_forward(const void* q, const void* k, const void* v, const float* beta, const float* gate,
                int F, int N, int H, int d_k, int d_v, void* out, hipStream_t stream) {
  return forward_impl(false, q, k, v, beta, gate, F, N, H, d_k, d_v, nullptr, out, stream);
}

int vda_forward_noalloc(const void* q, const void* k, const void* v, const float* beta,
                        const float* gate, int F, int N, int H, int d_k, int d_v, void* out,
                        hipStream_t stream) {
  return forward_noalloc_impl(q, k, v, beta, gate, F, N, H, d_k, d_v, out, stream);
}

int vda_forward_f32(const float* q, const float* k, const float* v, const float* beta,
                    const float* gate, int F, int N, int H, int d_k, int d_v, float* out,
                    hipStream_t stream) {
  return forward_impl(true, q, k, v, beta, gate, F, N, H, d_k, d_v, nullptr, out, stream);
}

int vda_forward_ex(const void* q, const void* k, const void* v, const float* beta,
                   const float* gate, int F, int N, int H, int d_k, int d_v,
                   const vda_options* opts, void* out, hipStream_t stream) {
  return forward_impl(false, q, k, v, beta, gate, F, N, H, d_k, d_v, opts, out, stream);
}

int vda_forward_ex_f32(const float* q, const float* k, const float* v, const float* beta,
                       const float* gate, int F, int N, int H, int d_k, int d_v,
                       const vda_options* opts, float* out, hipStream_t stream) {
  return forward_impl(true, q, k, v, beta, gate, F, N, H, d_k, d_v, opts, out, stream);
}

int vda_text_state(const void* k, const void* v, const float* beta, int L, int H, int d_k,
                   int d_v, int rule, int is_f32, float* S_T, hipStream_t stream) {
  return text_state_impl(k, v, beta, L, H, d_k, d_v, rule, is_f32, S_T, stream);
}

int vda_release_workspace(int device, size_t* bytes_freed) {
  if (bytes_freed) *bytes_freed = 0;
  int dev = 0;
  const int st = workspace_device(device, &dev);
  if (st != VDA_OK) return st;
  return release_cached_workspace(dev, bytes_freed);
}

int vda_workspace_bytes(int device, size_t* bytes) {
  if (!bytes) return VDA_ERR_NULL;
  *bytes = 0;
  int dev = 0;
  const int st = workspace_device(device, &dev);
  if (st != VDA_OK) return st;
  *bytes = cached_workspace_bytes(dev);
  return VDA_OK;
}

int vda_default_split_plan(int F, int N, int H, int d_k, int d_v, int is_f32, int* tail_frames,
                           int* splits) {
  if (!tail_frames || !splits) return VDA_ERR_NULL;
  int st = check_shape(F, N, H, d_k, d_v);
  if (st != VDA_OK) return st;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return VDA_ERR_HIP;
  const vda::SplitPlan p = default_plan(dev, F, N, H, d_k, d_v, is_f32 != 0);
  *tail_frames = p.tail;
  *splits = p.splits;
  return VDA_OK;
}

}  // extern "C"

namespace {

// Shared checks of a split plan over `count` frames of N tokens.
int check_plan(long long count, int N, int tail_frames, int splits) {
  if (splits < 1) return VDA_ERR_SIZE;
  if (splits == 1) return VDA_OK;  // no frame is split; tail_frames is ignored
  if (tail_frames < 1 || tail_frames > count || splits > ((long long)N + 63) / 64)
    return VDA_ERR_SIZE;
  const vda::SplitPlan p{tail_frames, splits};
  if (vda::stats_workgroups(count, p) > 0x7fffffffLL) return VDA_ERR_SIZE;
  return VDA_OK;
}

}  // namespace

extern "C" {

int vda_frame_stats(const void* k, const void* v, const float* beta, int F, int N, int H,
                    int d_k, int d_v, int tail_frames, int splits, int is_f32, float* A_part,
                    float* B_part, hipStream_t stream) {
  if (!k || !v || !beta || !A_part || !B_part) return VDA_ERR_NULL;
  int st = check_shape(F, N, H, d_k, d_v);
  if (st != VDA_OK) return st;
  const size_t fh = (size_t)H * F;
  st = check_plan((long long)fh, N, tail_frames, splits);
  if (st != VDA_OK) return st;
  if (!aligned(k, 16) || !aligned(v, 16) || !aligned(beta, 4) || !aligned(A_part, 16) ||
      !aligned(B_part, 16))
    return VDA_ERR_ALIGN;
  const vda::SplitPlan plan{splits > 1 ? tail_frames : 0, splits};
  const size_t parts = (size_t)vda::partial_count((long long)fh, plan);
  const Range ra = range_of(A_part, parts * d_k * d_k * 4);
  const Range rb = range_of(B_part, parts * d_v * d_k * 4);
  const size_t es = is_f32 ? 4 : 2;
  const Range rk = range_of(k, fh * N * d_k * es), rv = range_of(v, fh * N * d_v * es),
              rbeta = range_of(beta, fh * N * 4);
  if (overlaps(ra, rb) || overlaps(ra, rk) || overlaps(ra, rv) || overlaps(ra, rbeta) ||
      overlaps(rb, rk) || overlaps(rb, rv) || overlaps(rb, rbeta))
    return VDA_ERR_OVERLAP;
  return hip_status(vda::launch_frame_stats(is_f32 != 0, k, v, beta, F, N, H, d_k, d_v, plan,
                                            A_part, B_part, stream));
}

}  // extern "C"

namespace {

int frame_inverse(const float* A_part, float* B_part, int tail_frames, int splits, int count,
                  int d_k, int d_v, bool tiled, float* Inv, hipStream_t stream) {
  if (!A_part || !Inv || (splits > 1 && !B_part)) return VDA_ERR_NULL;
  if (count < 1 || (long long)count * 64 > 0x7fffffffLL) return VDA_ERR_SIZE;
  // N is not known here; any split count the statistics step accepted is fine.
  int st = check_plan(count, 0x7fffffff, tail_frames, splits);
  if (st != VDA_OK) return st;
  if (!supported_dim(d_k) || (splits > 1 && !supported_dim(d_v))) return VDA_ERR_UNSUPPORTED;
  if (!aligned(A_part, 16) || !aligned(Inv, 16) || !aligned(B_part, 16)) return VDA_ERR_ALIGN;
  const vda::SplitPlan plan{splits > 1 ? tail_frames : 0, splits};
  const size_t mat = (size_t)d_k * d_k * 4;
  const size_t parts = (size_t)vda::partial_count(count, plan);
  // Inv may be the first `count` partials (in place), but no other partial.
  const Range ri = range_of(Inv, count * mat);
  const Range ra = range_of(A_part, parts * mat);
  const Range rextra = range_of(reinterpret_cast<const char*>(A_part) + count * mat,
                                (parts - count) * mat);
  if (overlaps(ri, ra) && (ri.lo != ra.lo || overlaps(ri, rextra))) return VDA_ERR_OVERLAP;
  if (splits > 1) {
    const Range rb = range_of(B_part, parts * d_v * d_k * 4);
    if (overlaps(rb, ri) || overlaps(rb, ra)) return VDA_ERR_OVERLAP;
  }
  return hip_status(
      vda::launch_frame_inverse(A_part, B_part, plan, count, d_k, d_v, tiled, Inv, stream));
}

// Checks of the state-scan stage entry points (matrix operand of d_k*d_k*4
// bytes per frame in either layout).
int check_scan(const void* Inv, const float* B, int F, int H, int d_k, int d_v, float* S_fwd,
               float* S_rev) {
  if (!Inv || !B || !S_fwd || !S_rev) return VDA_ERR_NULL;
  int st = check_shape(F, 1, H, d_k, d_v);
  if (st != VDA_OK) return st;
  if (!aligned(Inv, 16) || !aligned(B, 16) || !aligned(S_fwd, 16) || !aligned(S_rev, 16))
    return VDA_ERR_ALIGN;
  const size_t fh = (size_t)H * F;
  const Range rf = range_of(S_fwd, fh * d_v * d_k * 4), rr = range_of(S_rev, fh * d_v * d_k * 4);
  const Range ri = range_of(Inv, fh * d_k * d_k * 4);
  const Range rb = range_of(B, fh * d_v * d_k * 4);
  if (overlaps(rf, rr) || overlaps(rf, ri) || overlaps(rf, rb) || overlaps(rr, ri) ||
      overlaps(rr, rb))
    return VDA_ERR_OVERLAP;
  return VDA_OK;
}

}  // namespace

extern "C" {

int vda_frame_inverse(const float* A_part, float* B_part, int tail_frames, int splits, int count,
                      int d_k, int d_v, float* Inv, hipStream_t stream) {
  return frame_inverse(A_part, B_part, tail_frames, splits, count, d_k, d_v, false, Inv, stream);
}

int vda_frame_inverse_tiles(const float* A_part, float* B_part, int tail_frames, int splits,
                            int count, int d_k, int d_v, void* Inv_tiles, hipStream_t stream) {
  return frame_inverse(A_part, B_part, tail_frames, splits, count, d_k, d_v, true,
                       static_cast<float*>(Inv_tiles), stream);
}

int vda_state_scan(const float* Inv, const float* B, int F, int H, int d_k, int d_v, int is_f32,
                   float* S_fwd, float* S_rev, hipStream_t stream) {
  const int st = check_scan(Inv, B, F, H, d_k, d_v, S_fwd, S_rev);
  if (st != VDA_OK) return st;
  return hip_status(vda::launch_state_scan(is_f32 != 0, Inv, B, F, H, d_k, d_v, vda::ScanOptions(),
                                           S_fwd, S_rev, stream));
}

size_t vda_state_scan_chunked_workspace(int F, int H, int d_k, int d_v, int chunk, int offset) {
  if (check_shape(F, 1, H, d_k, d_v) != VDA_OK || chunk < 1 || offset < 0 || offset >= chunk)
    return 0;
  return vda::chunked_scan_workspace(F, H, d_k, d_v, chunk, offset);
}

int vda_state_scan_chunked(const void* Inv_tiles, const float* B, const float* alpha,
                           const float* text_state, int F, int H, int d_k, int d_v, int chunk,
                           int offset, void* work, float* S_fwd, float* S_rev, hipStream_t stream) {
  if (!work) return VDA_ERR_NULL;
  int st = check_scan(Inv_tiles, B, F, H, d_k, d_v, S_fwd, S_rev);
  if (st != VDA_OK) return st;
  if (chunk < 1 || offset < 0 || offset >= chunk) return VDA_ERR_SIZE;
  if ((long long)F + 2LL * chunk > 0x3fffffffLL) return VDA_ERR_SIZE;
  if (!aligned(work, 16) || !aligned(alpha, 16) || !aligned(text_state, 16)) return VDA_ERR_ALIGN;
  const size_t fh = (size_t)H * F;
  const Range rw = range_of(work, vda::chunked_scan_workspace(F, H, d_k, d_v, chunk, offset));
  const Range rf = range_of(S_fwd, fh * d_v * d_k * 4), rr = range_of(S_rev, fh * d_v * d_k * 4);
  if (overlaps(rw, rf) || overlaps(rw, rr) || overlaps(rw, range_of(Inv_tiles, fh * d_k * d_k * 4)) ||
      overlaps(rw, range_of(B, fh * d_v * d_k * 4)) ||
      (alpha && (overlaps(rw, range_of(alpha, fh * d_k * 4)) ||
                 overlaps(rf, range_of(alpha, fh * d_k * 4)) ||
                 overlaps(rr, range_of(alpha, fh * d_k * 4)))) ||
      (text_state && (overlaps(rw, range_of(text_state, (size_t)H * d_v * d_k * 4)) ||
                      overlaps(rf, range_of(text_state, (size_t)H * d_v * d_k * 4)) ||
                      overlaps(rr, range_of(text_state, (size_t)H * d_v * d_k * 4)))))
    return VDA_ERR_OVERLAP;
  return hip_status(vda::launch_state_scan_chunked(Inv_tiles, B, alpha, text_state, F, H, d_k, d_v,
                                                   chunk, offset, work, S_fwd, S_rev, stream));
}

int vda_prep(const void* q, const void* k, const void* v, const float* wk_spatial,
             const float* wk_temporal, const float* wv_spatial, const float* wv_temporal, int B,
             int F, int grid_h, int grid_w, int H, int d_k, int d_v, void* q_out, void* k_out,
             void* v_out, hipStream_t stream) {
  // q and q_out may both be NULL: the queries are then left to a forward
  // call that normalises raw queries itself (vda_options.q_heads).
  if (!k || !v || !wk_spatial || !wk_temporal || !wv_spatial || !wv_temporal || !k_out ||
      !v_out || !q != !q_out)
    return VDA_ERR_NULL;
  if (B < 1 || F < 1 || grid_h < 1 || grid_w < 1 || H < 1) return VDA_ERR_SIZE;
  if ((d_k != 64 && d_k != 128) || (d_v != 64 && d_v != 128)) return VDA_ERR_UNSUPPORTED;
  const long long N = (long long)grid_h * grid_w;
  const long long dmax = d_k > d_v ? d_k : d_v;
  // Byte offsets within one clip's projections are 32-bit; grids are
  // one-dimensional.
  if ((long long)F * N * H * dmax * 2 > 0x7fffffffLL) return VDA_ERR_SIZE;
  if ((long long)B * H * ((grid_h + 3) / 4) * ((grid_w + 7) / 8) > 0x7fffffffLL ||
      (long long)B * F * H * N > 0x7fffffffLL)
    return VDA_ERR_SIZE;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(q_out, 16) ||
      !aligned(k_out, 16) || !aligned(v_out, 16) || !aligned(wk_spatial, 4) ||
      !aligned(wk_temporal, 4) || !aligned(wv_spatial, 4) || !aligned(wv_temporal, 4))
    return VDA_ERR_ALIGN;
  const size_t tk = (size_t)B * F * N * H * d_k * 2, tv = (size_t)B * F * N * H * d_v * 2;
  const Range in[] = {range_of(q, q ? tk : 0), range_of(k, tk), range_of(v, tv),
                      range_of(wk_spatial, (size_t)H * d_k * 25 * 4),
                      range_of(wk_temporal, (size_t)H * d_k * 5 * 4),
                      range_of(wv_spatial, (size_t)H * d_v * 25 * 4),
                      range_of(wv_temporal, (size_t)H * d_v * 5 * 4)};
  const Range outs[] = {range_of(q_out, q_out ? tk : 0), range_of(k_out, tk), range_of(v_out, tv)};
  for (const Range& o : outs)
    for (const Range& i : in)
      if (overlaps(o, i)) return VDA_ERR_OVERLAP;
  if (overlaps(outs[0], outs[1]) || overlaps(outs[0], outs[2]) || overlaps(outs[1], outs[2]))
    return VDA_ERR_OVERLAP;
  return hip_status(vda::launch_prep(q, k, v, wk_spatial, wk_temporal, wv_spatial, wv_temporal, B,
                                     F, grid_h, grid_w, H, d_k, d_v, q_out, k_out, v_out, stream));
}

int vda_state_scan_tiles(const void* Inv_tiles, const float* B, int F, int H, int d_k, int d_v,
                         float* S_fwd, float* S_rev, hipStream_t stream) {
  const int st = check_scan(Inv_tiles, B, F, H, d_k, d_v, S_fwd, S_rev);
  if (st != VDA_OK) return st;
  return hip_status(vda::launch_state_scan_tiled(Inv_tiles, B, F, H, d_k, d_v, vda::ScanOptions(),
                                                 S_fwd, S_rev, stream));
}

int vda_readout(const void* q, const float* S_fwd, const float* S_rev, const float* gate, int F,
                int N, int H, int d_k, int d_v, int is_f32, void* out, hipStream_t stream) {
  if (!q || !S_fwd || !S_rev || !gate || !out) return VDA_ERR_NULL;
  int st = check_shape(F, N, H, d_k, d_v);
  if (st != VDA_OK) return st;
  if (!aligned(q, 16) || !aligned(S_fwd, 16) || !aligned(S_rev, 16) || !aligned(gate, 4) ||
      !aligned(out, 16))
    return VDA_ERR_ALIGN;
  const size_t es = is_f32 ? 4 : 2;
  const size_t fh = (size_t)H * F;
  const Range ro = range_of(out, fh * N * d_v * es);
  if (overlaps(ro, range_of(q, fh * N * d_k * es)) ||
      overlaps(ro, range_of(S_fwd, fh * d_v * d_k * 4)) ||
      overlaps(ro, range_of(S_rev, fh * d_v * d_k * 4)) || overlaps(ro, range_of(gate, H * 4)))
    return VDA_ERR_OVERLAP;
  return hip_status(vda::launch_readout(is_f32 != 0, q, S_fwd, S_rev, gate, F, N, H, d_k, d_v,
                                        d_v, vda::GatherOptions(), out, stream));
}

}  // extern "C"
