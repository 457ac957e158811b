// C ABI of the VDA library: argument validation, workspace, launch order.
// Declarations and contracts are in include/vda.h.
#include <stdint.h>
#include <string.h>

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
  // Byte offsets within one frame of one head are 32-bit.
  const int dmax = padded_dim(d_k > d_v ? d_k : d_v);
  if ((long long)N * dmax * 4 > 0x7fffffffLL) return VDA_ERR_SIZE;
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
// and stay cached until the process ends (a free would synchronise the
// device).  A buffer is reused by a later call on the same stream (stream
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
    c.entries.push_back(e);
    pick = (int)c.entries.size() - 1;
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

int default_splits(int F, int N, int H) {
  // The statistics step runs two workgroups (row halves) per frame and split;
  // split the tokens only when that leaves fewer than about three workgroups
  // per compute unit, and never below 256 tokens per split.  Splits cost a
  // partial sum per split and a fold in the inverse step.
  const long long wg_per_split = 2LL * H * F;
  const long long target = 3LL * current_device_cus();
  long long s = (target + wg_per_split - 1) / wg_per_split;
  long long cap = N / 256;
  if (cap < 1) cap = 1;
  if (s > cap) s = cap;
  if (s < 1) s = 1;
  return (int)s;
}

struct Workspace {
  size_t a_part, b_part, s_fwd, s_rev, total;  // byte offsets / total
};

Workspace workspace_layout(int F, int H, int d_k, int d_v, int splits) {
  const size_t fh = (size_t)H * F;
  const size_t a = (size_t)splits * fh * d_k * d_k * sizeof(float);
  const size_t b = (size_t)splits * fh * d_v * d_k * sizeof(float);
  const size_t s = fh * d_v * d_k * sizeof(float);
  Workspace w;
  w.a_part = 0;
  w.b_part = a;
  w.s_fwd = a + b;
  w.s_rev = a + b + s;
  w.total = a + b + 2 * s;
  return w;
}

int forward_impl(bool is_f32, const void* q, const void* k, const void* v, const float* beta,
                 const float* gate, int F, int N, int H, int d_k, int d_v, void* out,
                 hipStream_t stream) {
  if (!q || !k || !v || !beta || !gate || !out) return VDA_ERR_NULL;
  int st = check_shape(F, N, H, d_k, d_v, true);
  if (st != VDA_OK) return st;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
      !aligned(beta, 4) || !aligned(gate, 4))
    return VDA_ERR_ALIGN;
  const size_t es = is_f32 ? 4 : 2;
  const size_t tok = (size_t)H * F * N;
  const Range ro = range_of(out, tok * d_v * es);
  if (overlaps(ro, range_of(q, tok * d_k * es)) || overlaps(ro, range_of(k, tok * d_k * es)) ||
      overlaps(ro, range_of(v, tok * d_v * es)) || overlaps(ro, range_of(beta, tok * 4)) ||
      overlaps(ro, range_of(gate, (size_t)H * 4)))
    return VDA_ERR_OVERLAP;

  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return VDA_ERR_HIP;
  const int splits = default_splits(F, N, H);
  // Heads narrower than 32 channels run as zero-padded 32-channel heads; the
  // padded q, k, v and output live after the state buffers.
  const int pk = padded_dim(d_k), pv = padded_dim(d_v);
  const Workspace w = workspace_layout(F, H, pk, pv, splits);
  const size_t qk_pad = pk != d_k ? round_up(tok * pk * es, 256) : 0;
  const size_t v_pad = pv != d_v ? round_up(tok * pv * es, 256) : 0;
  const size_t ws_bytes = round_up(w.total, 256) + 2 * qk_pad + 2 * v_pad;
  const int wsi = acquire_workspace(dev, ws_bytes, stream);
  if (wsi < 0) return VDA_ERR_NOMEM;
  char* base = static_cast<char*>(workspace_ptr(dev, wsi));
  float* A_part = reinterpret_cast<float*>(base + w.a_part);
  float* B_part = reinterpret_cast<float*>(base + w.b_part);
  float* S_fwd = reinterpret_cast<float*>(base + w.s_fwd);
  float* S_rev = reinterpret_cast<float*>(base + w.s_rev);
  float* Inv = A_part;  // the inverse overwrites the first partial
  char* pad_base = base + round_up(w.total, 256);
  const void* qx = q;
  const void* kx = k;
  const void* vx = v;
  void* ox = out;

  hipError_t e = hipSuccess;
  if (qk_pad) {
    void* qp = pad_base;
    void* kp = pad_base + qk_pad;
    e = vda::launch_pad_rows(q, qp, (long long)tok, (int)(d_k * es), (int)(pk * es), stream);
    if (e == hipSuccess)
      e = vda::launch_pad_rows(k, kp, (long long)tok, (int)(d_k * es), (int)(pk * es), stream);
    qx = qp;
    kx = kp;
  }
  if (v_pad && e == hipSuccess) {
    void* vp = pad_base + 2 * qk_pad;
    e = vda::launch_pad_rows(v, vp, (long long)tok, (int)(d_v * es), (int)(pv * es), stream);
    vx = vp;
    ox = pad_base + 2 * qk_pad + v_pad;
  }
  if (e == hipSuccess)
    e = vda::launch_frame_stats(is_f32, kx, vx, beta, F, N, H, pk, pv, splits, A_part, B_part,
                                stream);
  if (e == hipSuccess)
    e = vda::launch_frame_inverse(A_part, B_part, splits, (long long)H * F, pk, pv, Inv, stream);
  if (e == hipSuccess)
    e = vda::launch_state_scan(is_f32, Inv, B_part, F, H, pk, pv, S_fwd, S_rev, stream);
  if (e == hipSuccess)
    e = vda::launch_readout(is_f32, qx, S_fwd, S_rev, gate, F, N, H, pk, pv, d_v, ox, stream);
  if (e == hipSuccess && ox != out)
    e = vda::launch_unpad_rows(ox, out, (long long)tok, (int)(pv * es), (int)(d_v * es), stream);
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
    default: return "VDA: unknown status";
  }
}

int vda_forward(const void* q, const void* k, const void* v, const float* beta, const float* gate,
                int F, int N, int H, int d_k, int d_v, void* out, hipStream_t stream) {
  return forward_impl(false, q, k, v, beta, gate, F, N, H, d_k, d_v, out, stream);
}

int vda_forward_f32(const float* q, const float* k, const float* v, const float* beta,
                    const float* gate, int F, int N, int H, int d_k, int d_v, float* out,
                    hipStream_t stream) {
  return forward_impl(true, q, k, v, beta, gate, F, N, H, d_k, d_v, out, stream);
}

int vda_default_splits(int F, int N, int H) {
  if (F < 1 || N < 1 || H < 1) return 1;
  return default_splits(F, N, H);
}

int vda_frame_stats(const void* k, const void* v, const float* beta, int F, int N, int H,
                    int d_k, int d_v, int splits, int is_f32, float* A_part, float* B_part,
                    hipStream_t stream) {
  if (!k || !v || !beta || !A_part || !B_part) return VDA_ERR_NULL;
  int st = check_shape(F, N, H, d_k, d_v);
  if (st != VDA_OK) return st;
  if (splits < 1 || splits > (N + 63) / 64 || (long long)H * F * splits > 0x7fffffffLL)
    return VDA_ERR_SIZE;
  if (!aligned(k, 16) || !aligned(v, 16) || !aligned(beta, 4) || !aligned(A_part, 16) ||
      !aligned(B_part, 16))
    return VDA_ERR_ALIGN;
  const size_t fh = (size_t)H * F;
  const Range ra = range_of(A_part, (size_t)splits * fh * d_k * d_k * 4);
  const Range rb = range_of(B_part, (size_t)splits * fh * d_v * d_k * 4);
  const size_t es = is_f32 ? 4 : 2;
  const Range rk = range_of(k, fh * N * d_k * es), rv = range_of(v, fh * N * d_v * es),
              rbeta = range_of(beta, fh * N * 4);
  if (overlaps(ra, rb) || overlaps(ra, rk) || overlaps(ra, rv) || overlaps(ra, rbeta) ||
      overlaps(rb, rk) || overlaps(rb, rv) || overlaps(rb, rbeta))
    return VDA_ERR_OVERLAP;
  return hip_status(vda::launch_frame_stats(is_f32 != 0, k, v, beta, F, N, H, d_k, d_v, splits,
                                            A_part, B_part, stream));
}

int vda_frame_inverse(const float* A_part, float* B_part, int splits, int count, int d_k,
                      int d_v, float* Inv, hipStream_t stream) {
  if (!A_part || !Inv || (splits > 1 && !B_part)) return VDA_ERR_NULL;
  if (splits < 1 || count < 1 || (long long)count * 64 > 0x7fffffffLL) return VDA_ERR_SIZE;
  if (!supported_dim(d_k) || (splits > 1 && !supported_dim(d_v))) return VDA_ERR_UNSUPPORTED;
  if (!aligned(A_part, 16) || !aligned(Inv, 16) || !aligned(B_part, 16)) return VDA_ERR_ALIGN;
  const size_t mat = (size_t)count * d_k * d_k * 4;
  const Range ri = range_of(Inv, mat);
  for (int s = 0; s < splits; ++s) {
    const Range rs = range_of(reinterpret_cast<const char*>(A_part) + s * mat, mat);
    const bool same = rs.lo == ri.lo;
    if (overlaps(ri, rs) && !(same && s == 0)) return VDA_ERR_OVERLAP;
  }
  if (splits > 1) {
    const size_t bmat = (size_t)count * d_v * d_k * 4;
    const Range rb = range_of(B_part, splits * bmat);
    if (overlaps(rb, ri) || overlaps(rb, range_of(A_part, splits * mat))) return VDA_ERR_OVERLAP;
  }
  return hip_status(
      vda::launch_frame_inverse(A_part, B_part, splits, count, d_k, d_v, Inv, stream));
}

int vda_state_scan(const float* Inv, const float* B, int F, int H, int d_k, int d_v, int is_f32,
                   float* S_fwd, float* S_rev, hipStream_t stream) {
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
  return hip_status(
      vda::launch_state_scan(is_f32 != 0, Inv, B, F, H, d_k, d_v, S_fwd, S_rev, stream));
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
                                        d_v, out, stream));
}

}  // extern "C"
