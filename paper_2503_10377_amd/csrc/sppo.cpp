// libsppo host side: the C ABI declared in include/sppo.h.
//
// Owns, per context: the chunk partition (offsets c_0..c_N), a backward
// workspace on the device (Delta and LSE * log2 e), per-chunk events, and
// page-locked host slots holding each chunk's offload set.  The two
// non-blocking copy streams (device->host and host->device, default
// priority) are shared by every context on a device: each stream the process
// creates takes a hardware queue, and with more streams than queues the
// runtime puts several streams on one in-order queue, so a compute stream
// sharing a queue with a copy stream waited for that stream's copies (about
// 80 ms per 128K-token step was measured with four contexts alive).  One
// pair per device keeps the library at two streams whatever the number of
// contexts (one per layer of a model, say); copies of different contexts
// then run one after another, as they would on the single host link anyway.
// Kernels run on the caller's stream; copies run on the copy streams and are
// ordered against the caller's stream with events only, so nothing blocks
// the host.
//
// Offload protocol for chunk i (two-level activation management, Sec. 5.1;
// sequence-aware offloading overlaps chunk i's copy with chunk i+1's
// compute, Sec. 5.2):
//   offload_issue(i): record E_fwd[i] on the caller stream; the D2H stream
//                     waits for it, copies the offload set to host slot i
//                     and records E_off[i].
//   prefetch(i)     : record E_call[i] on the caller stream; the H2D stream
//                     waits for E_call[i] and E_off[i], copies Q/O/LSE back
//                     and records E_pf[i].
//   bwd_chunk(i)    : the caller stream waits for E_pf[i] before its kernels.
// With K/V eviction (QKVOL_EVICT) the K/V cache rows of offloaded chunks are
// dead once the forward walk is over:
//   prefetch_kv(j)  : like prefetch, for K_j/V_j, recording E_kv[j];
//   bwd_chunk(N-1)  : dK/dV kernel once per KV chunk j = N-1..0, the launch
//                     for chunk j after E_kv[j]; dQ after all of them.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "sppo.h"
#include "sppo_kernels.h"

namespace {

struct EventPair {
  hipEvent_t start = nullptr, stop = nullptr;
  bool pending = false;  // recorded and not yet folded into the totals
};

struct HostSlot {
  void* base = nullptr;  // one pinned allocation per chunk
  void* q = nullptr;
  void* o = nullptr;
  void* lse = nullptr;
  void* k = nullptr;
  void* v = nullptr;
  std::vector<void*> extra;  // extra planes, same order as the problem's
};

}  // namespace

struct sppo_ctx {
  sppo_problem prob{};
  std::vector<int64_t> off;
  std::vector<size_t> extra_rb;  // row bytes of the extra planes
  int64_t s_max = 0;
  size_t elt = 0;
  float scale = 0.f;
  int device = 0;
  int n_cu = 0;
  hipStream_t d2h = nullptr, h2d = nullptr;
  float* delta = nullptr;
  int* tiles = nullptr;  // the dK/dV kernel's tile queues, at the end of the delta allocation
  std::vector<HostSlot> slots;
  std::vector<hipEvent_t> ev_fwd, ev_off, ev_call, ev_pf, ev_kv;
  std::vector<EventPair> t_d2h, t_h2d, t_h2d_kv;
  std::vector<uint8_t> offloaded, prefetched, kv_prefetched, bwd_done;
  // Where offload_issue(i) left chunk i's rows [rows_i, s_i): in a keep
  // buffer (keep_ptr[i]), or in the source buffers (src_q[i] etc.), which a
  // prefetch without a keep buffer must then target.
  std::vector<void*> keep_ptr, src_q, src_o, src_lse;
  std::vector<std::vector<void*>> src_extra;
  std::vector<int64_t> rows;  // offloaded row prefix of each chunk (default s_i)
  bool in_bwd = false;
  int next_fwd = 0, next_bwd = -1;
  uint64_t bytes_d2h = 0, bytes_h2d = 0;
  double ms_d2h = 0.0, ms_h2d = 0.0;
  int32_t n_d2h = 0, n_h2d = 0;
  bool ktiming = false;
  std::vector<EventPair> t_kern[SPPO_KERNEL_COUNT];
  double kms[SPPO_KERNEL_COUNT] = {};
  int32_t klaunch[SPPO_KERNEL_COUNT] = {};
  std::string err;
};

namespace {

thread_local std::string g_create_error;

sppo_status fail(sppo_ctx* ctx, sppo_status st, const std::string& msg) {
  if (ctx) {
    ctx->err = msg;
  } else {
    g_create_error = msg;
  }
  return st;
}

sppo_status hip_fail(sppo_ctx* ctx, hipError_t e, const char* what) {
  return fail(ctx, SPPO_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define SPPO_HIP(ctx, call)                                  \
  do {                                                       \
    hipError_t e_ = (call);                                  \
    if (e_ != hipSuccess) return hip_fail((ctx), e_, #call); \
  } while (0)

bool aligned16(const void* p) { return p && (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// The copy streams shared by the contexts of each device (reference counted;
// the last context on a device destroys them).
struct CopyStreams {
  hipStream_t d2h = nullptr, h2d = nullptr;
  int refs = 0;
};
constexpr int kMaxDevices = 64;
CopyStreams g_copy[kMaxDevices];
std::mutex g_copy_mu;

hipError_t acquire_copy_streams(int dev, hipStream_t* d2h, hipStream_t* h2d) {
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_copy_mu);
  CopyStreams& cs = g_copy[dev];
  if (cs.refs == 0) {
    hipError_t e = hipStreamCreateWithFlags(&cs.d2h, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&cs.h2d, hipStreamNonBlocking);
    if (e != hipSuccess) {
      if (cs.d2h) (void)hipStreamDestroy(cs.d2h);
      cs.d2h = cs.h2d = nullptr;
      return e;
    }
  }
  cs.refs += 1;
  *d2h = cs.d2h;
  *h2d = cs.h2d;
  return hipSuccess;
}

void release_copy_streams(int dev) {
  std::lock_guard<std::mutex> lock(g_copy_mu);
  CopyStreams& cs = g_copy[dev];
  if (--cs.refs == 0) {
    (void)hipStreamDestroy(cs.d2h);
    (void)hipStreamDestroy(cs.h2d);
    cs.d2h = cs.h2d = nullptr;
  }
}

int64_t chunk_len(const sppo_ctx* c, int i) { return c->off[i + 1] - c->off[i]; }

size_t bytes_q(const sppo_ctx* c, int i) {  // also O
  return (size_t)c->prob.batch * chunk_len(c, i) * c->prob.n_q_heads * c->prob.head_dim * c->elt;
}
size_t bytes_lse(const sppo_ctx* c, int i) {
  return (size_t)c->prob.batch * c->prob.n_q_heads * chunk_len(c, i) * sizeof(float);
}
size_t bytes_kv_row_block(const sppo_ctx* c, int i) {  // one batch entry's K_i rows
  return (size_t)chunk_len(c, i) * c->prob.n_kv_heads * c->prob.head_dim * c->elt;
}
bool offload_kv(const sppo_ctx* c) {
  return c->prob.offload == SPPO_OFFLOAD_QKVOL || c->prob.offload == SPPO_OFFLOAD_QKVOL_EVICT;
}
bool evict_kv(const sppo_ctx* c) { return c->prob.offload == SPPO_OFFLOAD_QKVOL_EVICT; }

sppo_status check_ctx_index(sppo_ctx* ctx, int32_t i) {
  if (!ctx) return SPPO_ERR_INVALID_ARG;
  if (i < 0 || i >= ctx->prob.n_chunks) {
    return fail(ctx, SPPO_ERR_INVALID_ARG, "chunk index " + std::to_string(i) + " out of range");
  }
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != ctx->device) {
    return fail(ctx, SPPO_ERR_STATE, "the context's device is not the current device");
  }
  return SPPO_OK;
}

sppo_status check_ptr(sppo_ctx* ctx, const void* p, const char* name) {
  if (!aligned16(p)) {
    return fail(ctx, SPPO_ERR_INVALID_ARG, std::string(name) + " is null or not 16-byte aligned");
  }
  return SPPO_OK;
}

sppo_status check_extra(sppo_ctx* ctx, void* const* extra, const char* name) {
  if (ctx->extra_rb.empty()) return SPPO_OK;
  if (!extra) return fail(ctx, SPPO_ERR_INVALID_ARG, std::string(name) + " is null but the problem has extra planes");
  for (size_t k = 0; k < ctx->extra_rb.size(); ++k) {
    sppo_status st = check_ptr(ctx, extra[k], name);
    if (st != SPPO_OK) return st;
  }
  return SPPO_OK;
}

sppo::ChunkArgs make_args(const sppo_ctx* c, int i) {
  sppo::ChunkArgs a{};
  a.B = c->prob.batch;
  a.S = c->prob.seq_len;
  a.c0 = c->off[i];
  a.c1 = c->off[i + 1];
  a.Hq = c->prob.n_q_heads;
  a.Hkv = c->prob.n_kv_heads;
  a.D = c->prob.head_dim;
  a.scale = c->scale;
  a.delta = c->delta;
  a.lse2 = c->delta + (size_t)c->prob.batch * c->prob.n_q_heads * c->s_max;
  a.kv0 = 0;
  a.kv1 = a.c1;
  a.tiles = c->tiles;
  a.n_cu = c->n_cu;
  return a;
}

// Device->host copy of n contiguous bytes.  Issued as rect copies (rows of
// 1 MiB plus a tail row) because the runtime serves those with the SDMA
// engines, whereas a linear device->host hipMemcpyAsync is served by a blit
// kernel that must find free compute units next to the attention kernels.
hipError_t copy_d2h(void* dst, const void* src, size_t n, hipStream_t s) {
  constexpr size_t W = size_t(1) << 20;
  const size_t rows = n / W, tail = n % W;
  hipError_t e = hipSuccess;
  if (rows) e = hipMemcpy2DAsync(dst, W, src, W, W, rows, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess && tail) {
    e = hipMemcpy2DAsync(static_cast<char*>(dst) + rows * W, tail, static_cast<const char*>(src) + rows * W,
                         tail, tail, 1, hipMemcpyDeviceToHost, s);
  }
  return e;
}

// `height` rows of `width` bytes with the given pitches.  Contiguous spans
// take one linear copy (device->host through copy_d2h); strided ones a rect
// copy.
hipError_t copy_rows(void* dst, size_t dpitch, const void* src, size_t spitch, size_t width, size_t height,
                     hipMemcpyKind kind, hipStream_t s) {
  if (width == 0 || height == 0) return hipSuccess;
  if (height == 1 || (width == dpitch && width == spitch)) {
    const size_t n = width * height;
    return kind == hipMemcpyDeviceToHost ? copy_d2h(dst, src, n, s) : hipMemcpyAsync(dst, src, n, kind, s);
  }
  return hipMemcpy2DAsync(dst, dpitch, src, spitch, width, height, kind, s);
}

// Move the first r rows of chunk i's Q, O and LSE between the device
// buffers and host slot i (the slot mirrors the chunk-local layout):
//   Q_i, O_i [B, s_i, Hq, D]: B spans of r*Hq*D elements, pitch s_i*Hq*D
//   LSE_i   [B, Hq, s_i]    : B*Hq spans of r floats, pitch s_i
// Returns the bytes moved through *bytes.
hipError_t move_qol(sppo_ctx* c, int i, int64_t r, void* q, void* o, float* lse, void* const* extra, bool to_host,
                    hipStream_t s, uint64_t* bytes) {
  const size_t row = (size_t)c->prob.n_q_heads * c->prob.head_dim * c->elt;
  const size_t si = (size_t)chunk_len(c, i), B = (size_t)c->prob.batch, BH = B * c->prob.n_q_heads;
  const hipMemcpyKind kind = to_host ? hipMemcpyDeviceToHost : hipMemcpyHostToDevice;
  HostSlot& h = c->slots[i];
  hipError_t e = hipSuccess;
  void* dev[2] = {q, o};
  void* host[2] = {h.q, h.o};
  for (int t = 0; t < 2 && e == hipSuccess; ++t) {
    e = to_host ? copy_rows(host[t], si * row, dev[t], si * row, r * row, B, kind, s)
                : copy_rows(dev[t], si * row, host[t], si * row, r * row, B, kind, s);
  }
  if (e == hipSuccess) {
    const size_t lp = si * sizeof(float), lw = (size_t)r * sizeof(float);
    e = to_host ? copy_rows(h.lse, lp, lse, lp, lw, BH, kind, s) : copy_rows(lse, lp, h.lse, lp, lw, BH, kind, s);
  }
  *bytes = 2 * (uint64_t)r * row * B + (uint64_t)r * sizeof(float) * BH;
  // extra planes [B, s_i, rb]: B spans of r*rb bytes, pitch s_i*rb
  for (size_t k = 0; k < c->extra_rb.size() && e == hipSuccess; ++k) {
    const size_t rb = c->extra_rb[k];
    e = to_host ? copy_rows(h.extra[k], si * rb, extra[k], si * rb, r * rb, B, kind, s)
                : copy_rows(extra[k], si * rb, h.extra[k], si * rb, r * rb, B, kind, s);
    *bytes += (uint64_t)r * rb * B;
  }
  return e;
}

// Move the first r rows of chunk i's K/V cache rows ([c_i, c_i + r) of the
// full [B, S, Hkv, D] tensors) between the device and host slot i (B spans,
// pitch s_i rows on the host, S rows on the device).
hipError_t move_kv(sppo_ctx* c, int i, int64_t r, void* k, void* v, bool to_host, hipStream_t s, uint64_t* bytes) {
  const size_t row = (size_t)c->prob.n_kv_heads * c->prob.head_dim * c->elt;
  const size_t si = (size_t)chunk_len(c, i), B = (size_t)c->prob.batch, S = (size_t)c->prob.seq_len;
  const size_t off = (size_t)c->off[i] * row;
  const hipMemcpyKind kind = to_host ? hipMemcpyDeviceToHost : hipMemcpyHostToDevice;
  HostSlot& h = c->slots[i];
  hipError_t e = hipSuccess;
  char* dev[2] = {static_cast<char*>(k) + off, static_cast<char*>(v) + off};
  void* host[2] = {h.k, h.v};
  for (int t = 0; t < 2 && e == hipSuccess; ++t) {
    e = to_host ? copy_rows(host[t], si * row, dev[t], S * row, r * row, B, kind, s)
                : copy_rows(dev[t], S * row, host[t], si * row, r * row, B, kind, s);
  }
  *bytes = 2 * (uint64_t)r * row * B;
  return e;
}

// Bytes of chunk i's keep buffer: rows [rows_i, s_i) of every tensor of
// the offload set but K/V (Q_i, O_i, LSE_i, the extra planes), each part
// starting on a 256-byte boundary.
size_t keep_bytes(const sppo_ctx* c, int i) {
  const size_t t = (size_t)(chunk_len(c, i) - c->rows[i]), B = (size_t)c->prob.batch;
  if (t == 0) return 0;
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t row = (size_t)c->prob.n_q_heads * c->prob.head_dim * c->elt;
  size_t n = 2 * up(B * t * row) + up(B * c->prob.n_q_heads * t * sizeof(float));
  for (size_t rb : c->extra_rb) n += up(B * t * rb);
  return n;
}

// Device-to-device move of chunk i's rows [r, s_i) between its chunk-local
// buffers and a keep buffer laid out as [B, s_i - r, ...] per tensor (the
// order and alignment of keep_bytes).
hipError_t move_keep(sppo_ctx* c, int i, int64_t r, void* q, void* o, float* lse, void* const* extra, void* keep,
                     bool to_keep, hipStream_t s) {
  const size_t si = (size_t)chunk_len(c, i), t = si - (size_t)r, B = (size_t)c->prob.batch;
  if (t == 0) return hipSuccess;
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t row = (size_t)c->prob.n_q_heads * c->prob.head_dim * c->elt;
  char* kp = static_cast<char*>(keep);
  hipError_t e = hipSuccess;
  // [B, s_i, w] plane: B spans of t*w bytes at row r, pitch s_i*w <-> t*w.
  // Moved by a kernel on the caller's stream (sppo::launch_copy_rows).
  auto plane = [&](void* dev, size_t w) {
    char* d = static_cast<char*>(dev) + (size_t)r * w;
    hipError_t x = to_keep ? sppo::launch_copy_rows(kp, t * w, d, si * w, t * w, B, s)
                           : sppo::launch_copy_rows(d, si * w, kp, t * w, t * w, B, s);
    kp += up(B * t * w);
    return x;
  };
  e = plane(q, row);
  if (e == hipSuccess) e = plane(o, row);
  if (e == hipSuccess) {  // LSE_i [B, Hq, s_i]: B*Hq spans of t floats
    const size_t BH = B * c->prob.n_q_heads;
    char* d = reinterpret_cast<char*>(lse + r);
    e = to_keep ? sppo::launch_copy_rows(kp, t * 4, d, si * 4, t * 4, BH, s)
                : sppo::launch_copy_rows(d, si * 4, kp, t * 4, t * 4, BH, s);
    kp += up(BH * t * 4);
  }
  for (size_t k = 0; k < c->extra_rb.size() && e == hipSuccess; ++k) e = plane(extra[k], c->extra_rb[k]);
  return e;
}

// Fold a finished timing pair into the totals (waits for it if needed).
void fold(EventPair& p, double& total) {
  if (!p.pending) return;
  float ms = 0.f;
  if (hipEventSynchronize(p.stop) == hipSuccess && hipEventElapsedTime(&ms, p.start, p.stop) == hipSuccess) {
    total += ms;
  }
  p.pending = false;
}

// Launch one kernel, bracketed by timing events when kernel timing is on.
// `slot` < 2N picks the event pair (chunk i uses slot i; the extra dK/dV
// launches of an evicting bwd(N-1) use N + j).
template <class F>
hipError_t timed_launch(sppo_ctx* c, int kind, int i, hipStream_t s, F&& launch) {
  if (!c->ktiming) return launch();
  EventPair& p = c->t_kern[kind][i];
  fold(p, c->kms[kind]);
  hipError_t e = hipEventRecord(p.start, s);
  if (e != hipSuccess) return e;
  if ((e = launch()) != hipSuccess) return e;
  if ((e = hipEventRecord(p.stop, s)) != hipSuccess) return e;
  p.pending = true;
  c->klaunch[kind] += 1;
  return hipSuccess;
}

void destroy_all(sppo_ctx* c) {
  if (c->d2h) (void)hipStreamSynchronize(c->d2h);
  if (c->h2d) (void)hipStreamSynchronize(c->h2d);
  for (auto* v : {&c->ev_fwd, &c->ev_off, &c->ev_call, &c->ev_pf, &c->ev_kv}) {
    for (hipEvent_t e : *v) {
      if (e) (void)hipEventDestroy(e);
    }
  }
  auto destroy_pairs = [](std::vector<EventPair>& v) {
    for (EventPair& p : v) {
      if (p.start) (void)hipEventDestroy(p.start);
      if (p.stop) (void)hipEventDestroy(p.stop);
    }
  };
  for (auto* v : {&c->t_d2h, &c->t_h2d, &c->t_h2d_kv}) destroy_pairs(*v);
  for (auto& v : c->t_kern) destroy_pairs(v);
  for (HostSlot& s : c->slots) {
    if (s.base) (void)hipHostFree(s.base);
  }
  if (c->delta) (void)hipFree(c->delta);
  if (c->d2h) release_copy_streams(c->device);
  delete c;
}

}  // namespace

namespace sppo {
void set_thread_error(const std::string& msg) { g_create_error = msg; }
}  // namespace sppo

extern "C" {

const char* sppo_status_string(sppo_status s) {
  switch (s) {
    case SPPO_OK: return "SPPO_OK";
    case SPPO_ERR_INVALID_ARG: return "SPPO_ERR_INVALID_ARG";
    case SPPO_ERR_UNSUPPORTED: return "SPPO_ERR_UNSUPPORTED";
    case SPPO_ERR_ORDER: return "SPPO_ERR_ORDER";
    case SPPO_ERR_STATE: return "SPPO_ERR_STATE";
    case SPPO_ERR_OOM: return "SPPO_ERR_OOM";
    case SPPO_ERR_HIP: return "SPPO_ERR_HIP";
  }
  return "SPPO_ERR_UNKNOWN";
}

const char* sppo_last_error(const sppo_ctx* ctx) {
  return ctx ? ctx->err.c_str() : g_create_error.c_str();
}

sppo_status sppo_create(const sppo_problem* p, sppo_ctx** out) {
  g_create_error.clear();
  if (!p || !out) return fail(nullptr, SPPO_ERR_INVALID_ARG, "null problem or output pointer");
  if (p->batch < 1 || p->seq_len < 1 || p->n_chunks < 1 || p->n_chunks > p->seq_len) {
    return fail(nullptr, SPPO_ERR_INVALID_ARG, "need batch >= 1, seq_len >= 1, 1 <= n_chunks <= seq_len");
  }
  if (p->n_q_heads < 1 || p->n_kv_heads < 1 || p->n_q_heads % p->n_kv_heads != 0) {
    return fail(nullptr, SPPO_ERR_INVALID_ARG, "need n_q_heads a positive multiple of n_kv_heads");
  }
  if (p->seq_len > 0x7fffffff) {
    return fail(nullptr, SPPO_ERR_UNSUPPORTED, "seq_len of 2^31 or more is not supported");
  }
  if (p->n_q_heads > 65535 || p->n_kv_heads > 65535 || p->batch > 65535) {
    return fail(nullptr, SPPO_ERR_UNSUPPORTED, "batch and head counts above 65535 are not supported");
  }
  if (p->dtype != SPPO_F32 && p->dtype != SPPO_BF16) {
    return fail(nullptr, SPPO_ERR_INVALID_ARG, "unknown dtype");
  }
  if (p->head_dim != 64 && p->head_dim != 128) {
    return fail(nullptr, SPPO_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  }
  // Sizes and offsets are 64-bit products of these counts: keep every
  // [B, S, H, D] tensor (and so the workspace and host slots) below 2^62 bytes.
  if ((double)p->batch * (double)p->seq_len * (double)std::max(p->n_q_heads, p->n_kv_heads) *
          (double)p->head_dim * 4.0 > 0x1p62) {
    return fail(nullptr, SPPO_ERR_UNSUPPORTED, "a [B, S, H, D] tensor of this problem would exceed 2^62 bytes");
  }
  if (p->offload != SPPO_OFFLOAD_NONE && p->offload != SPPO_OFFLOAD_QOL && p->offload != SPPO_OFFLOAD_QKVOL &&
      p->offload != SPPO_OFFLOAD_QKVOL_EVICT) {
    return fail(nullptr, SPPO_ERR_INVALID_ARG, "unknown offload mode");
  }
  if (p->n_extra < 0 || p->n_extra > 16 || (p->n_extra > 0 && !p->extra_row_bytes)) {
    return fail(nullptr, SPPO_ERR_INVALID_ARG, "n_extra must be 0..16 with extra_row_bytes given");
  }
  for (int k = 0; k < p->n_extra; ++k) {
    if (p->extra_row_bytes[k] == 0 || p->extra_row_bytes[k] % 4) {
      return fail(nullptr, SPPO_ERR_INVALID_ARG, "extra_row_bytes must be positive multiples of 4");
    }
  }
  if (!(p->softmax_scale >= 0.f) || std::isinf(p->softmax_scale)) {
    return fail(nullptr, SPPO_ERR_INVALID_ARG, "softmax_scale must be finite and >= 0 (0 = 1/sqrt(D))");
  }
  std::vector<int64_t> off(p->n_chunks + 1);
  if (p->chunk_offsets) {
    for (int i = 0; i <= p->n_chunks; ++i) off[i] = p->chunk_offsets[i];
    if (off[0] != 0 || off[p->n_chunks] != p->seq_len) {
      return fail(nullptr, SPPO_ERR_INVALID_ARG, "chunk_offsets must start at 0 and end at seq_len");
    }
    for (int i = 0; i < p->n_chunks; ++i) {
      if (off[i + 1] <= off[i]) return fail(nullptr, SPPO_ERR_INVALID_ARG, "chunk_offsets must increase strictly");
    }
  } else {
    if (p->seq_len % p->n_chunks != 0) {
      return fail(nullptr, SPPO_ERR_INVALID_ARG, "equal chunks need seq_len % n_chunks == 0");
    }
    for (int i = 0; i <= p->n_chunks; ++i) off[i] = (p->seq_len / p->n_chunks) * i;
  }

  sppo_ctx* c = new (std::nothrow) sppo_ctx();
  if (!c) return fail(nullptr, SPPO_ERR_OOM, "host allocation of the context failed");
  c->prob = *p;
  c->prob.chunk_offsets = nullptr;
  c->prob.extra_row_bytes = nullptr;
  c->extra_rb.assign(p->extra_row_bytes, p->extra_row_bytes + p->n_extra);
  c->off = std::move(off);
  c->elt = p->dtype == SPPO_BF16 ? 2 : 4;
  c->scale = p->softmax_scale > 0.f ? p->softmax_scale : 1.0f / std::sqrt((float)p->head_dim);
  for (int i = 0; i < p->n_chunks; ++i) c->s_max = std::max<int64_t>(c->s_max, chunk_len(c, i));

  auto bail = [&](sppo_status st, const std::string& msg) {
    destroy_all(c);
    return fail(nullptr, st, msg);
  };
  hipError_t e = hipGetDevice(&c->device);
  if (e != hipSuccess) return bail(SPPO_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  e = hipDeviceGetAttribute(&c->n_cu, hipDeviceAttributeMultiprocessorCount, c->device);
  if (e != hipSuccess || c->n_cu < 1) {
    return bail(SPPO_ERR_HIP, std::string("compute unit count: ") + hipGetErrorString(e));
  }
  // Backward workspace: Delta and LSE * log2(e), [B, Hq, s_max] each, then
  // the dK/dV tile queues (zeroed here; every launch leaves them zero).
  const size_t delta_bytes = (size_t)p->batch * p->n_q_heads * c->s_max * sizeof(float);
  const size_t tiles_off = (2 * delta_bytes + 255) & ~(size_t)255;
  e = hipMalloc(&c->delta, tiles_off + sppo::kTileQueueInts * sizeof(int));
  if (e != hipSuccess) {
    c->delta = nullptr;
    return bail(e == hipErrorOutOfMemory ? SPPO_ERR_OOM : SPPO_ERR_HIP,
                std::string("hipMalloc(delta): ") + hipGetErrorString(e));
  }
  c->tiles = reinterpret_cast<int*>(reinterpret_cast<char*>(c->delta) + tiles_off);
  if ((e = hipMemset(c->tiles, 0, sppo::kTileQueueInts * sizeof(int))) != hipSuccess) {
    return bail(SPPO_ERR_HIP, std::string("hipMemset(tile queues): ") + hipGetErrorString(e));
  }
  if ((e = acquire_copy_streams(c->device, &c->d2h, &c->h2d)) != hipSuccess) {
    c->d2h = c->h2d = nullptr;
    return bail(SPPO_ERR_HIP, std::string("copy streams: ") + hipGetErrorString(e));
  }
  const int N = p->n_chunks;
  for (auto* v : {&c->ev_fwd, &c->ev_off, &c->ev_call, &c->ev_pf, &c->ev_kv}) {
    v->assign(N, nullptr);
    for (int i = 0; i < N; ++i) {
      if ((e = hipEventCreateWithFlags(&(*v)[i], hipEventDisableTiming)) != hipSuccess) {
        (*v)[i] = nullptr;
        return bail(SPPO_ERR_HIP, std::string("hipEventCreate: ") + hipGetErrorString(e));
      }
    }
  }
  for (auto* v : {&c->t_d2h, &c->t_h2d, &c->t_h2d_kv}) {
    v->assign(N, EventPair{});
    for (int i = 0; i < N; ++i) {
      if ((e = hipEventCreate(&(*v)[i].start)) != hipSuccess || (e = hipEventCreate(&(*v)[i].stop)) != hipSuccess) {
        return bail(SPPO_ERR_HIP, std::string("hipEventCreate: ") + hipGetErrorString(e));
      }
    }
  }
  c->offloaded.assign(N, 0);
  c->prefetched.assign(N, 0);
  c->kv_prefetched.assign(N, 0);
  c->bwd_done.assign(N, 0);
  c->keep_ptr.assign(N, nullptr);
  c->src_q.assign(N, nullptr);
  c->src_o.assign(N, nullptr);
  c->src_lse.assign(N, nullptr);
  c->src_extra.assign(N, {});
  c->rows.resize(N);
  for (int i = 0; i < N; ++i) c->rows[i] = chunk_len(c, i);
  c->slots.assign(N, HostSlot{});
  if (p->offload != SPPO_OFFLOAD_NONE) {
    for (int i = 0; i < N; ++i) {
      const size_t bq = bytes_q(c, i), bl = bytes_lse(c, i);
      const size_t bkv = offload_kv(c) ? bytes_kv_row_block(c, i) * p->batch : 0;
      auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
      size_t bx = 0;
      for (size_t rb : c->extra_rb) bx += up(rb * (size_t)chunk_len(c, i) * (size_t)p->batch);
      const size_t total = 2 * up(bq) + up(bl) + 2 * up(bkv) + bx;
      void* base = nullptr;
      e = hipHostMalloc(&base, total, hipHostMallocDefault);
      if (e != hipSuccess || !base) {
        return bail(SPPO_ERR_OOM, "hipHostMalloc of " + std::to_string(total) + " pinned bytes for chunk " +
                                      std::to_string(i) + " failed: " + hipGetErrorString(e));
      }
      HostSlot& s = c->slots[i];
      char* b = static_cast<char*>(base);
      s.base = base;
      s.q = b;
      s.o = b + up(bq);
      s.lse = b + 2 * up(bq);
      if (bkv) {
        s.k = b + 2 * up(bq) + up(bl);
        s.v = b + 2 * up(bq) + up(bl) + up(bkv);
      }
      char* xb = b + 2 * up(bq) + up(bl) + 2 * up(bkv);
      for (size_t rb : c->extra_rb) {
        s.extra.push_back(xb);
        xb += up(rb * (size_t)chunk_len(c, i) * (size_t)p->batch);
      }
    }
  }
  *out = c;
  return SPPO_OK;
}

sppo_status sppo_destroy(sppo_ctx* ctx) {
  if (!ctx) return SPPO_OK;
  destroy_all(ctx);
  return SPPO_OK;
}

sppo_status sppo_get_offsets(const sppo_ctx* ctx, int64_t* out, int32_t capacity) {
  if (!ctx || !out || capacity < ctx->prob.n_chunks + 1) return SPPO_ERR_INVALID_ARG;
  for (int i = 0; i <= ctx->prob.n_chunks; ++i) out[i] = ctx->off[i];
  return SPPO_OK;
}

sppo_status sppo_attn_fwd_chunk(sppo_ctx* ctx, int32_t i, const void* q_i, const void* k, const void* v,
                                void* o_i, float* lse_i, void* stream) {
  sppo_status st = check_ctx_index(ctx, i);
  if (st != SPPO_OK) return st;
  if ((st = check_ptr(ctx, q_i, "q_i")) || (st = check_ptr(ctx, k, "k")) || (st = check_ptr(ctx, v, "v")) ||
      (st = check_ptr(ctx, o_i, "o_i")) || (st = check_ptr(ctx, lse_i, "lse_i"))) {
    return st;
  }
  if (ctx->in_bwd || i != ctx->next_fwd) {
    return fail(ctx, SPPO_ERR_ORDER, "forward of chunk " + std::to_string(i) + " out of order (expected " +
                                         (ctx->in_bwd ? std::string("a backward call") : std::to_string(ctx->next_fwd)) + ")");
  }
  sppo::ChunkArgs a = make_args(ctx, i);
  a.q = q_i;
  a.k = k;
  a.v = v;
  a.o = o_i;
  a.lse = lse_i;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool bf16 = ctx->prob.dtype == SPPO_BF16;
  hipError_t e = timed_launch(ctx, SPPO_KERNEL_FWD, i, s, [&] {
    return bf16 ? sppo::launch_fwd_bf16(a, s) : sppo::launch_fwd_f32(a, s);
  });
  if (e != hipSuccess) return hip_fail(ctx, e, "forward kernel launch");
  if (i == 0) {
    std::fill(ctx->offloaded.begin(), ctx->offloaded.end(), 0);
    std::fill(ctx->prefetched.begin(), ctx->prefetched.end(), 0);
    std::fill(ctx->kv_prefetched.begin(), ctx->kv_prefetched.end(), 0);
    std::fill(ctx->bwd_done.begin(), ctx->bwd_done.end(), 0);
  }
  if (++ctx->next_fwd == ctx->prob.n_chunks) {
    ctx->in_bwd = true;
    ctx->next_bwd = ctx->prob.n_chunks - 1;
  }
  return SPPO_OK;
}

sppo_status sppo_attn_bwd_chunk(sppo_ctx* ctx, int32_t i, const void* q_i, const void* k, const void* v,
                                const void* o_i, const float* lse_i, const void* do_i, void* dq_i,
                                float* dk_acc, float* dv_acc, void* stream) {
  sppo_status st = check_ctx_index(ctx, i);
  if (st != SPPO_OK) return st;
  if ((st = check_ptr(ctx, q_i, "q_i")) || (st = check_ptr(ctx, k, "k")) || (st = check_ptr(ctx, v, "v")) ||
      (st = check_ptr(ctx, o_i, "o_i")) || (st = check_ptr(ctx, lse_i, "lse_i")) ||
      (st = check_ptr(ctx, do_i, "do_i")) || (st = check_ptr(ctx, dq_i, "dq_i")) ||
      (st = check_ptr(ctx, dk_acc, "dk_acc")) || (st = check_ptr(ctx, dv_acc, "dv_acc"))) {
    return st;
  }
  if (dk_acc == dv_acc) return fail(ctx, SPPO_ERR_INVALID_ARG, "dk_acc and dv_acc must be distinct buffers");
  if (!ctx->in_bwd || i != ctx->next_bwd) {
    return fail(ctx, SPPO_ERR_ORDER, "backward of chunk " + std::to_string(i) + " out of order (expected " +
                                         (ctx->in_bwd ? std::to_string(ctx->next_bwd) : std::string("the forward pass to finish")) + ")");
  }
  if (ctx->offloaded[i] && !ctx->prefetched[i]) {
    return fail(ctx, SPPO_ERR_STATE, "chunk " + std::to_string(i) + " was offloaded but not prefetched");
  }
  const int N = ctx->prob.n_chunks;
  const bool pieces = evict_kv(ctx) && i == N - 1;
  if (pieces) {
    for (int j = 0; j < N; ++j) {
      if (ctx->offloaded[j] && !ctx->kv_prefetched[j]) {
        return fail(ctx, SPPO_ERR_STATE, "K/V of chunk " + std::to_string(j) + " evicted and not prefetched");
      }
    }
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (ctx->prefetched[i]) SPPO_HIP(ctx, hipStreamWaitEvent(s, ctx->ev_pf[i], 0));
  sppo::ChunkArgs a = make_args(ctx, i);
  a.q = q_i;
  a.k = k;
  a.v = v;
  a.o = const_cast<void*>(o_i);
  a.lse = const_cast<float*>(lse_i);
  a.dout = do_i;
  a.dq = dq_i;
  a.dk = dk_acc;
  a.dv = dv_acc;
  a.accumulate = (i == ctx->prob.n_chunks - 1) ? 0 : 1;
  const bool bf16 = ctx->prob.dtype == SPPO_BF16;
  hipError_t e = timed_launch(ctx, SPPO_KERNEL_BWD_PRE, i, s, [&] {
    return bf16 ? sppo::launch_bwd_pre_bf16(a, s) : sppo::launch_bwd_pre_f32(a, s);
  });
  if (e == hipSuccess && !pieces) {
    e = timed_launch(ctx, SPPO_KERNEL_BWD_DKDV, i, s, [&] {
      return bf16 ? sppo::launch_bwd_dkdv_bf16(a, s) : sppo::launch_bwd_dkdv_f32(a, s);
    });
  }
  // Evicting bwd(N-1): key rows of chunk j only once chunk j's K/V are back;
  // the pieces cover [0, c_N) disjointly, so overwriting is still right.
  for (int j = N - 1; pieces && j >= 0 && e == hipSuccess; --j) {
    if (ctx->kv_prefetched[j]) e = hipStreamWaitEvent(s, ctx->ev_kv[j], 0);
    if (e != hipSuccess) break;
    sppo::ChunkArgs aj = a;
    aj.kv0 = ctx->off[j];
    aj.kv1 = ctx->off[j + 1];
    e = timed_launch(ctx, SPPO_KERNEL_BWD_DKDV, j == N - 1 ? j : N + j, s, [&] {
      return bf16 ? sppo::launch_bwd_dkdv_bf16(aj, s) : sppo::launch_bwd_dkdv_f32(aj, s);
    });
  }
  if (e == hipSuccess) {
    e = timed_launch(ctx, SPPO_KERNEL_BWD_DQ, i, s, [&] {
      return bf16 ? sppo::launch_bwd_dq_bf16(a, s) : sppo::launch_bwd_dq_f32(a, s);
    });
  }
  if (e != hipSuccess) return hip_fail(ctx, e, "backward kernel launch");
  ctx->bwd_done[i] = 1;
  if (--ctx->next_bwd < 0) {
    ctx->in_bwd = false;
    ctx->next_fwd = 0;
  }
  return SPPO_OK;
}

sppo_status sppo_offload_issue(sppo_ctx* ctx, int32_t i, const sppo_chunk_bufs* src, void* stream) {
  sppo_status st = check_ctx_index(ctx, i);
  if (st != SPPO_OK) return st;
  if (ctx->prob.offload == SPPO_OFFLOAD_NONE) return fail(ctx, SPPO_ERR_STATE, "context created with offload NONE");
  if (!src) return fail(ctx, SPPO_ERR_INVALID_ARG, "null chunk buffers");
  if ((st = check_ptr(ctx, src->q, "src.q")) || (st = check_ptr(ctx, src->o, "src.o")) ||
      (st = check_ptr(ctx, src->lse, "src.lse"))) {
    return st;
  }
  if (offload_kv(ctx) && ((st = check_ptr(ctx, src->k, "src.k")) || (st = check_ptr(ctx, src->v, "src.v")))) return st;
  if ((st = check_extra(ctx, src->extra, "src.extra")) != SPPO_OK) return st;
  const bool fwd_done = ctx->in_bwd || i < ctx->next_fwd;
  if (!fwd_done) return fail(ctx, SPPO_ERR_STATE, "offload of chunk " + std::to_string(i) + " before its forward");
  if (ctx->offloaded[i]) return fail(ctx, SPPO_ERR_STATE, "chunk " + std::to_string(i) + " already offloaded");

  const int64_t r = ctx->rows[i];
  const bool has_rest = r < chunk_len(ctx, i);
  if (has_rest && src->keep && !aligned16(src->keep)) {
    return fail(ctx, SPPO_ERR_INVALID_ARG, "src.keep is not 16-byte aligned");
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  // Rows [r, s_i) stay on the device: into the keep buffer, on the caller's
  // stream, so the source buffers are free as a whole after E_off[i].
  if (has_rest && src->keep) {
    SPPO_HIP(ctx, move_keep(ctx, i, r, src->q, src->o, src->lse, src->extra, src->keep, true, s));
  }
  ctx->keep_ptr[i] = has_rest ? src->keep : nullptr;
  ctx->src_q[i] = src->q;
  ctx->src_o[i] = src->o;
  ctx->src_lse[i] = src->lse;
  ctx->src_extra[i].assign(src->extra ? src->extra : nullptr,
                           src->extra ? src->extra + ctx->extra_rb.size() : nullptr);
  fold(ctx->t_d2h[i], ctx->ms_d2h);
  SPPO_HIP(ctx, hipEventRecord(ctx->ev_fwd[i], s));
  SPPO_HIP(ctx, hipStreamWaitEvent(ctx->d2h, ctx->ev_fwd[i], 0));
  SPPO_HIP(ctx, hipEventRecord(ctx->t_d2h[i].start, ctx->d2h));
  uint64_t bytes = 0, kv_bytes = 0;
  SPPO_HIP(ctx, move_qol(ctx, i, r, src->q, src->o, src->lse, src->extra, true, ctx->d2h, &bytes));
  if (offload_kv(ctx)) SPPO_HIP(ctx, move_kv(ctx, i, r, src->k, src->v, true, ctx->d2h, &kv_bytes));
  bytes += kv_bytes;
  SPPO_HIP(ctx, hipEventRecord(ctx->t_d2h[i].stop, ctx->d2h));
  SPPO_HIP(ctx, hipEventRecord(ctx->ev_off[i], ctx->d2h));
  ctx->t_d2h[i].pending = true;
  ctx->offloaded[i] = 1;
  ctx->prefetched[i] = 0;
  ctx->bytes_d2h += bytes;
  ctx->n_d2h += 1;
  return SPPO_OK;
}

sppo_status sppo_offload_wait(sppo_ctx* ctx, int32_t i, void* stream) {
  sppo_status st = check_ctx_index(ctx, i);
  if (st != SPPO_OK) return st;
  if (!ctx->offloaded[i]) return fail(ctx, SPPO_ERR_STATE, "chunk " + std::to_string(i) + " was not offloaded");
  SPPO_HIP(ctx, hipStreamWaitEvent(static_cast<hipStream_t>(stream), ctx->ev_off[i], 0));
  return SPPO_OK;
}

sppo_status sppo_prefetch(sppo_ctx* ctx, int32_t i, const sppo_chunk_bufs* dst, void* stream) {
  sppo_status st = check_ctx_index(ctx, i);
  if (st != SPPO_OK) return st;
  if (!dst) return fail(ctx, SPPO_ERR_INVALID_ARG, "null chunk buffers");
  if ((st = check_ptr(ctx, dst->q, "dst.q")) || (st = check_ptr(ctx, dst->o, "dst.o")) ||
      (st = check_ptr(ctx, dst->lse, "dst.lse"))) {
    return st;
  }
  if ((st = check_extra(ctx, dst->extra, "dst.extra")) != SPPO_OK) return st;
  if (!ctx->offloaded[i]) return fail(ctx, SPPO_ERR_STATE, "prefetch of chunk " + std::to_string(i) + " that was not offloaded");
  if (ctx->prefetched[i]) return fail(ctx, SPPO_ERR_STATE, "chunk " + std::to_string(i) + " already prefetched");
  const int64_t r = ctx->rows[i];
  if (r < chunk_len(ctx, i)) {
    if (ctx->keep_ptr[i]) {
      if (dst->keep != ctx->keep_ptr[i]) {
        return fail(ctx, SPPO_ERR_INVALID_ARG, "dst.keep of chunk " + std::to_string(i) +
                                                   " is not the keep buffer its offload filled");
      }
    } else {
      bool same = dst->q == ctx->src_q[i] && dst->o == ctx->src_o[i] && dst->lse == ctx->src_lse[i];
      for (size_t k = 0; same && k < ctx->extra_rb.size(); ++k) same = dst->extra[k] == ctx->src_extra[i][k];
      if (!same) {
        return fail(ctx, SPPO_ERR_STATE, "rows of chunk " + std::to_string(i) +
                                             " past its offloaded prefix stayed in the offload's source buffers "
                                             "(no keep buffer): the prefetch must target those buffers");
      }
    }
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (r < chunk_len(ctx, i) && ctx->keep_ptr[i]) {
    SPPO_HIP(ctx, move_keep(ctx, i, r, dst->q, dst->o, dst->lse, dst->extra, ctx->keep_ptr[i], false, s));
  }
  fold(ctx->t_h2d[i], ctx->ms_h2d);
  SPPO_HIP(ctx, hipEventRecord(ctx->ev_call[i], s));
  SPPO_HIP(ctx, hipStreamWaitEvent(ctx->h2d, ctx->ev_call[i], 0));
  SPPO_HIP(ctx, hipStreamWaitEvent(ctx->h2d, ctx->ev_off[i], 0));
  SPPO_HIP(ctx, hipEventRecord(ctx->t_h2d[i].start, ctx->h2d));
  uint64_t bytes = 0;
  SPPO_HIP(ctx, move_qol(ctx, i, r, dst->q, dst->o, dst->lse, dst->extra, false, ctx->h2d, &bytes));
  SPPO_HIP(ctx, hipEventRecord(ctx->t_h2d[i].stop, ctx->h2d));
  SPPO_HIP(ctx, hipEventRecord(ctx->ev_pf[i], ctx->h2d));
  ctx->t_h2d[i].pending = true;
  ctx->prefetched[i] = 1;
  ctx->bytes_h2d += bytes;
  ctx->n_h2d += 1;
  return SPPO_OK;
}

sppo_status sppo_prefetch_wait(sppo_ctx* ctx, int32_t i, void* stream) {
  sppo_status st = check_ctx_index(ctx, i);
  if (st != SPPO_OK) return st;
  if (!ctx->prefetched[i]) return fail(ctx, SPPO_ERR_STATE, "chunk " + std::to_string(i) + " was not prefetched");
  SPPO_HIP(ctx, hipStreamWaitEvent(static_cast<hipStream_t>(stream), ctx->ev_pf[i], 0));
  return SPPO_OK;
}

sppo_status sppo_prefetch_kv(sppo_ctx* ctx, int32_t i, void* k, void* v, void* stream) {
  sppo_status st = check_ctx_index(ctx, i);
  if (st != SPPO_OK) return st;
  if (!evict_kv(ctx)) return fail(ctx, SPPO_ERR_STATE, "K/V prefetch needs a context created with QKVOL_EVICT");
  if ((st = check_ptr(ctx, k, "k")) || (st = check_ptr(ctx, v, "v"))) return st;
  if (!ctx->in_bwd) return fail(ctx, SPPO_ERR_STATE, "K/V prefetch before the forward walk is over");
  if (ctx->next_bwd != ctx->prob.n_chunks - 1) {
    return fail(ctx, SPPO_ERR_STATE, "K/V prefetch after the backward walk has started");
  }
  if (!ctx->offloaded[i]) return fail(ctx, SPPO_ERR_STATE, "K/V prefetch of chunk " + std::to_string(i) + " that was not offloaded");
  if (ctx->kv_prefetched[i]) return fail(ctx, SPPO_ERR_STATE, "K/V of chunk " + std::to_string(i) + " already prefetched");
  hipStream_t s = static_cast<hipStream_t>(stream);
  fold(ctx->t_h2d_kv[i], ctx->ms_h2d);
  SPPO_HIP(ctx, hipEventRecord(ctx->ev_call[i], s));
  SPPO_HIP(ctx, hipStreamWaitEvent(ctx->h2d, ctx->ev_call[i], 0));
  SPPO_HIP(ctx, hipStreamWaitEvent(ctx->h2d, ctx->ev_off[i], 0));
  SPPO_HIP(ctx, hipEventRecord(ctx->t_h2d_kv[i].start, ctx->h2d));
  uint64_t bytes = 0;
  SPPO_HIP(ctx, move_kv(ctx, i, ctx->rows[i], k, v, false, ctx->h2d, &bytes));
  SPPO_HIP(ctx, hipEventRecord(ctx->t_h2d_kv[i].stop, ctx->h2d));
  SPPO_HIP(ctx, hipEventRecord(ctx->ev_kv[i], ctx->h2d));
  ctx->t_h2d_kv[i].pending = true;
  ctx->kv_prefetched[i] = 1;
  ctx->bytes_h2d += bytes;
  return SPPO_OK;
}

sppo_status sppo_set_offload_rows(sppo_ctx* ctx, int32_t i, int64_t rows) {
  sppo_status st = check_ctx_index(ctx, i);
  if (st != SPPO_OK) return st;
  if (rows < 0 || rows > chunk_len(ctx, i)) {
    return fail(ctx, SPPO_ERR_INVALID_ARG, "offload rows of chunk " + std::to_string(i) + " outside [0, s_i]");
  }
  if (ctx->in_bwd || ctx->next_fwd != 0) return fail(ctx, SPPO_ERR_STATE, "offload rows changed during a walk");
  ctx->rows[i] = rows;
  return SPPO_OK;
}

sppo_status sppo_get_offload_rows(const sppo_ctx* ctx, int64_t* out, int32_t capacity) {
  if (!ctx || !out || capacity < ctx->prob.n_chunks) return SPPO_ERR_INVALID_ARG;
  for (int i = 0; i < ctx->prob.n_chunks; ++i) out[i] = ctx->rows[i];
  return SPPO_OK;
}

sppo_status sppo_reset(sppo_ctx* ctx) {
  if (!ctx) return SPPO_ERR_INVALID_ARG;
  // Copies of the abandoned walk may still read or write device buffers
  // that the next walk reuses (and host slots that its offloads refill):
  // wait for both copy streams (each also waits for the caller-stream
  // events its copies were ordered behind) before forgetting them.
  SPPO_HIP(ctx, hipStreamSynchronize(ctx->d2h));
  SPPO_HIP(ctx, hipStreamSynchronize(ctx->h2d));
  ctx->in_bwd = false;
  ctx->next_fwd = 0;
  ctx->next_bwd = -1;
  std::fill(ctx->offloaded.begin(), ctx->offloaded.end(), 0);
  std::fill(ctx->prefetched.begin(), ctx->prefetched.end(), 0);
  std::fill(ctx->kv_prefetched.begin(), ctx->kv_prefetched.end(), 0);
  std::fill(ctx->bwd_done.begin(), ctx->bwd_done.end(), 0);
  return SPPO_OK;
}

size_t sppo_keep_bytes(const sppo_ctx* ctx, int32_t i) {
  if (!ctx || i < 0 || i >= ctx->prob.n_chunks) return 0;
  return keep_bytes(ctx, i);
}

sppo_status sppo_attn_finalize_chunk(sppo_ctx* ctx, int32_t i, const float* dk_acc, const float* dv_acc,
                                     void* dk_out, void* dv_out, void* stream) {
  sppo_status st = check_ctx_index(ctx, i);
  if (st != SPPO_OK) return st;
  if ((st = check_ptr(ctx, dk_acc, "dk_acc")) || (st = check_ptr(ctx, dv_acc, "dv_acc")) ||
      (st = check_ptr(ctx, dk_out, "dk_out")) || (st = check_ptr(ctx, dv_out, "dv_out"))) {
    return st;
  }
  if (dk_out == dv_out) return fail(ctx, SPPO_ERR_INVALID_ARG, "dk_out and dv_out must be distinct buffers");
  if (!ctx->bwd_done[i]) {
    return fail(ctx, SPPO_ERR_STATE, "finalize of chunk " + std::to_string(i) +
                                         " before its backward in this walk");
  }
  sppo::FinalizeArgs a{};
  a.dk = dk_acc;
  a.dv = dv_acc;
  a.out_k = dk_out;
  a.out_v = dv_out;
  a.B = ctx->prob.batch;
  a.S = ctx->prob.seq_len;
  a.W = (int64_t)ctx->prob.n_kv_heads * ctx->prob.head_dim;
  a.row0 = ctx->off[i];
  a.rows = chunk_len(ctx, i);
  a.bf16 = ctx->prob.dtype == SPPO_BF16;
  hipError_t e = sppo::launch_finalize(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(ctx, e, "finalize kernel launch");
  return SPPO_OK;
}

sppo_status sppo_link_probe(sppo_ctx* ctx, size_t bytes, sppo_link_rates_t* out) {
  if (!ctx || !out) return SPPO_ERR_INVALID_ARG;
  if (bytes < (size_t(1) << 20)) return fail(ctx, SPPO_ERR_INVALID_ARG, "link probe needs at least 1 MiB");
  void* dev = nullptr;
  void* host = nullptr;
  hipEvent_t ev[6] = {};
  hipError_t e = hipMalloc(&dev, bytes);
  if (e == hipSuccess) e = hipHostMalloc(&host, bytes, hipHostMallocDefault);
  for (int k = 0; k < 6 && e == hipSuccess; ++k) e = hipEventCreate(&ev[k]);
  float ms[3] = {};
  if (e == hipSuccess) e = hipMemset(dev, 0, bytes);
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->d2h);
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->h2d);
  // D2H alone, H2D alone (each on its own stream), then both at once.
  if (e == hipSuccess) e = hipEventRecord(ev[0], ctx->d2h);
  if (e == hipSuccess) e = copy_d2h(host, dev, bytes, ctx->d2h);
  if (e == hipSuccess) e = hipEventRecord(ev[1], ctx->d2h);
  if (e == hipSuccess) e = hipEventSynchronize(ev[1]);
  if (e == hipSuccess) e = hipEventElapsedTime(&ms[0], ev[0], ev[1]);
  if (e == hipSuccess) e = hipEventRecord(ev[2], ctx->h2d);
  if (e == hipSuccess) e = hipMemcpyAsync(dev, host, bytes, hipMemcpyHostToDevice, ctx->h2d);
  if (e == hipSuccess) e = hipEventRecord(ev[3], ctx->h2d);
  if (e == hipSuccess) e = hipEventSynchronize(ev[3]);
  if (e == hipSuccess) e = hipEventElapsedTime(&ms[1], ev[2], ev[3]);
  // Duplex: the halves of each buffer move in opposite directions.
  const size_t half = bytes / 2;
  if (e == hipSuccess) e = hipEventRecord(ev[4], ctx->d2h);
  if (e == hipSuccess) e = hipStreamWaitEvent(ctx->h2d, ev[4], 0);
  if (e == hipSuccess) e = copy_d2h(host, dev, half, ctx->d2h);
  if (e == hipSuccess) e = hipMemcpyAsync(static_cast<char*>(dev) + half, static_cast<char*>(host) + half, half,
                                          hipMemcpyHostToDevice, ctx->h2d);
  if (e == hipSuccess) e = hipEventRecord(ev[5], ctx->h2d);
  if (e == hipSuccess) e = hipStreamWaitEvent(ctx->d2h, ev[5], 0);
  if (e == hipSuccess) e = hipEventRecord(ev[5], ctx->d2h);
  if (e == hipSuccess) e = hipEventSynchronize(ev[5]);
  if (e == hipSuccess) e = hipEventElapsedTime(&ms[2], ev[4], ev[5]);
  for (hipEvent_t x : ev) {
    if (x) (void)hipEventDestroy(x);
  }
  if (host) (void)hipHostFree(host);
  if (dev) (void)hipFree(dev);
  if (e != hipSuccess) return hip_fail(ctx, e, "link probe");
  out->d2h_GBps = bytes / (ms[0] * 1e6);
  out->h2d_GBps = bytes / (ms[1] * 1e6);
  out->duplex_GBps = 2.0 * half / (ms[2] * 1e6);
  return SPPO_OK;
}

sppo_status sppo_set_kernel_timing(sppo_ctx* ctx, int32_t enable) {
  if (!ctx) return SPPO_ERR_INVALID_ARG;
  if (enable && ctx->t_kern[0].empty()) {
    for (auto& v : ctx->t_kern) {
      v.assign(2 * (size_t)ctx->prob.n_chunks, EventPair{});
      for (EventPair& p : v) {
        SPPO_HIP(ctx, hipEventCreate(&p.start));
        SPPO_HIP(ctx, hipEventCreate(&p.stop));
      }
    }
  }
  ctx->ktiming = enable != 0;
  return SPPO_OK;
}

sppo_status sppo_kernel_times(sppo_ctx* ctx, sppo_kernel_times_t* out, int32_t reset_after) {
  if (!ctx || !out) return SPPO_ERR_INVALID_ARG;
  for (int k = 0; k < SPPO_KERNEL_COUNT; ++k) {
    for (EventPair& p : ctx->t_kern[k]) fold(p, ctx->kms[k]);
    out->ms[k] = ctx->kms[k];
    out->launches[k] = ctx->klaunch[k];
    if (reset_after) {
      ctx->kms[k] = 0.0;
      ctx->klaunch[k] = 0;
    }
  }
  return SPPO_OK;
}

sppo_status sppo_sync(sppo_ctx* ctx) {
  if (!ctx) return SPPO_ERR_INVALID_ARG;
  SPPO_HIP(ctx, hipStreamSynchronize(ctx->d2h));
  SPPO_HIP(ctx, hipStreamSynchronize(ctx->h2d));
  return SPPO_OK;
}

sppo_status sppo_copy_stats(sppo_ctx* ctx, sppo_copy_stats_t* out, int32_t reset_after) {
  if (!ctx || !out) return SPPO_ERR_INVALID_ARG;
  SPPO_HIP(ctx, hipStreamSynchronize(ctx->d2h));
  SPPO_HIP(ctx, hipStreamSynchronize(ctx->h2d));
  for (EventPair& p : ctx->t_d2h) fold(p, ctx->ms_d2h);
  for (EventPair& p : ctx->t_h2d) fold(p, ctx->ms_h2d);
  for (EventPair& p : ctx->t_h2d_kv) fold(p, ctx->ms_h2d);
  out->bytes_d2h = ctx->bytes_d2h;
  out->bytes_h2d = ctx->bytes_h2d;
  out->ms_d2h = ctx->ms_d2h;
  out->ms_h2d = ctx->ms_h2d;
  out->n_d2h = ctx->n_d2h;
  out->n_h2d = ctx->n_h2d;
  if (reset_after) {
    ctx->bytes_d2h = ctx->bytes_h2d = 0;
    ctx->ms_d2h = ctx->ms_h2d = 0.0;
    ctx->n_d2h = ctx->n_h2d = 0;
  }
  return SPPO_OK;
}

sppo_status sppo_balanced_offsets(int64_t seq_len, int32_t n_chunks, int64_t align, int64_t* out) {
  if (!out || seq_len < 1 || n_chunks < 1 || align < 1 || (int64_t)n_chunks * align > seq_len) {
    return SPPO_ERR_INVALID_ARG;
  }
  const int N = n_chunks;
  out[0] = 0;
  out[N] = seq_len;
  for (int k = 1; k < N; ++k) {
    const double c = (double)seq_len * std::sqrt((double)k / N);
    out[k] = (int64_t)std::llround(c / align) * align;
  }
  // Every chunk at least `align` rows long: push up from the front, then
  // down from the back (room exists since N * align <= S).
  for (int k = 1; k < N; ++k) out[k] = std::max(out[k], out[k - 1] + align);
  for (int k = N - 1; k >= 1; --k) out[k] = std::min(out[k], out[k + 1] - align);
  return SPPO_OK;
}

sppo_status sppo_plan_offload_rows(const int64_t* offsets, int32_t n_chunks, double bytes_per_row, double bw_GBps,
                                   const double* t_overlap_ms, int64_t align, int64_t* rows_out) {
  if (!offsets || !t_overlap_ms || !rows_out || n_chunks < 1 || !(bytes_per_row > 0.0) || !(bw_GBps > 0.0) ||
      align < 1) {
    return SPPO_ERR_INVALID_ARG;
  }
  for (int i = 0; i < n_chunks; ++i) {
    const int64_t si = offsets[i + 1] - offsets[i];
    if (si < 1 || !(t_overlap_ms[i] >= 0.0)) return SPPO_ERR_INVALID_ARG;
    if (i == n_chunks - 1) {
      rows_out[i] = 0;  // its backward follows its forward directly
      continue;
    }
    // Bytes the link moves while the overlapped compute runs.
    const double fit = bw_GBps * 1e6 * t_overlap_ms[i] / bytes_per_row;
    int64_t r = fit >= (double)si ? si : (int64_t)std::floor(fit);
    if (r < si) r = (r / align) * align;
    rows_out[i] = r;
  }
  return SPPO_OK;
}

}  // extern "C"
