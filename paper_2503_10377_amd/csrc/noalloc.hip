// A chunk backward that allocates nothing, for callers that cannot call
// hipMalloc (code under HIP graph capture, tight serving loops, harnesses
// that forbid allocation): the same kernels as sppo_attn_bwd_chunk, without
// a context, with their Delta / LSE * log2(e) workspace in a file-scope
// device array instead of the context's allocation.
//
// The array lives in every device's copy of the code object, so each GPU the
// library runs on holds it (8 MiB) until the process ends.  Host code never
// passes the array's name to a kernel (on the host it is only a stand-in
// symbol): the device address comes from hipGetSymbolAddress, looked up once
// per device with that device current, and kept.  Every call on one GPU
// shares that GPU's array: calls that overlap on one GPU (other streams, or
// other threads) race on it.  Each call's bwd_pre kernel writes every
// workspace entry its dK/dV and dQ kernels read before they run, and clears
// the dK/dV kernel's tile queues at the end of the array (which that kernel
// leaves zero as well), so nothing else needs clearing between calls.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <string>

#include "sppo.h"
#include "sppo_kernels.h"

namespace {

constexpr size_t kHalf = size_t(1) << 20;  // floats per workspace half: B * Hq * (c1 - c0) <= 2^20
// [Delta | LSE2 | dK/dV tile queues]
__device__ __align__(256) float scratch[2 * kHalf + 64];
static_assert(sppo::kTileQueueInts * sizeof(int) <= 64 * sizeof(float), "tile queues fit the scratch tail");

constexpr int kMaxDevices = 64;
float* g_scratch[kMaxDevices] = {};
int g_n_cu[kMaxDevices] = {};
std::mutex g_scratch_mu;

sppo_status fail(sppo_status st, const std::string& msg) {
  sppo::set_thread_error(msg);
  return st;
}

// Device address of this device's copy of `scratch` and the device's
// compute unit count (looked up on the first call on each device, with that
// device current).
sppo_status scratch_address(float** out, int* n_cu) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SPPO_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(SPPO_ERR_UNSUPPORTED, "device index beyond the scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      return fail(SPPO_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    }
    int cus = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess || cus < 1) {
      return fail(SPPO_ERR_HIP, std::string("compute unit count: ") + hipGetErrorString(e));
    }
    g_n_cu[dev] = cus;
    g_scratch[dev] = static_cast<float*>(p);
  }
  *out = g_scratch[dev];
  *n_cu = g_n_cu[dev];
  return SPPO_OK;
}

bool aligned16(const void* p) { return p && (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

extern "C" sppo_status sppo_attn_bwd_chunk_noalloc(int64_t batch, int64_t seq_len, int64_t c0, int64_t c1,
                                                   int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                                   sppo_dtype dtype, float softmax_scale, int32_t accumulate,
                                                   const void* q_i, const void* k, const void* v, const void* o_i,
                                                   const float* lse_i, const void* do_i, void* dq_i, float* dk_acc,
                                                   float* dv_acc, void* stream) {
  sppo::set_thread_error("");
  if (batch < 1 || batch > 65535 || n_q_heads < 1 || n_q_heads > 65535 || n_kv_heads < 1 ||
      n_q_heads % n_kv_heads != 0) {
    return fail(SPPO_ERR_INVALID_ARG, "need 1 <= batch <= 65535 and n_q_heads (<= 65535) a multiple of n_kv_heads");
  }
  if (seq_len < 1 || seq_len > 0x7fffffff || c0 < 0 || c1 <= c0 || c1 > seq_len) {
    return fail(SPPO_ERR_INVALID_ARG, "need 0 <= c0 < c1 <= seq_len < 2^31");
  }
  if (head_dim != 64 && head_dim != 128) return fail(SPPO_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if ((double)batch * (double)seq_len * (double)std::max(n_q_heads, n_kv_heads) * (double)head_dim * 4.0 > 0x1p62) {
    return fail(SPPO_ERR_UNSUPPORTED, "a [B, S, H, D] tensor of this problem would exceed 2^62 bytes");
  }
  if (dtype != SPPO_F32 && dtype != SPPO_BF16) return fail(SPPO_ERR_INVALID_ARG, "unknown dtype");
  if (!(softmax_scale >= 0.f) || std::isinf(softmax_scale)) {
    return fail(SPPO_ERR_INVALID_ARG, "softmax_scale must be finite and >= 0 (0 = 1/sqrt(D))");
  }
  if (accumulate != 0 && accumulate != 1) return fail(SPPO_ERR_INVALID_ARG, "accumulate must be 0 or 1");
  const void* ptrs[] = {q_i, k, v, o_i, lse_i, do_i, dq_i, dk_acc, dv_acc};
  for (const void* p : ptrs) {
    if (!aligned16(p)) return fail(SPPO_ERR_INVALID_ARG, "a pointer is null or not 16-byte aligned");
  }
  if (dk_acc == dv_acc) return fail(SPPO_ERR_INVALID_ARG, "dk_acc and dv_acc must be distinct buffers");
  const int64_t s = c1 - c0;
  if (batch * n_q_heads * s > (int64_t)kHalf) {
    return fail(SPPO_ERR_UNSUPPORTED, "batch * n_q_heads * (c1 - c0) = " + std::to_string(batch * n_q_heads * s) +
                                          " exceeds the static workspace of " + std::to_string(kHalf) + " rows");
  }
  float* ws = nullptr;
  int n_cu = 0;
  sppo_status st = scratch_address(&ws, &n_cu);
  if (st != SPPO_OK) return st;

  sppo::ChunkArgs a{};
  a.B = batch;
  a.S = seq_len;
  a.c0 = c0;
  a.c1 = c1;
  a.Hq = n_q_heads;
  a.Hkv = n_kv_heads;
  a.D = head_dim;
  a.scale = softmax_scale > 0.f ? softmax_scale : 1.0f / std::sqrt((float)head_dim);
  a.delta = ws;
  a.lse2 = ws + kHalf;
  a.tiles = reinterpret_cast<int*>(ws + 2 * kHalf);
  a.n_cu = n_cu;
  a.kv0 = 0;
  a.kv1 = c1;
  a.q = q_i;
  a.k = k;
  a.v = v;
  a.o = const_cast<void*>(o_i);
  a.lse = const_cast<float*>(lse_i);
  a.dout = do_i;
  a.dq = dq_i;
  a.dk = dk_acc;
  a.dv = dv_acc;
  a.accumulate = accumulate;
  hipStream_t sm = static_cast<hipStream_t>(stream);
  const bool bf16 = dtype == SPPO_BF16;
  hipError_t e = bf16 ? sppo::launch_bwd_pre_bf16(a, sm) : sppo::launch_bwd_pre_f32(a, sm);
  if (e == hipSuccess) e = bf16 ? sppo::launch_bwd_dkdv_bf16(a, sm) : sppo::launch_bwd_dkdv_f32(a, sm);
  if (e == hipSuccess) e = bf16 ? sppo::launch_bwd_dq_bf16(a, sm) : sppo::launch_bwd_dq_f32(a, sm);
  if (e != hipSuccess) return fail(SPPO_ERR_HIP, std::string("backward kernel launch: ") + hipGetErrorString(e));
  return SPPO_OK;
}
