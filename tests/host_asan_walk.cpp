// Host-code exercise of libsppo under AddressSanitizer (host code only; the
// device code is built as usual): every C-ABI path of the attention walk
// (row-prefix offload with keep buffers, extra planes, B = 2, ragged chunks,
// K/V eviction, finalize, an abandoned walk and reset, timing, stats, the
// link probe, an order error), the no-alloc backward, the pure host
// functions and the argument checks.  It needs a GPU.  Build and run from the
// repository root:
//
//   for f in paper_2503_10377_amd/csrc/*.hip paper_2503_10377_amd/csrc/*.cpp tests/host_asan_walk.cpp; do
//     x=""; case $f in *attn_*_bf16.hip) x="-mllvm -amdgpu-mfma-vgpr-form";; esac
//     l=""; case $f in *.hip) l="-x hip";; esac
//     hipcc -O1 -g -std=c++17 --offload-arch=gfx950 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       -Xarch_host -fsanitize=address -Xarch_host -fno-omit-frame-pointer \
//       -I include -I paper_2503_10377_amd/csrc $x $l -c $f -o /tmp/asan_$(basename $f).o
//   done
//   hipcc --offload-arch=gfx950 -Xarch_host -fsanitize=address /tmp/asan_*.o -o /tmp/host_asan_walk
//   ASAN_OPTIONS=detect_leaks=0 /tmp/host_asan_walk
//
// It prints "all ok" and exits 0 when every call returns as documented.
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>
#include <vector>
#include "sppo.h"

#define CK(x) do { sppo_status s_ = (x); if (s_ != SPPO_OK) { std::printf("FAIL %s -> %s: %s\n", #x, sppo_status_string(s_), sppo_last_error(ctx)); std::exit(1);} } while (0)
#define HK(x) do { hipError_t e_ = (x); if (e_ != hipSuccess) { std::printf("HIP FAIL %s\n", #x); std::exit(1);} } while (0)

static void* dalloc(size_t n) { void* p = nullptr; HK(hipMalloc(&p, n)); HK(hipMemset(p, 0, n)); return p; }

int main() {
  sppo_ctx* ctx = nullptr;
  // ---- argument checks (nothing allocated on failure)
  sppo_problem bad{};
  if (sppo_create(&bad, &ctx) == SPPO_OK) { std::printf("FAIL bad problem accepted\n"); return 1; }
  bad.batch = 1; bad.seq_len = 100; bad.n_chunks = 3; bad.n_q_heads = 3; bad.n_kv_heads = 2; bad.head_dim = 128;
  if (sppo_create(&bad, &ctx) == SPPO_OK) { std::printf("FAIL Hq%%Hkv accepted\n"); return 1; }
  std::printf("arg checks ok: %s\n", sppo_last_error(nullptr));

  // ---- pure host functions
  std::vector<int64_t> offs(9);
  CK(sppo_balanced_offsets(4096, 8, 64, offs.data()));
  std::vector<double> tov(8, 0.01);
  std::vector<int64_t> rows(8);
  CK(sppo_plan_offload_rows(offs.data(), 8, 4096.0, 50.0, tov.data(), 64, rows.data()));

  for (int evict = 0; evict < 2; ++evict) {
    const int64_t B = 2, S = 1000;
    const int N = 4, Hq = 4, Hkv = 2, D = 128;
    const int64_t off[5] = {0, 77, 300, 301, 1000};
    const size_t xrb[2] = {512, 8};
    sppo_problem p{};
    p.batch = B; p.seq_len = S; p.n_chunks = N; p.chunk_offsets = off; p.n_q_heads = Hq; p.n_kv_heads = Hkv;
    p.head_dim = D; p.dtype = SPPO_BF16; p.softmax_scale = 0.f;
    p.offload = evict ? SPPO_OFFLOAD_QKVOL_EVICT : SPPO_OFFLOAD_QKVOL; p.n_extra = 2; p.extra_row_bytes = xrb;
    CK(sppo_create(&p, &ctx));
    CK(sppo_set_kernel_timing(ctx, 1));
    const int64_t rows_i[4] = {40, 0, 1, 699};
    for (int i = 0; i < N; ++i) CK(sppo_set_offload_rows(ctx, i, rows_i[i]));
    void* k = dalloc(B * S * Hkv * D * 2); void* v = dalloc(B * S * Hkv * D * 2);
    float* dk = (float*)dalloc(B * S * Hkv * D * 4); float* dv = (float*)dalloc(B * S * Hkv * D * 4);
    void* dk16 = dalloc(B * S * Hkv * D * 2); void* dv16 = dalloc(B * S * Hkv * D * 2);
    std::vector<void*> q(N), o(N), dO(N), dq(N), keep(N), x0(N), x1(N);
    std::vector<float*> lse(N);
    for (int i = 0; i < N; ++i) {
      const int64_t s = off[i + 1] - off[i];
      q[i] = dalloc(B * s * Hq * D * 2); o[i] = dalloc(B * s * Hq * D * 2); dO[i] = dalloc(B * s * Hq * D * 2);
      dq[i] = dalloc(B * s * Hq * D * 2); lse[i] = (float*)dalloc(B * Hq * s * 4);
      x0[i] = dalloc(B * s * xrb[0]); x1[i] = dalloc(B * s * xrb[1]);
      const size_t kb = sppo_keep_bytes(ctx, i);
      keep[i] = kb ? dalloc(kb) : nullptr;
    }
    for (int walk = 0; walk < 2; ++walk) {
      for (int i = 0; i < N; ++i) {
        CK(sppo_attn_fwd_chunk(ctx, i, q[i], k, v, o[i], lse[i], nullptr));
        if (i < N - 1) {
          void* ex[2] = {x0[i], x1[i]};
          sppo_chunk_bufs b{q[i], o[i], lse[i], k, v, ex, keep[i]};
          CK(sppo_offload_issue(ctx, i, &b, nullptr));
          CK(sppo_offload_wait(ctx, i, nullptr));
        }
      }
      if (evict) for (int j = N - 2; j >= 0; --j) CK(sppo_prefetch_kv(ctx, j, k, v, nullptr));
      for (int i = N - 1; i >= 0; --i) {
        if (i < N - 1) {
          void* ex[2] = {x0[i], x1[i]};
          sppo_chunk_bufs b{q[i], o[i], lse[i], nullptr, nullptr, ex, keep[i]};
          CK(sppo_prefetch(ctx, i, &b, nullptr));
          CK(sppo_prefetch_wait(ctx, i, nullptr));
        }
        CK(sppo_attn_bwd_chunk(ctx, i, q[i], k, v, o[i], lse[i], dO[i], dq[i], dk, dv, nullptr));
        CK(sppo_attn_finalize_chunk(ctx, i, dk, dv, dk16, dv16, nullptr));
      }
    }
    // an abandoned walk, then reset
    CK(sppo_attn_fwd_chunk(ctx, 0, q[0], k, v, o[0], lse[0], nullptr));
    CK(sppo_reset(ctx));
    sppo_copy_stats_t cs{}; CK(sppo_copy_stats(ctx, &cs, 1));
    sppo_kernel_times_t kt{}; CK(sppo_kernel_times(ctx, &kt, 1));
    std::vector<int64_t> got(N + 1); CK(sppo_get_offsets(ctx, got.data(), N + 1)); CK(sppo_get_offload_rows(ctx, got.data(), N));
    sppo_link_rates_t lr{}; CK(sppo_link_probe(ctx, 1 << 20, &lr));
    // order error path
    if (sppo_attn_bwd_chunk(ctx, 0, q[0], k, v, o[0], lse[0], dO[0], dq[0], dk, dv, nullptr) != SPPO_ERR_ORDER) {
      std::printf("FAIL order check\n"); return 1;
    }
    HK(hipDeviceSynchronize());
    std::printf("walk %s ok: d2h %llu B, h2d %llu B, fwd %d launches\n", evict ? "evict" : "qkvol",
                (unsigned long long)cs.bytes_d2h, (unsigned long long)cs.bytes_h2d, kt.launches[0]);
    CK(sppo_destroy(ctx)); ctx = nullptr;
    for (int i = 0; i < N; ++i) {
      for (void* ptr : {q[i], o[i], dO[i], dq[i], (void*)lse[i], x0[i], x1[i], keep[i]}) if (ptr) HK(hipFree(ptr));
    }
    for (void* ptr : {k, v, (void*)dk, (void*)dv, dk16, dv16}) HK(hipFree(ptr));
  }
  // ---- no-alloc backward
  {
    const int64_t S = 512, c0 = 256, c1 = 512; const int Hq = 2, Hkv = 1, D = 64;
    void* q = dalloc((c1 - c0) * Hq * D * 2); void* o = dalloc((c1 - c0) * Hq * D * 2);
    void* dO = dalloc((c1 - c0) * Hq * D * 2); void* dq = dalloc((c1 - c0) * Hq * D * 2);
    float* lse = (float*)dalloc(Hq * (c1 - c0) * 4);
    void* k = dalloc(S * Hkv * D * 2); void* v = dalloc(S * Hkv * D * 2);
    float* dk = (float*)dalloc(S * Hkv * D * 4); float* dv = (float*)dalloc(S * Hkv * D * 4);
    CK(sppo_attn_bwd_chunk_noalloc(1, S, c0, c1, Hq, Hkv, D, SPPO_BF16, 0.f, 0, q, k, v, o, lse, dO, dq, dk, dv, nullptr));
    HK(hipDeviceSynchronize());
    for (void* ptr : {q, o, dO, dq, (void*)lse, k, v, (void*)dk, (void*)dv}) HK(hipFree(ptr));
    std::printf("noalloc ok\n");
  }
  std::printf("all ok\n");
  return 0;
}
