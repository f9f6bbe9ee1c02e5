// C ABI of the full-layer building blocks (GEMM, LayerNorm, GELU, transpose,
// dQKV packing).  Context-free: each call validates its arguments on the
// host, enqueues its kernels on the given stream, and returns a status.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "sppo.h"
#include "sppo_kernels.h"

namespace {

bool al16(const void* p) { return p && (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

sppo_status launched(hipError_t e) { return e == hipSuccess ? SPPO_OK : SPPO_ERR_HIP; }

constexpr int kLnRowsPerBlock = 16;

}  // namespace

extern "C" {

sppo_status sppo_gemm_bf16(int32_t layout, int64_t M, int64_t N, int64_t K, const void* a, int64_t lda,
                           const void* b, int64_t ldb, void* c, int64_t ldc, int32_t epilogue, void* aux,
                           int64_t ldaux, void* stream) {
  if (M <= 0 || N <= 0 || K <= 0) return SPPO_ERR_INVALID_ARG;
  if (!al16(a) || !al16(b) || !al16(c)) return SPPO_ERR_INVALID_ARG;
  if (lda % 8 || ldb % 8 || ldc <= 0 || ldc % 4 || N % 4) return SPPO_ERR_INVALID_ARG;
  if (epilogue < SPPO_EPI_BF16 || epilogue > SPPO_EPI_F32) return SPPO_ERR_INVALID_ARG;
  const bool needs_aux = epilogue == SPPO_EPI_ADD_BF16 || epilogue == SPPO_EPI_GELU || epilogue == SPPO_EPI_DGELU;
  if (needs_aux && (!aux || ldaux < N || ldaux % 4 || (reinterpret_cast<uintptr_t>(aux) & 7))) return SPPO_ERR_INVALID_ARG;
  if (ldc < N) return SPPO_ERR_INVALID_ARG;
  if (layout == SPPO_GEMM_NT) {
    if (K % 64 || lda < K || ldb < K) return SPPO_ERR_INVALID_ARG;
  } else if (layout == SPPO_GEMM_TN) {
    if (M % 256 || N % 256 || lda < M || ldb < N) return SPPO_ERR_INVALID_ARG;
  } else {
    return SPPO_ERR_INVALID_ARG;
  }
  // the epilogue addresses C and aux by 32-bit element offsets
  if (M * ldc >= ((int64_t)1 << 31) || (aux && M * ldaux >= ((int64_t)1 << 31))) return SPPO_ERR_UNSUPPORTED;
  // the DMA byte ranges of one tile fit 32 bits
  if ((layout == SPPO_GEMM_NT ? 256 : 64) * (lda > ldb ? lda : ldb) * 2 > INT32_MAX) return SPPO_ERR_UNSUPPORTED;
  sppo::GemmArgs g{};
  g.M = M; g.N = N; g.K = K;
  g.a = static_cast<const uint16_t*>(a); g.lda = lda;
  g.b = static_cast<const uint16_t*>(b); g.ldb = ldb;
  g.c = c; g.ldc = ldc;
  g.aux = aux; g.ldaux = ldaux;
  g.epi = epilogue;
  g.tn = layout == SPPO_GEMM_TN;
  return launched(sppo::launch_gemm_bf16(g, static_cast<hipStream_t>(stream)));
}

sppo_status sppo_layernorm_fwd(int64_t rows, int32_t H, const void* x, int64_t ldx, const float* gamma,
                               const float* beta, float eps, void* y, int64_t ldy, float* mean, float* rstd,
                               void* stream) {
  if (rows <= 0 || H <= 0 || H % 8 || H > 8192 || ldx < H || ldy < H || ldx % 8 || ldy % 8 || !(eps > 0.f))
    return SPPO_ERR_INVALID_ARG;
  if (!al16(x) || !al16(y) || !gamma || !beta || !mean || !rstd) return SPPO_ERR_INVALID_ARG;
  sppo::LnArgs l{};
  l.rows = rows; l.H = H;
  l.x = static_cast<const uint16_t*>(x); l.ldx = ldx;
  l.y = static_cast<uint16_t*>(y); l.ldy = ldy;
  l.gamma = gamma; l.beta = beta; l.mean = mean; l.rstd = rstd; l.eps = eps;
  return launched(sppo::launch_ln_fwd(l, static_cast<hipStream_t>(stream)));
}

size_t sppo_layernorm_bwd_workspace(int64_t rows, int32_t H) {
  if (rows <= 0 || H <= 0) return 0;
  const int64_t nb = (rows + kLnRowsPerBlock - 1) / kLnRowsPerBlock;
  return (size_t)nb * 2 * (size_t)H * sizeof(float);
}

sppo_status sppo_layernorm_bwd(int64_t rows, int32_t H, const void* x, int64_t ldx, const float* gamma,
                               const float* mean, const float* rstd, const void* dy, int64_t lddy,
                               const void* dres, int64_t lddres, void* dx, int64_t lddx, float* dgamma,
                               float* dbeta, int32_t accumulate, float* workspace, size_t workspace_bytes,
                               void* stream) {
  if (rows <= 0 || H <= 0 || H % 8 || H > 8192) return SPPO_ERR_INVALID_ARG;
  if (ldx < H || lddy < H || lddres < H || lddx < H || ldx % 8 || lddy % 8 || lddres % 8 || lddx % 8)
    return SPPO_ERR_INVALID_ARG;
  if (!al16(x) || !al16(dy) || !al16(dres) || !al16(dx) || !gamma || !mean || !rstd || !dgamma || !dbeta ||
      !workspace)
    return SPPO_ERR_INVALID_ARG;
  if (workspace_bytes < sppo_layernorm_bwd_workspace(rows, H)) return SPPO_ERR_INVALID_ARG;
  sppo::LnArgs l{};
  l.rows = rows; l.H = H;
  l.x = static_cast<const uint16_t*>(x); l.ldx = ldx;
  l.y = static_cast<uint16_t*>(dx); l.ldy = lddx;
  l.gamma = gamma;
  l.mean = const_cast<float*>(mean); l.rstd = const_cast<float*>(rstd);
  l.dy = static_cast<const uint16_t*>(dy); l.lddy = lddy;
  l.dres = static_cast<const uint16_t*>(dres); l.lddres = lddres;
  l.dgamma = dgamma; l.dbeta = dbeta; l.part = workspace;
  l.rows_per_block = kLnRowsPerBlock;
  l.accumulate = accumulate != 0;
  return launched(sppo::launch_ln_bwd(l, static_cast<hipStream_t>(stream)));
}

sppo_status sppo_gelu_bf16(const void* x, void* y, int64_t n, void* stream) {
  if (n <= 0 || n % 8 || !al16(x) || !al16(y)) return SPPO_ERR_INVALID_ARG;
  return launched(sppo::launch_gelu(static_cast<const uint16_t*>(x), static_cast<uint16_t*>(y), n,
                                    static_cast<hipStream_t>(stream)));
}

sppo_status sppo_transpose_bf16(const void* in, void* out, int64_t rows, int64_t cols, void* stream) {
  if (rows <= 0 || cols <= 0 || !in || !out || in == out) return SPPO_ERR_INVALID_ARG;
  return launched(sppo::launch_transpose(static_cast<const uint16_t*>(in), static_cast<uint16_t*>(out), rows, cols,
                                         static_cast<hipStream_t>(stream)));
}

sppo_status sppo_pack_qkv_grad(int64_t rows, int32_t wq, int32_t wkv, const void* dq, const float* dk,
                               const float* dv, int64_t row0, void* out, void* stream) {
  if (rows <= 0 || wq <= 0 || wkv <= 0 || wq % 8 || wkv % 8 || row0 < 0) return SPPO_ERR_INVALID_ARG;
  if (!al16(dq) || !al16(dk) || !al16(dv) || !al16(out)) return SPPO_ERR_INVALID_ARG;
  sppo::PackArgs p{};
  p.rows = rows; p.wq = wq; p.wkv = wkv;
  p.dq = static_cast<const uint16_t*>(dq); p.dk = dk; p.dv = dv; p.c = row0;
  p.out = static_cast<uint16_t*>(out);
  return launched(sppo::launch_pack_dqkv(p, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
