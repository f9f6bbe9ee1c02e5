/*
 * libsppo -- sequence-chunked causal attention (forward + backward) with
 * per-chunk activation offload to pinned host memory, for one MI355X (gfx950).
 *
 * The method is the single-GPU slice of Sequence Pipeline Parallel Offloading
 * (SPPO, arXiv 2503.10377):
 *   - The sequence of length S is split into N subsequences ("chunks") with
 *     offsets c_0 = 0 < c_1 < ... < c_N = S (notation table: S, N, s_i).
 *   - A query of chunk i attends to the keys/values of chunks 0..i
 *     (Sec. 5.1, two-level activation management): every earlier chunk is
 *     fully visible, the diagonal block carries the causal mask.  Keys and
 *     values are the "skeletal" tensors and stay resident on the GPU.
 *   - The other saved activations of chunk i (here Q_i, O_i, LSE_i, and
 *     optionally a host copy of K_i/V_i) are offloaded to host memory while
 *     the next chunk computes, and must be back on the device before the
 *     backward of chunk i begins (Sec. 5.1, Sec. 5.2); page-locked host
 *     buffers give the full host-link bandwidth (Sec. 7, implementation).
 *   - The backward walks the chunks in reverse order and accumulates dK/dV.
 *
 * Layout (token-major BSHD, all tensors contiguous, device pointers unless
 * stated otherwise, every pointer 16-byte aligned):
 *   chunk-local  Q_i, O_i, dO_i, dQ_i : [B, s_i, Hq, D]   dtype of the problem
 *   chunk-local  LSE_i                : [B, Hq, s_i]      fp32, natural log
 *   full-length  K, V                 : [B, S, Hkv, D]    dtype of the problem
 *   full-length  dK, dV accumulators  : [B, S, Hkv, D]    fp32
 * Query head h reads KV head h / (Hq / Hkv).  With B = 1, chunk i of a full
 * [1, S, H, D] tensor is the contiguous slab starting at row c_i.
 *
 * Threading and streams: a context is used from one host thread at a time.
 * Every call is asynchronous with respect to the host on the stream it is
 * given (a hipStream_t passed as void*; NULL is the legacy null stream),
 * except sppo_copy_stats, sppo_sync and sppo_destroy, which block.  All
 * backward calls of one context must be issued on one stream (they share the
 * context's Delta workspace).
 *
 * Errors: every call returns an sppo_status.  Arguments are validated on the
 * host before anything is enqueued; a failed call enqueues nothing.  A HIP
 * error maps to SPPO_ERR_HIP; asynchronous device faults surface at the next
 * call that synchronises.  sppo_last_error() holds a message for the last
 * failure of that context.  Nothing aborts or throws across this ABI.
 */
#ifndef SPPO_H
#define SPPO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sppo_ctx sppo_ctx;

typedef enum {
  SPPO_OK = 0,
  SPPO_ERR_INVALID_ARG = 1, /* null/misaligned pointer, bad shape, bad index */
  SPPO_ERR_UNSUPPORTED = 2, /* valid but not implemented (e.g. head_dim)     */
  SPPO_ERR_ORDER = 3,       /* fwd not 0..N-1, or bwd not N-1..0           */
  SPPO_ERR_STATE = 4,       /* e.g. prefetch of a chunk never offloaded    */
  SPPO_ERR_OOM = 5,         /* device or pinned host allocation failed     */
  SPPO_ERR_HIP = 6          /* a HIP runtime call failed                   */
} sppo_status;

typedef enum { SPPO_F32 = 0, SPPO_BF16 = 1 } sppo_dtype;

/* Which saved activations of a chunk travel to host memory after its
 * forward (two-level activation management, Sec. 5.1).  In the first three
 * modes K/V stay resident on the device as the skeletal level. */
typedef enum {
  SPPO_OFFLOAD_NONE = 0,  /* nothing leaves the device                      */
  SPPO_OFFLOAD_QOL = 1,   /* Q_i, O_i, LSE_i offloaded and prefetched back  */
  SPPO_OFFLOAD_QKVOL = 2, /* as QOL, plus a host copy of K_i and V_i; the
                             resident K/V cache is not re-fetched           */
  SPPO_OFFLOAD_QKVOL_EVICT = 3
                          /* as QKVOL, but once the forward walk is over the
                             K/V cache rows of offloaded chunks count as
                             evicted (the caller may reuse that memory
                             after sppo_offload_wait): they come back with
                             sppo_prefetch_kv, and the backward of the last
                             chunk, the only one that runs before all of
                             them are back, does its dK/dV work one KV
                             chunk at a time, each piece waiting only for
                             its own rows, so the K/V copies stream in
                             under it                                      */
} sppo_offload;

/* The problem, in the paper's notation (B, S, N, s_i) plus the attention
 * shape (query heads, KV heads, head dim).  Copied by sppo_create, which
 * returns UNSUPPORTED when B or a head count exceeds 65535 or a
 * [B, S, max(Hq, Hkv), D] tensor would exceed 2^62 bytes. */
typedef struct {
  int64_t batch;                 /* B >= 1                                  */
  int64_t seq_len;               /* 1 <= S < 2^31 (kernels index keys in int) */
  int32_t n_chunks;              /* N, 1 <= N <= S                          */
  const int64_t* chunk_offsets;  /* host array of N+1 offsets, strictly
                                    increasing from 0 to S; NULL means N
                                    equal chunks (requires S % N == 0)      */
  int32_t n_q_heads;             /* Hq >= 1                                 */
  int32_t n_kv_heads;            /* Hkv >= 1, Hq % Hkv == 0                 */
  int32_t head_dim;              /* D in {64, 128}                          */
  sppo_dtype dtype;              /* element type of Q, K, V, O, dO, dQ      */
  float softmax_scale;           /* 0 means 1/sqrt(D)                       */
  sppo_offload offload;          /* offload set; NONE allocates no host mem */
  int32_t n_extra;               /* 0..16 further saved-activation planes
                                    that travel with Q/O/LSE (the rest of a
                                    full layer's saved tensors, Sec. 5.1:
                                    everything but K/V is offloadable)      */
  const size_t* extra_row_bytes; /* host array of n_extra row sizes (bytes
                                    per token, positive multiples of 4);
                                    plane k of chunk i is a
                                    chunk-local [B, s_i, extra_row_bytes[k]]
                                    byte array; NULL when n_extra == 0      */
} sppo_problem;

/* Device pointers of one chunk's saved activations, for offload/prefetch. */
typedef struct {
  void* q;      /* Q_i   [B, s_i, Hq, D]  chunk-local                        */
  void* o;      /* O_i   [B, s_i, Hq, D]  chunk-local                        */
  float* lse;   /* LSE_i [B, Hq, s_i]     chunk-local                        */
  void* k;      /* base of the full K cache [B, S, Hkv, D]; rows of chunk i  */
  void* v;      /* base of the full V cache [B, S, Hkv, D]; rows of chunk i  */
  void* const* extra; /* n_extra device pointers (planes of chunk i), or
                         NULL when the problem has no extra planes          */
  void* keep;   /* device buffer of sppo_keep_bytes(ctx, i) bytes, 16-byte
                   aligned, or NULL.  With sequence-aware offloading (rows_i
                   < s_i, see sppo_set_offload_rows) the rows [rows_i, s_i)
                   of Q_i, O_i, LSE_i and the extra planes stay on the
                   device.  With a keep buffer, sppo_offload_issue moves
                   them there (a copy kernel on its stream), so
                   the source buffers are dead as a whole after
                   sppo_offload_wait and can be reused (a device staging
                   ring), and sppo_prefetch moves them back into its
                   destination buffers (a copy kernel on its stream) -- pass the same
                   keep pointer to both.  Without one, they stay in the
                   source buffers, and the prefetch must target those same
                   buffers.  Ignored when rows_i == s_i.  The caller owns
                   the buffer and keeps it untouched from the offload to
                   the prefetch of chunk i.                                 */
} sppo_chunk_bufs;

typedef struct {
  uint64_t bytes_d2h;    /* bytes copied device->host since create/reset  */
  uint64_t bytes_h2d;    /* bytes copied host->device                     */
  double ms_d2h;         /* sum over chunks of event-timed D2H durations   */
  double ms_h2d;         /* sum over chunks of event-timed H2D durations   */
  int32_t n_d2h;         /* chunks offloaded                               */
  int32_t n_h2d;         /* chunks prefetched                              */
} sppo_copy_stats_t;

/* Kernels of one chunk, for per-kernel timing. */
typedef enum {
  SPPO_KERNEL_FWD = 0,       /* forward of a chunk                          */
  SPPO_KERNEL_BWD_PRE = 1,   /* Delta = rowsum(dO * O)                      */
  SPPO_KERNEL_BWD_DKDV = 2,  /* dK/dV accumulation over the chunk's queries */
  SPPO_KERNEL_BWD_DQ = 3,    /* dQ of the chunk                             */
  SPPO_KERNEL_COUNT = 4
} sppo_kernel;

typedef struct {
  double ms[SPPO_KERNEL_COUNT];         /* summed event-timed durations     */
  int32_t launches[SPPO_KERNEL_COUNT];  /* launches timed                   */
} sppo_kernel_times_t;

/* Create a context: validates the problem, copies the offsets, allocates
 * the Delta workspace (fp32 [B, Hq, max s_i]) on the current device and
 * per-chunk events, takes a reference on the device's two copy streams
 * (device->host and host->device, default priority, created by the first
 * context on the device and shared by all of its contexts, so the library
 * adds two streams to a process however many contexts it has), and --
 * unless offload is NONE -- allocates page-locked host slots for every
 * chunk's offload set.
 * *out is set only on success.  Errors: INVALID_ARG, UNSUPPORTED, OOM, HIP. */
sppo_status sppo_create(const sppo_problem* problem, sppo_ctx** out);

/* Synchronise the copy streams (which also waits for copies that other
 * contexts on the device have enqueued) and free everything the context
 * owns (the copy streams go when the last context on the device is
 * destroyed).  Safe on NULL. */
sppo_status sppo_destroy(sppo_ctx* ctx);

/* Forward of chunk i (Sec. 5.1): for rows r in [c_i, c_{i+1}) and every
 * query head, O_i[r] = softmax over keys j <= r (global positions) of
 * scale * Q_i[r].K[j], applied to V; LSE_i[r] = log sum_j exp(scale*Q.K).
 * Reads K/V rows [0, c_{i+1}).  Calls must come in order i = 0..N-1 (the
 * first call after create, after sppo_reset, or after bwd(0) must be
 * i = 0); otherwise ORDER and nothing is enqueued. */
sppo_status sppo_attn_fwd_chunk(sppo_ctx* ctx, int32_t i, const void* q_i,
                                const void* k, const void* v, void* o_i,
                                float* lse_i, void* stream);

/* Backward of chunk i in the reverse walk (Sec. 5.2): with Delta_r =
 * <dO_r, O_r>, P = exp(scale*Q.K - LSE), dS = P (dO.V - Delta):
 *   dQ_i = scale * dS K                         (written)
 *   dK[0, c_{i+1}) += scale * dS^T Q_i,  dV[0, c_{i+1}) += P^T dO_i
 * For i = N-1 (the first backward call) dK/dV rows [0, S) are overwritten,
 * so the accumulators need no zeroing; rows >= c_{i+1} are never touched.
 * Calls must come in order i = N-1..0 after fwd(N-1).  If chunk i was
 * offloaded, the stream first waits for the prefetch of chunk i, which must
 * have been issued (otherwise STATE).  With QKVOL_EVICT, bwd(N-1) requires
 * sppo_prefetch_kv of every offloaded chunk (otherwise STATE) and runs its
 * dK/dV kernel once per KV chunk j = N-1..0, each launch after chunk j's
 * K/V-ready event, then dQ. */
sppo_status sppo_attn_bwd_chunk(sppo_ctx* ctx, int32_t i, const void* q_i,
                                const void* k, const void* v, const void* o_i,
                                const float* lse_i, const void* do_i,
                                void* dq_i, float* dk_acc, float* dv_acc,
                                void* stream);

/* Offload chunk i's saved activations (the set chosen by problem.offload)
 * from the device pointers in *src to the context's pinned host slot i.
 * Records an event on `stream` (after the fwd of chunk i); the context's
 * D2H stream waits for it, copies, and records the chunk's offload-done
 * event.  The device sources must not be overwritten until that event --
 * see sppo_offload_wait.  Requires fwd(i) issued, offload != NONE. */
sppo_status sppo_offload_issue(sppo_ctx* ctx, int32_t i,
                               const sppo_chunk_bufs* src, void* stream);

/* Make `stream` wait until chunk i's offload copies have completed (its
 * device buffers may then be reused or overwritten).  Requires the offload
 * of chunk i to have been issued. */
sppo_status sppo_offload_wait(sppo_ctx* ctx, int32_t i, void* stream);

/* Prefetch chunk i's offloaded Q/O/LSE from host slot i into the device
 * pointers in *dst (K/V are never re-fetched: the cache is resident).  The
 * H2D stream waits for an event recorded now on `stream` (so dst may be
 * written after everything already enqueued there) and for chunk i's
 * offload-done event; the backward of chunk i then waits for the copy.
 * Requires the offload of chunk i to have been issued. */
sppo_status sppo_prefetch(sppo_ctx* ctx, int32_t i, const sppo_chunk_bufs* dst,
                          void* stream);

/* QKVOL_EVICT only: copy chunk i's K_i/V_i rows from host slot i back into
 * the device K/V cache (k, v: base pointers of the full [B, S, Hkv, D]
 * tensors) on the context's H2D stream, after everything already enqueued
 * on `stream` and after chunk i's offload has completed, and record chunk
 * i's K/V-ready event.  Allowed once the forward walk is over (in_bwd) and
 * before the backward of chunk N-1, which requires it for every offloaded
 * chunk and waits for chunk j's K/V-ready event right before the dK/dV work
 * on chunk j's key rows.  Errors: STATE (other mode, forward walk not over,
 * chunk not offloaded, already prefetched, backward already started),
 * INVALID_ARG. */
sppo_status sppo_prefetch_kv(sppo_ctx* ctx, int32_t i, void* k, void* v, void* stream);

/* Sequence-aware offloading (Sec. 5.2, adaptive offloading ratio alpha_i):
 * offload only the first `rows` rows (0 <= rows <= s_i) of chunk i's
 * offload set -- a row prefix of Q_i, O_i, LSE_i (and of K_i/V_i with
 * QKVOL*) -- and keep the rest resident; alpha_i = rows / s_i.  The default
 * is rows = s_i.  offload_issue, prefetch and prefetch_kv of chunk i then
 * move that prefix only (rows = 0 moves nothing but still orders the
 * streams).  Allowed only between walks (after create, reset or bwd(0)).
 * Errors: INVALID_ARG (index, rows out of range), STATE (mid-walk). */
sppo_status sppo_set_offload_rows(sppo_ctx* ctx, int32_t i, int64_t rows);

/* The offloaded row prefix of every chunk (n_chunks values). */
sppo_status sppo_get_offload_rows(const sppo_ctx* ctx, int64_t* out, int32_t capacity);

/* FLOPs-balanced partition (Sec. 3, computation imbalance of causal
 * attention; Sec. 5.2, FLOPs-based partition): chunk k of a causal
 * sequence covers about S^2 (2k+1) / (2N^2) of the S^2/2 visible (query,
 * key) pairs, so equal work per chunk needs c_k = S sqrt(k/N): long chunks
 * first, shorter ones later.  Writes N+1 offsets to out, each interior
 * offset rounded to a multiple of `align` and every chunk at least `align`
 * rows long.  Pure host function.  Errors: INVALID_ARG (S < N * align,
 * null out, N < 1, align < 1). */
sppo_status sppo_balanced_offsets(int64_t seq_len, int32_t n_chunks, int64_t align, int64_t* out);

/* Offload plan of sequence-aware offloading (Sec. 5.2): the copy of chunk i
 * should take no longer than the compute it overlaps, t_overlap_ms[i]
 * (normally the forward of chunk i+1), so with a device->host rate of
 * bw_GBps and bytes_per_row bytes of offload set per token row,
 *   rows_i = min(s_i, floor(bw * t_overlap_i / bytes_per_row)),
 * rounded down to a multiple of `align` when below s_i; the last chunk gets
 * rows = 0.  alpha_i = rows_i / s_i; alpha_i * A_i is then bounded by the
 * bytes the link moves in t_overlap_i.  Pure host function.  Errors:
 * INVALID_ARG. */
sppo_status sppo_plan_offload_rows(const int64_t* offsets, int32_t n_chunks, double bytes_per_row,
                                   double bw_GBps, const double* t_overlap_ms, int64_t align,
                                   int64_t* rows_out);

/* Bytes of chunk i's keep buffer (see sppo_chunk_bufs.keep) for its
 * current offload row count: 0 when the whole chunk is offloaded, or for an
 * invalid context or index. */
size_t sppo_keep_bytes(const sppo_ctx* ctx, int32_t i);

/* Finalize step of the reverse walk (optional): key j receives gradient
 * only from query rows r >= j, and the walk runs the backward of chunks
 * N-1, ..., 0 (Sec. 5.2), so once bwd(i) has been issued the dK/dV rows
 * [c_i, c_{i+1}) are final.  Writes those rows of every batch entry of
 * dk_out/dv_out ([B, S, Hkv, D] in the problem's dtype: fp32 accumulators
 * rounded to nearest even for bf16, copied for fp32) on `stream`, after
 * the backward enqueued there.  Rows outside the chunk are not touched.
 * Errors: STATE (bwd(i) not issued since the last fwd(0) or reset),
 * INVALID_ARG (null/misaligned pointers, dk_out == dv_out). */
sppo_status sppo_attn_finalize_chunk(sppo_ctx* ctx, int32_t i, const float* dk_acc, const float* dv_acc,
                                     void* dk_out, void* dv_out, void* stream);

/* Abandon the current forward/backward walk (e.g. after a forward-only run):
 * the next call must be fwd(0).  Blocks until the device's copy streams are
 * idle (copies of the abandoned walk may still read or write its device
 * buffers and host slots; the streams are shared, so this also waits for
 * copies other contexts have enqueued), then clears per-chunk offload state. */
sppo_status sppo_reset(sppo_ctx* ctx);

/* Block until the context's copy streams are idle. */
sppo_status sppo_sync(sppo_ctx* ctx);

/* Synchronise the copy streams and return cumulative copy statistics;
 * `reset_after` != 0 zeroes them afterwards. */
sppo_status sppo_copy_stats(sppo_ctx* ctx, sppo_copy_stats_t* out, int32_t reset_after);

/* Host-link rates of the context's own copy path, measured in isolation
 * (the "T_copy_iso" of the offload-hidden figure): allocates a device buffer
 * and a page-locked host buffer of `bytes` each, then times, on the
 * context's copy streams with events, one device->host copy, one
 * host->device copy, and both at once; frees the buffers and returns GB/s
 * (1e9 bytes per second).  Blocks the host.  Errors: INVALID_ARG (bytes <
 * 1 MiB), OOM, HIP. */
typedef struct {
  double d2h_GBps;     /* device->host alone                               */
  double h2d_GBps;     /* host->device alone                               */
  double duplex_GBps;  /* both directions at once, bytes of both / time    */
} sppo_link_rates_t;
sppo_status sppo_link_probe(sppo_ctx* ctx, size_t bytes, sppo_link_rates_t* out);

/* Enable (1) or disable (0) per-kernel timing: while enabled, every kernel
 * launch is bracketed by two events on the caller's stream.  Creates the
 * events on first use. */
sppo_status sppo_set_kernel_timing(sppo_ctx* ctx, int32_t enable);

/* Wait for the timed kernels and return the summed durations and launch
 * counts per kernel since the last reset; `reset_after` != 0 zeroes them. */
sppo_status sppo_kernel_times(sppo_ctx* ctx, sppo_kernel_times_t* out, int32_t reset_after);

/* The stream waits until chunk i's prefetch (sppo_prefetch) has landed, for
 * work other than the attention backward (which waits by itself) that
 * reads the prefetched tensors, e.g. the rest of a layer's backward.
 * STATE if chunk i's prefetch was not issued. */
sppo_status sppo_prefetch_wait(sppo_ctx* ctx, int32_t i, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * backward of one chunk [c0, c1) as sppo_attn_bwd_chunk enqueues it (same
 * kernels, same results bit for bit), without a context and without any
 * allocation.  Its Delta / LSE workspace and the dK/dV kernel's tile
 * queues are a static device array of the library (8 MiB on every GPU the
 * library runs on, held until the process ends; the queues are cleared by
 * each call and left zero), so batch * n_q_heads * (c1 - c0) must not
 * exceed 2^20 (UNSUPPORTED otherwise, as for the size limits of
 * sppo_create).  Every call on one GPU shares that GPU's array: calls that
 * overlap on one GPU (several streams or threads) race, so the caller
 * orders them (e.g. one stream).  Arguments as in sppo_create and
 * sppo_attn_bwd_chunk: q_i, o_i, do_i, dq_i [B, c1 - c0, Hq, D] and lse_i
 * [B, Hq, c1 - c0] chunk-local; k, v [B, S, Hkv, D]; dk_acc, dv_acc fp32
 * [B, S, Hkv, D], rows [0, c1) overwritten (accumulate = 0) or added to
 * (accumulate = 1), rows >= c1 untouched.  No call-order checks (there is
 * no walk state).  Errors: INVALID_ARG, UNSUPPORTED, HIP, with the message
 * in sppo_last_error(NULL) on the calling thread. */
sppo_status sppo_attn_bwd_chunk_noalloc(int64_t batch, int64_t seq_len, int64_t c0, int64_t c1,
                                        int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                        sppo_dtype dtype, float softmax_scale, int32_t accumulate,
                                        const void* q_i, const void* k, const void* v, const void* o_i,
                                        const float* lse_i, const void* do_i, void* dq_i, float* dk_acc,
                                        float* dv_acc, void* stream);

/* Chunk offsets as stored by the context (n_chunks + 1 values). */
sppo_status sppo_get_offsets(const sppo_ctx* ctx, int64_t* out, int32_t capacity);

/* Message for the last failure of this context ("" if none); with
 * ctx == NULL, the message of the last failed sppo_create or context-free
 * attention call on this thread. */
const char* sppo_last_error(const sppo_ctx* ctx);

/* Static name of a status code. */
const char* sppo_status_string(sppo_status s);

/* ------------------------------------------------------------------------
 * Full-layer building blocks.  A transformer layer chunk (Sec. 5.1: the
 * subsequence's tensors of one layer -- LayerNorm, the QKV projection,
 * attention, the output projection and the MLP; Sec. 3.3: attention and the
 * GEMMs are the compute-bound operators) is composed from the attention
 * calls above and the calls below.  They need no context: each validates
 * its arguments on the host, enqueues on `stream` and returns a status
 * (INVALID_ARG, UNSUPPORTED or HIP); nothing is enqueued on failure.
 * Activations are bf16, statistics and parameter gradients fp32, every
 * pointer a device pointer, 16-byte aligned where it is bf16 data, every
 * leading dimension (ld*, in elements) a multiple of 8.
 * ---------------------------------------------------------------------- */

/* C[M, N] (op)= sum_k A(m, k) B(k, n), bf16 operands, fp32 accumulation.
 *   SPPO_GEMM_NT: A is [M, K] (row stride lda), B is [N, K] (ldb), so
 *                 C = A B^T; K % 64 == 0.  x W = x (W^T)^T with W^T
 *                 [out, in], and dY W^T with W [in, out].
 *   SPPO_GEMM_TN: A is stored [K, M], B stored [K, N], so C = A^T B;
 *                 M % 256 == 0, N % 256 == 0.  The weight gradient X^T dY.
 * Rows past M (NT) or K (TN) read as zero, only C[m < M][n < N] is
 * written.  Epilogues (aux: bf16 [M, N] with row stride ldaux):
 *   BF16      C = acc (bf16)
 *   ADD_BF16  C = acc + aux (bf16): the residual add
 *   GELU      aux = bf16(acc) (the pre-activation, kept for the backward),
 *             C = gelu(aux) with gelu(a) = a/2 (1 + tanh(sqrt(2/pi)(a +
 *             0.044715 a^3)))
 *   DGELU     C = acc * gelu'(aux) (bf16)
 *   ACC_F32   C += acc (fp32): gradients accumulated over chunks
 *   F32       C = acc (fp32)
 * N, ldc and ldaux must be multiples of 4 and aux 8-byte aligned (the
 * epilogues use 8- and 16-byte vector accesses): SPPO_ERR_INVALID_ARG
 * otherwise.  M * ldc and M * ldaux must stay below 2^31 elements (the
 * epilogue addresses C and aux by 32-bit element offsets):
 * SPPO_ERR_UNSUPPORTED otherwise. */
typedef enum { SPPO_GEMM_NT = 0, SPPO_GEMM_TN = 1 } sppo_gemm_layout;
typedef enum {
  SPPO_EPI_BF16 = 0,
  SPPO_EPI_ADD_BF16 = 1,
  SPPO_EPI_GELU = 2,
  SPPO_EPI_DGELU = 3,
  SPPO_EPI_ACC_F32 = 4,
  SPPO_EPI_F32 = 5
} sppo_epilogue;
sppo_status sppo_gemm_bf16(int32_t layout, int64_t M, int64_t N, int64_t K, const void* a, int64_t lda,
                           const void* b, int64_t ldb, void* c, int64_t ldc, int32_t epilogue, void* aux,
                           int64_t ldaux, void* stream);

/* LayerNorm of `rows` rows of H (H % 8 == 0, H <= 8192):
 * y = (x - mean) * rstd * gamma + beta, rstd = 1/sqrt(var + eps) with the
 * biased variance; mean and rstd (fp32 [rows]) are written for the
 * backward.  gamma, beta fp32 [H]. */
sppo_status sppo_layernorm_fwd(int64_t rows, int32_t H, const void* x, int64_t ldx, const float* gamma,
                               const float* beta, float eps, void* y, int64_t ldy, float* mean, float* rstd,
                               void* stream);

/* Backward of the LayerNorm above, with the residual branch folded in:
 *   dx = dres + rstd * (g - mean_j g - xhat * mean_j(g xhat)),
 *   g = dy * gamma, xhat = (x - mean) * rstd,
 * and dgamma (+)= sum_rows dy * xhat, dbeta (+)= sum_rows dy (fp32 [H];
 * accumulate != 0 adds, 0 overwrites; the sums run in a fixed order, so
 * results are reproducible bit for bit).  workspace: device fp32 scratch
 * of sppo_layernorm_bwd_workspace bytes. */
size_t sppo_layernorm_bwd_workspace(int64_t rows, int32_t H);
sppo_status sppo_layernorm_bwd(int64_t rows, int32_t H, const void* x, int64_t ldx, const float* gamma,
                               const float* mean, const float* rstd, const void* dy, int64_t lddy,
                               const void* dres, int64_t lddres, void* dx, int64_t lddx, float* dgamma,
                               float* dbeta, int32_t accumulate, float* workspace, size_t workspace_bytes,
                               void* stream);

/* y = gelu(x) (the tanh form above) over n bf16 values, n % 8 == 0. */
sppo_status sppo_gelu_bf16(const void* x, void* y, int64_t n, void* stream);

/* out [cols, rows] = in [rows, cols]^T, bf16, both contiguous. */
sppo_status sppo_transpose_bf16(const void* in, void* out, int64_t rows, int64_t cols, void* stream);

/* Row t < rows of out [rows, wq + 2 wkv] (bf16) = [dq[t] | dk[row0 + t] |
 * dv[row0 + t]]: the chunk's dQ (bf16 [rows, wq]) beside its rows of the
 * fp32 dK/dV accumulators ([.., wkv]) rounded to bf16 -- the gradient of
 * the fused QKV projection's output (B = 1). */
sppo_status sppo_pack_qkv_grad(int64_t rows, int32_t wq, int32_t wkv, const void* dq, const float* dk,
                               const float* dv, int64_t row0, void* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SPPO_H */
