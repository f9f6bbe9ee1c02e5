"""ctypes binding of libsppo (include/sppo.h): argument marshalling only.

Every function here has the name of the C entry point it calls.  Tensor
arguments may be torch tensors (their ``data_ptr()`` is passed) or integer
device addresses; streams may be torch streams, raw ``hipStream_t`` integers,
or None for torch's current stream.  A non-OK status raises ``SppoError``
carrying the status and the library's message.  The library must have been
built (``python -m paper_2503_10377_amd.build``); there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import re

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsppo.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "sppo.h")

SPPO_OK = 0
SPPO_ERR_INVALID_ARG = 1
SPPO_ERR_UNSUPPORTED = 2
SPPO_ERR_ORDER = 3
SPPO_ERR_STATE = 4
SPPO_ERR_OOM = 5
SPPO_ERR_HIP = 6

SPPO_F32 = 0
SPPO_BF16 = 1

SPPO_OFFLOAD_NONE = 0
SPPO_OFFLOAD_QOL = 1
SPPO_OFFLOAD_QKVOL = 2
SPPO_OFFLOAD_QKVOL_EVICT = 3

OFFLOAD_MODES = {"none": SPPO_OFFLOAD_NONE, "qol": SPPO_OFFLOAD_QOL, "qkvol": SPPO_OFFLOAD_QKVOL,
                 "qkvol_evict": SPPO_OFFLOAD_QKVOL_EVICT}


class sppo_problem(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int64),
        ("seq_len", ctypes.c_int64),
        ("n_chunks", ctypes.c_int32),
        ("chunk_offsets", ctypes.POINTER(ctypes.c_int64)),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("dtype", ctypes.c_int),
        ("softmax_scale", ctypes.c_float),
        ("offload", ctypes.c_int),
        ("n_extra", ctypes.c_int32),
        ("extra_row_bytes", ctypes.POINTER(ctypes.c_size_t)),
    ]


class sppo_chunk_bufs(ctypes.Structure):
    _fields_ = [
        ("q", ctypes.c_void_p),
        ("o", ctypes.c_void_p),
        ("lse", ctypes.c_void_p),
        ("k", ctypes.c_void_p),
        ("v", ctypes.c_void_p),
        ("extra", ctypes.POINTER(ctypes.c_void_p)),
        ("keep", ctypes.c_void_p),
    ]


class sppo_copy_stats_t(ctypes.Structure):
    _fields_ = [
        ("bytes_d2h", ctypes.c_uint64),
        ("bytes_h2d", ctypes.c_uint64),
        ("ms_d2h", ctypes.c_double),
        ("ms_h2d", ctypes.c_double),
        ("n_d2h", ctypes.c_int32),
        ("n_h2d", ctypes.c_int32),
    ]


KERNELS = ("fwd", "bwd_pre", "bwd_dkdv", "bwd_dq")


class sppo_kernel_times_t(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double * 4), ("launches", ctypes.c_int32 * 4)]


class sppo_link_rates_t(ctypes.Structure):
    _fields_ = [("d2h_GBps", ctypes.c_double), ("h2d_GBps", ctypes.c_double), ("duplex_GBps", ctypes.c_double)]


class SppoError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        super().__init__(f"{status_name(status)}: {message}")


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libsppo; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with python -m paper_2503_10377_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, VP = ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p
        sig = {
            "sppo_create": ([ctypes.POINTER(sppo_problem), ctypes.POINTER(P)], ctypes.c_int),
            "sppo_destroy": ([P], ctypes.c_int),
            "sppo_attn_fwd_chunk": ([P, I32, VP, VP, VP, VP, VP, VP], ctypes.c_int),
            "sppo_attn_bwd_chunk": ([P, I32, VP, VP, VP, VP, VP, VP, VP, VP, VP, VP], ctypes.c_int),
            "sppo_offload_issue": ([P, I32, ctypes.POINTER(sppo_chunk_bufs), VP], ctypes.c_int),
            "sppo_offload_wait": ([P, I32, VP], ctypes.c_int),
            "sppo_prefetch": ([P, I32, ctypes.POINTER(sppo_chunk_bufs), VP], ctypes.c_int),
            "sppo_prefetch_kv": ([P, I32, VP, VP, VP], ctypes.c_int),
            "sppo_reset": ([P], ctypes.c_int),
            "sppo_sync": ([P], ctypes.c_int),
            "sppo_copy_stats": ([P, ctypes.POINTER(sppo_copy_stats_t), I32], ctypes.c_int),
            "sppo_set_kernel_timing": ([P, I32], ctypes.c_int),
            "sppo_link_probe": ([P, ctypes.c_size_t, ctypes.POINTER(sppo_link_rates_t)], ctypes.c_int),
            "sppo_set_offload_rows": ([P, I32, ctypes.c_int64], ctypes.c_int),
            "sppo_get_offload_rows": ([P, ctypes.POINTER(ctypes.c_int64), I32], ctypes.c_int),
            "sppo_balanced_offsets": ([ctypes.c_int64, I32, ctypes.c_int64, ctypes.POINTER(ctypes.c_int64)],
                                      ctypes.c_int),
            "sppo_plan_offload_rows": ([ctypes.POINTER(ctypes.c_int64), I32, ctypes.c_double, ctypes.c_double,
                                        ctypes.POINTER(ctypes.c_double), ctypes.c_int64,
                                        ctypes.POINTER(ctypes.c_int64)], ctypes.c_int),
            "sppo_kernel_times": ([P, ctypes.POINTER(sppo_kernel_times_t), I32], ctypes.c_int),
            "sppo_get_offsets": ([P, ctypes.POINTER(ctypes.c_int64), I32], ctypes.c_int),
            "sppo_last_error": ([P], ctypes.c_char_p),
            "sppo_gemm_bf16": ([I32, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, VP, ctypes.c_int64, VP,
                                ctypes.c_int64, VP, ctypes.c_int64, I32, VP, ctypes.c_int64, VP], ctypes.c_int),
            "sppo_layernorm_fwd": ([ctypes.c_int64, I32, VP, ctypes.c_int64, VP, VP, ctypes.c_float, VP,
                                    ctypes.c_int64, VP, VP, VP], ctypes.c_int),
            "sppo_layernorm_bwd_workspace": ([ctypes.c_int64, I32], ctypes.c_size_t),
            "sppo_layernorm_bwd": ([ctypes.c_int64, I32, VP, ctypes.c_int64, VP, VP, VP, VP, ctypes.c_int64, VP,
                                    ctypes.c_int64, VP, ctypes.c_int64, VP, VP, I32, VP, ctypes.c_size_t, VP],
                                   ctypes.c_int),
            "sppo_prefetch_wait": ([P, I32, VP], ctypes.c_int),
            "sppo_gelu_bf16": ([VP, VP, ctypes.c_int64, VP], ctypes.c_int),
            "sppo_transpose_bf16": ([VP, VP, ctypes.c_int64, ctypes.c_int64, VP], ctypes.c_int),
            "sppo_pack_qkv_grad": ([ctypes.c_int64, I32, I32, VP, VP, VP, ctypes.c_int64, VP, VP], ctypes.c_int),
            "sppo_status_string": ([ctypes.c_int], ctypes.c_char_p),
            "sppo_keep_bytes": ([P, I32], ctypes.c_size_t),
            "sppo_attn_bwd_chunk_noalloc": ([ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, I32,
                                             I32, I32, ctypes.c_int, ctypes.c_float, I32, VP, VP, VP, VP, VP, VP,
                                             VP, VP, VP, VP], ctypes.c_int),
            "sppo_attn_finalize_chunk": ([P, I32, VP, VP, VP, VP, VP], ctypes.c_int),
        }
        for name, (args, res) in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def header_functions(path: str = HEADER_PATH) -> list[str]:
    """Names of the entry points declared in include/sppo.h."""
    with open(path) as f:
        text = f.read()
    return re.findall(r"^(?:sppo_status|const char\*|size_t)\s+(sppo_\w+)\s*\(", text, flags=re.M)


def status_name(status: int) -> str:
    try:
        return lib().sppo_status_string(status).decode()
    except Exception:  # pragma: no cover - only while formatting an error
        return f"status {status}"


def _ptr(x) -> int | None:
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    return int(x)


def _stream(s) -> int | None:
    if s is None:
        import torch

        return torch.cuda.current_stream().cuda_stream
    if hasattr(s, "cuda_stream"):
        return s.cuda_stream
    return int(s)


class Ctx:
    """Owning handle of an ``sppo_ctx*``."""

    def __init__(self, handle: int, problem: dict):
        self.handle = handle
        self.problem = problem

    @property
    def _as_parameter_(self):
        return ctypes.c_void_p(self.handle)

    def close(self):
        if self.handle:
            lib().sppo_destroy(ctypes.c_void_p(self.handle))
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _check(ctx, status: int):
    if status != SPPO_OK:
        h = ctypes.c_void_p(ctx.handle) if isinstance(ctx, Ctx) and ctx.handle else None
        msg = lib().sppo_last_error(h)
        raise SppoError(status, msg.decode() if msg else "")


def _handle(ctx):
    if isinstance(ctx, Ctx):
        return ctypes.c_void_p(ctx.handle) if ctx.handle else None
    return ctx


def sppo_create(batch, seq_len, n_chunks, n_q_heads, n_kv_heads, head_dim, dtype="bf16",
                chunk_offsets=None, softmax_scale=0.0, offload="none", extra_row_bytes=()) -> Ctx:
    dt = {"bf16": SPPO_BF16, "f32": SPPO_F32, "fp32": SPPO_F32}.get(dtype, dtype)
    off = OFFLOAD_MODES.get(offload, offload)
    p = sppo_problem(batch, seq_len, n_chunks, None, n_q_heads, n_kv_heads, head_dim, dt,
                     softmax_scale, off, len(extra_row_bytes), None)
    arr = None
    if chunk_offsets is not None:
        arr = (ctypes.c_int64 * len(chunk_offsets))(*[int(x) for x in chunk_offsets])
        p.chunk_offsets = arr
    xrb = None
    if len(extra_row_bytes):
        xrb = (ctypes.c_size_t * len(extra_row_bytes))(*[int(x) for x in extra_row_bytes])
        p.extra_row_bytes = xrb
    out = ctypes.c_void_p()
    st = lib().sppo_create(ctypes.byref(p), ctypes.byref(out))
    if st != SPPO_OK:
        raise SppoError(st, lib().sppo_last_error(None).decode())
    problem = dict(batch=batch, seq_len=seq_len, n_chunks=n_chunks, n_q_heads=n_q_heads,
                   n_kv_heads=n_kv_heads, head_dim=head_dim, dtype=dt, softmax_scale=softmax_scale,
                   offload=off, extra_row_bytes=tuple(int(x) for x in extra_row_bytes))
    return Ctx(out.value, problem)


def sppo_destroy(ctx: Ctx):
    ctx.close()


def sppo_attn_fwd_chunk(ctx, i, q_i, k, v, o_i, lse_i, stream=None):
    _check(ctx, lib().sppo_attn_fwd_chunk(_handle(ctx), i, _ptr(q_i), _ptr(k), _ptr(v), _ptr(o_i),
                                          _ptr(lse_i), _stream(stream)))


def sppo_attn_bwd_chunk(ctx, i, q_i, k, v, o_i, lse_i, do_i, dq_i, dk_acc, dv_acc, stream=None):
    _check(ctx, lib().sppo_attn_bwd_chunk(_handle(ctx), i, _ptr(q_i), _ptr(k), _ptr(v), _ptr(o_i),
                                          _ptr(lse_i), _ptr(do_i), _ptr(dq_i), _ptr(dk_acc),
                                          _ptr(dv_acc), _stream(stream)))


def chunk_bufs(q=None, o=None, lse=None, k=None, v=None, extra=(), keep=None) -> sppo_chunk_bufs:
    b = sppo_chunk_bufs(_ptr(q), _ptr(o), _ptr(lse), _ptr(k), _ptr(v), None, _ptr(keep))
    if len(extra):
        arr = (ctypes.c_void_p * len(extra))(*[_ptr(x) for x in extra])
        b.extra = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p))
        b._extra_keepalive = arr  # the array must outlive the struct's use
    return b


def sppo_offload_issue(ctx, i, src: sppo_chunk_bufs, stream=None):
    _check(ctx, lib().sppo_offload_issue(_handle(ctx), i, ctypes.byref(src), _stream(stream)))


def sppo_offload_wait(ctx, i, stream=None):
    _check(ctx, lib().sppo_offload_wait(_handle(ctx), i, _stream(stream)))


def sppo_prefetch(ctx, i, dst: sppo_chunk_bufs, stream=None):
    _check(ctx, lib().sppo_prefetch(_handle(ctx), i, ctypes.byref(dst), _stream(stream)))


def sppo_prefetch_kv(ctx, i, k, v, stream=None):
    _check(ctx, lib().sppo_prefetch_kv(_handle(ctx), i, _ptr(k), _ptr(v), _stream(stream)))


def sppo_attn_bwd_chunk_noalloc(batch, seq_len, c0, c1, n_q_heads, n_kv_heads, head_dim, dtype, softmax_scale,
                                accumulate, q_i, k, v, o_i, lse_i, do_i, dq_i, dk_acc, dv_acc, stream=None):
    dt = {"bf16": SPPO_BF16, "f32": SPPO_F32, "fp32": SPPO_F32}.get(dtype, dtype)
    st = lib().sppo_attn_bwd_chunk_noalloc(batch, seq_len, c0, c1, n_q_heads, n_kv_heads, head_dim, dt,
                                           softmax_scale, int(accumulate), _ptr(q_i), _ptr(k), _ptr(v), _ptr(o_i),
                                           _ptr(lse_i), _ptr(do_i), _ptr(dq_i), _ptr(dk_acc), _ptr(dv_acc),
                                           _stream(stream))
    if st != SPPO_OK:
        raise SppoError(st, lib().sppo_last_error(None).decode())


def sppo_keep_bytes(ctx, i) -> int:
    return int(lib().sppo_keep_bytes(_handle(ctx), i))


def sppo_attn_finalize_chunk(ctx, i, dk_acc, dv_acc, dk_out, dv_out, stream=None):
    _check(ctx, lib().sppo_attn_finalize_chunk(_handle(ctx), i, _ptr(dk_acc), _ptr(dv_acc), _ptr(dk_out),
                                               _ptr(dv_out), _stream(stream)))


def sppo_reset(ctx):
    _check(ctx, lib().sppo_reset(_handle(ctx)))


def sppo_sync(ctx):
    _check(ctx, lib().sppo_sync(_handle(ctx)))


def sppo_copy_stats(ctx, reset_after=False) -> dict:
    out = sppo_copy_stats_t()
    _check(ctx, lib().sppo_copy_stats(_handle(ctx), ctypes.byref(out), 1 if reset_after else 0))
    return {n: getattr(out, n) for n, _ in sppo_copy_stats_t._fields_}


def sppo_set_kernel_timing(ctx, enable=True):
    _check(ctx, lib().sppo_set_kernel_timing(_handle(ctx), 1 if enable else 0))


def sppo_kernel_times(ctx, reset_after=False) -> dict:
    out = sppo_kernel_times_t()
    _check(ctx, lib().sppo_kernel_times(_handle(ctx), ctypes.byref(out), 1 if reset_after else 0))
    return {k: {"ms": out.ms[n], "launches": out.launches[n]} for n, k in enumerate(KERNELS)}


def sppo_link_probe(ctx, nbytes) -> dict:
    out = sppo_link_rates_t()
    _check(ctx, lib().sppo_link_probe(_handle(ctx), nbytes, ctypes.byref(out)))
    return {"d2h_GBps": out.d2h_GBps, "h2d_GBps": out.h2d_GBps, "duplex_GBps": out.duplex_GBps}


def sppo_set_offload_rows(ctx, i, rows):
    _check(ctx, lib().sppo_set_offload_rows(_handle(ctx), i, int(rows)))


def sppo_get_offload_rows(ctx) -> list[int]:
    n = ctx.problem["n_chunks"]
    arr = (ctypes.c_int64 * n)()
    _check(ctx, lib().sppo_get_offload_rows(_handle(ctx), arr, n))
    return list(arr)


def _status_check(st, what):
    if st != SPPO_OK:
        raise SppoError(st, what)


def sppo_balanced_offsets(seq_len, n_chunks, align=1) -> list[int]:
    arr = (ctypes.c_int64 * (n_chunks + 1))()
    _status_check(lib().sppo_balanced_offsets(seq_len, n_chunks, align, arr),
                  f"balanced offsets S={seq_len} N={n_chunks} align={align}")
    return list(arr)


def sppo_plan_offload_rows(offsets, bytes_per_row, bw_GBps, t_overlap_ms, align=1) -> list[int]:
    n = len(offsets) - 1
    if len(t_overlap_ms) != n:
        raise ValueError("t_overlap_ms needs one value per chunk")
    off = (ctypes.c_int64 * (n + 1))(*offsets)
    t = (ctypes.c_double * n)(*t_overlap_ms)
    rows = (ctypes.c_int64 * n)()
    _status_check(lib().sppo_plan_offload_rows(off, n, float(bytes_per_row), float(bw_GBps), t, align, rows),
                  "offload plan")
    return list(rows)


def sppo_get_offsets(ctx) -> list[int]:
    n = ctx.problem["n_chunks"] + 1
    arr = (ctypes.c_int64 * n)()
    _check(ctx, lib().sppo_get_offsets(_handle(ctx), arr, n))
    return list(arr)


def sppo_last_error(ctx) -> str:
    msg = lib().sppo_last_error(_handle(ctx))
    return msg.decode() if msg else ""


def sppo_status_string(status: int) -> str:
    return lib().sppo_status_string(status).decode()


# ---------------------------------------------------------------- full layer
SPPO_GEMM_NT, SPPO_GEMM_TN = 0, 1
EPILOGUES = {"bf16": 0, "add_bf16": 1, "gelu": 2, "dgelu": 3, "acc_f32": 4, "f32": 5}


def _plain(status: int):
    if status != SPPO_OK:
        raise SppoError(status, status_name(status))


def sppo_gemm_bf16(layout, M, N, K, a, lda, b, ldb, c, ldc, epilogue="bf16", aux=None, ldaux=0, stream=None):
    lay = {"nt": SPPO_GEMM_NT, "tn": SPPO_GEMM_TN}.get(layout, layout)
    epi = EPILOGUES.get(epilogue, epilogue)
    _plain(lib().sppo_gemm_bf16(lay, M, N, K, _ptr(a), lda, _ptr(b), ldb, _ptr(c), ldc, epi, _ptr(aux), ldaux,
                                _stream(stream)))


def sppo_layernorm_fwd(rows, H, x, ldx, gamma, beta, eps, y, ldy, mean, rstd, stream=None):
    _plain(lib().sppo_layernorm_fwd(rows, H, _ptr(x), ldx, _ptr(gamma), _ptr(beta), eps, _ptr(y), ldy, _ptr(mean),
                                    _ptr(rstd), _stream(stream)))


def sppo_layernorm_bwd_workspace(rows, H) -> int:
    return int(lib().sppo_layernorm_bwd_workspace(rows, H))


def sppo_layernorm_bwd(rows, H, x, ldx, gamma, mean, rstd, dy, lddy, dres, lddres, dx, lddx, dgamma, dbeta,
                       workspace, workspace_bytes, accumulate=1, stream=None):
    _plain(lib().sppo_layernorm_bwd(rows, H, _ptr(x), ldx, _ptr(gamma), _ptr(mean), _ptr(rstd), _ptr(dy), lddy,
                                    _ptr(dres), lddres, _ptr(dx), lddx, _ptr(dgamma), _ptr(dbeta), int(accumulate),
                                    _ptr(workspace), workspace_bytes, _stream(stream)))


def sppo_prefetch_wait(ctx, i, stream=None):
    _check(ctx, lib().sppo_prefetch_wait(_handle(ctx), i, _stream(stream)))


def sppo_gelu_bf16(x, y, n, stream=None):
    _plain(lib().sppo_gelu_bf16(_ptr(x), _ptr(y), n, _stream(stream)))


def sppo_transpose_bf16(x, y, rows, cols, stream=None):
    _plain(lib().sppo_transpose_bf16(_ptr(x), _ptr(y), rows, cols, _stream(stream)))


def sppo_pack_qkv_grad(rows, wq, wkv, dq, dk, dv, row0, out, stream=None):
    _plain(lib().sppo_pack_qkv_grad(rows, wq, wkv, _ptr(dq), _ptr(dk), _ptr(dv), row0, _ptr(out), _stream(stream)))
