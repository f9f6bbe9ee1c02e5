"""The C-ABI library loads, exports every entry point include/sppo.h
declares, and rejects invalid problems before touching the GPU (CPU only);
the public headers compile as C and C++."""
import ctypes
import os

import pytest

from paper_2503_10377_amd import sppo as L


def test_library_exports_every_declared_symbol():
    names = L.header_functions()
    assert {"sppo_create", "sppo_attn_fwd_chunk", "sppo_attn_bwd_chunk", "sppo_offload_issue",
            "sppo_prefetch"} <= set(names)
    lib = L.lib()
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings():
    assert L.sppo_status_string(L.SPPO_OK) == "SPPO_OK"
    assert L.sppo_status_string(L.SPPO_ERR_ORDER) == "SPPO_ERR_ORDER"
    assert L.sppo_status_string(99) == "SPPO_ERR_UNKNOWN"


def test_struct_layouts_match_c():
    # int64, int64, int32(+pad), ptr, int32 x3, enum, float, enum, int32(+pad), ptr
    assert ctypes.sizeof(L.sppo_problem) == 72
    assert L.sppo_problem.extra_row_bytes.offset == 64
    assert ctypes.sizeof(L.sppo_chunk_bufs) == 56
    assert L.sppo_chunk_bufs.keep.offset == 48
    assert ctypes.sizeof(L.sppo_copy_stats_t) == 40
    assert ctypes.sizeof(L.sppo_link_rates_t) == 24


GOOD = dict(batch=1, seq_len=1024, n_chunks=4, n_q_heads=8, n_kv_heads=2, head_dim=128)


@pytest.mark.parametrize("change,status", [
    (dict(head_dim=96), L.SPPO_ERR_UNSUPPORTED),
    (dict(head_dim=0), L.SPPO_ERR_UNSUPPORTED),
    (dict(seq_len=2**31, n_chunks=1), L.SPPO_ERR_UNSUPPORTED),   # key indices are int32
    (dict(batch=65535, seq_len=2**31 - 1, n_chunks=1, n_q_heads=65535, n_kv_heads=65535),
     L.SPPO_ERR_UNSUPPORTED),                                     # tensor bytes beyond 2^62
    (dict(batch=4096, seq_len=2**30, n_chunks=1, n_q_heads=4096, n_kv_heads=4096),
     L.SPPO_ERR_UNSUPPORTED),
    (dict(n_kv_heads=3), L.SPPO_ERR_INVALID_ARG),
    (dict(n_kv_heads=0), L.SPPO_ERR_INVALID_ARG),
    (dict(batch=0), L.SPPO_ERR_INVALID_ARG),
    (dict(seq_len=1000, n_chunks=3), L.SPPO_ERR_INVALID_ARG),     # S % N != 0, no offsets
    (dict(n_chunks=2000), L.SPPO_ERR_INVALID_ARG),                # N > S
    (dict(chunk_offsets=[0, 10, 10, 500, 1024]), L.SPPO_ERR_INVALID_ARG),  # not increasing
    (dict(chunk_offsets=[1, 10, 20, 500, 1024]), L.SPPO_ERR_INVALID_ARG),  # not from 0
    (dict(chunk_offsets=[0, 10, 20, 500, 1023]), L.SPPO_ERR_INVALID_ARG),  # not to S
    (dict(softmax_scale=-1.0), L.SPPO_ERR_INVALID_ARG),
    (dict(softmax_scale=float("nan")), L.SPPO_ERR_INVALID_ARG),
    (dict(dtype=7), L.SPPO_ERR_INVALID_ARG),
    (dict(offload=9), L.SPPO_ERR_INVALID_ARG),
    (dict(extra_row_bytes=[16, 0]), L.SPPO_ERR_INVALID_ARG),      # empty extra plane
    (dict(extra_row_bytes=[16, 6]), L.SPPO_ERR_INVALID_ARG),      # row bytes not a multiple of 4
    (dict(extra_row_bytes=[8] * 17), L.SPPO_ERR_INVALID_ARG),     # too many planes
])
def test_create_rejects_invalid_problems(change, status):
    kw = dict(GOOD)
    kw.update(change)
    with pytest.raises(L.SppoError) as ei:
        L.sppo_create(**kw)
    assert ei.value.status == status
    assert L.sppo_last_error(None)


def test_null_context_is_rejected():
    lib = L.lib()
    assert lib.sppo_attn_fwd_chunk(None, 0, None, None, None, None, None, None) == L.SPPO_ERR_INVALID_ARG
    assert lib.sppo_attn_bwd_chunk(None, 0, *([None] * 10)) == L.SPPO_ERR_INVALID_ARG
    assert lib.sppo_offload_issue(None, 0, None, None) == L.SPPO_ERR_INVALID_ARG
    assert lib.sppo_prefetch(None, 0, None, None) == L.SPPO_ERR_INVALID_ARG
    assert lib.sppo_offload_wait(None, 0, None) == L.SPPO_ERR_INVALID_ARG
    assert lib.sppo_reset(None) == L.SPPO_ERR_INVALID_ARG
    assert lib.sppo_sync(None) == L.SPPO_ERR_INVALID_ARG
    assert lib.sppo_copy_stats(None, None, 0) == L.SPPO_ERR_INVALID_ARG
    assert lib.sppo_prefetch_wait(None, 0, None) == L.SPPO_ERR_INVALID_ARG
    assert lib.sppo_destroy(None) == L.SPPO_OK
    assert lib.sppo_create(None, None) == L.SPPO_ERR_INVALID_ARG


def test_layer_ops_reject_invalid_arguments_before_launch():
    lib = L.lib()
    a = 4096  # any 16-byte aligned non-null value: nothing is launched on rejection
    bad = L.SPPO_ERR_INVALID_ARG
    # NT needs K % 64 == 0; TN needs M, N % 256 == 0; unknown layout/epilogue; misaligned pointers
    assert lib.sppo_gemm_bf16(0, 128, 256, 100, a, 128, a, 128, a, 256, 0, None, 0, None) == bad
    assert lib.sppo_gemm_bf16(1, 128, 256, 64, a, 128, a, 256, a, 256, 0, None, 0, None) == bad
    assert lib.sppo_gemm_bf16(2, 128, 256, 64, a, 64, a, 64, a, 256, 0, None, 0, None) == bad
    assert lib.sppo_gemm_bf16(0, 128, 256, 64, a, 64, a, 64, a, 256, 9, None, 0, None) == bad
    assert lib.sppo_gemm_bf16(0, 128, 256, 64, a + 2, 64, a, 64, a, 256, 0, None, 0, None) == bad
    assert lib.sppo_gemm_bf16(0, 128, 256, 64, a, 64, a, 64, a, 256, 1, None, 0, None) == bad  # ADD needs aux
    assert lib.sppo_gemm_bf16(0, 0, 256, 64, a, 64, a, 64, a, 256, 0, None, 0, None) == bad
    # vector epilogues: N, ldc and ldaux multiples of 4, aux 8-byte aligned
    assert lib.sppo_gemm_bf16(0, 128, 254, 64, a, 64, a, 64, a, 256, 0, None, 0, None) == bad
    assert lib.sppo_gemm_bf16(0, 128, 256, 64, a, 64, a, 64, a, 258, 0, None, 0, None) == bad
    assert lib.sppo_gemm_bf16(0, 128, 256, 64, a, 64, a, 64, a, 256, 1, a, 258, None) == bad
    assert lib.sppo_gemm_bf16(0, 128, 256, 64, a, 64, a, 64, a, 256, 1, a + 4, 256, None) == bad
    # the epilogue's 32-bit element offsets: M * ldc (and M * ldaux) below 2^31
    unsup = 2  # SPPO_ERR_UNSUPPORTED
    assert lib.sppo_gemm_bf16(0, 1 << 20, 4096, 64, a, 64, a, 64, a, 4096, 0, None, 0, None) == unsup
    assert lib.sppo_gemm_bf16(0, 1 << 19, 256, 64, a, 64, a, 64, a, 256, 1, a, 8192, None) == unsup
    # LayerNorm: H % 8, H > 8192, eps <= 0
    assert lib.sppo_layernorm_fwd(4, 100, a, 100, a, a, 1e-5, a, 100, a, a, None) == bad
    assert lib.sppo_layernorm_fwd(4, 8200, a, 8200, a, a, 1e-5, a, 8200, a, a, None) == bad
    assert lib.sppo_layernorm_fwd(4, 64, a, 64, a, a, 0.0, a, 64, a, a, None) == bad
    ws = lib.sppo_layernorm_bwd_workspace(100, 64)
    assert ws == 7 * 2 * 64 * 4  # ceil(100 / 16) blocks of [2, H] fp32
    assert lib.sppo_layernorm_bwd(100, 64, a, 64, a, a, a, a, 64, a, 64, a, 64, a, a, 1, a, ws - 4, None) == bad
    assert lib.sppo_gelu_bf16(a, a, 12, None) == bad
    assert lib.sppo_transpose_bf16(a, a, 4, 4, None) == bad          # in place
    assert lib.sppo_pack_qkv_grad(4, 12, 8, a, a, a, 0, a, None) == bad  # wq % 8


@pytest.mark.parametrize("change,status", [
    (dict(S=65536, c1=65536, Hq=32), L.SPPO_ERR_UNSUPPORTED),  # B * Hq * (c1 - c0) > 2^20 workspace rows
    (dict(B=65535, S=2**31 - 1, c1=1, Hq=65535, Hkv=65535), L.SPPO_ERR_UNSUPPORTED),  # tensor bytes beyond 2^62
    (dict(D=96), L.SPPO_ERR_UNSUPPORTED),
    (dict(c0=10, c1=10), L.SPPO_ERR_INVALID_ARG),
    (dict(c1=5000), L.SPPO_ERR_INVALID_ARG),             # past seq_len
    (dict(Hkv=3), L.SPPO_ERR_INVALID_ARG),
    (dict(acc=2), L.SPPO_ERR_INVALID_ARG),
    (dict(align=8), L.SPPO_ERR_INVALID_ARG),
    (dict(same_dkdv=True), L.SPPO_ERR_INVALID_ARG),
])
def test_noalloc_backward_checks_arguments_on_the_host(change, status):
    """The allocation-free backward validates everything before any HIP call
    (so these run without a GPU)."""
    a = dict(B=1, S=4096, c0=0, c1=1024, Hq=4, Hkv=2, D=128, acc=0, align=16, same_dkdv=False)
    a.update(change)
    p = [(1 << 20) + 16 * n if a["align"] == 16 else (1 << 20) + 8 for n in range(9)]
    if a["same_dkdv"]:
        p[8] = p[7]
    with pytest.raises(L.SppoError) as ei:
        L.sppo_attn_bwd_chunk_noalloc(a["B"], a["S"], a["c0"], a["c1"], a["Hq"], a["Hkv"], a["D"], "bf16", 0.0,
                                      a["acc"], *p, stream=0)
    assert ei.value.status == status
    assert L.sppo_last_error(None)


def test_headers_compile_as_c99_and_cxx(tmp_path):
    """Every public header is valid C (C99, warnings as errors) and C++: a C
    caller gets the same declarations through extern "C"."""
    import glob
    import shutil
    import subprocess
    inc = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
    heads = sorted(os.path.basename(h) for h in glob.glob(os.path.join(inc, "*.h")))
    assert heads
    src = "".join(f'#include "{h}"\n' for h in heads) + "int main(void) { return 0; }\n"
    for cc, ext, std in (("gcc", "c", "-std=c99"), ("g++", "cpp", "-std=c++17")):
        if shutil.which(cc) is None:
            pytest.skip(f"{cc} not available")
        f = tmp_path / f"h.{ext}"
        f.write_text(src)
        r = subprocess.run([cc, std, "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", inc, "-c", str(f),
                            "-o", str(tmp_path / f"h_{ext}.o")], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr
