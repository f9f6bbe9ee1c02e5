"""GPU parity at sizes the fp64 oracle finishes in seconds: the HIP path,
called through the C ABI, against the oracle element by element on the same
seeded inputs (full tensors), spanning several tiles and ragged tails."""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2503_10377_amd import sppo as L
from paper_2503_10377_amd.chunked import ChunkedAttention
from paper_2503_10377_amd.inputs import make_inputs
from parity import check_all, check_structured, to_np

pytestmark = pytest.mark.gpu

TORCH_DT = {"bf16": torch.bfloat16, "f32": torch.float32}


def announce(msg):
    print(f"\n[case] {msg}", file=sys.stderr, flush=True)


def run_case(B, S, Hq, Hkv, D, dtype, N=None, offsets=None, seed=0, kind="randn",
             offload="none", lookahead=2, poison=False, rows=None, softmax_scale=None, fwd_slots=4):
    if offsets is None:
        offsets = list(oracle.equal_offsets(S, N))
    N = len(offsets) - 1
    announce(f"B={B} S={S} Hq={Hq} Hkv={Hkv} D={D} {dtype} offsets={offsets[:6]}.. N={N} "
             f"seed={seed} kind={kind} offload={offload} poison={poison}")
    inp = make_inputs(B, S, Hq, Hkv, D, TORCH_DT[dtype], seed=seed, device="cuda", kind=kind)
    host = {n: to_np(t) for n, t in inp.items()}  # taken before the HIP path runs
    ca = ChunkedAttention(B, S, N, Hq, Hkv, D, dtype=dtype, offsets=offsets, offload=offload,
                          scale=softmax_scale or 0.0, fwd_slots=fwd_slots)
    if rows is not None:
        ca.set_offload_rows(rows)
    out = ca.alloc_outputs()
    ca.step(inp, out, lookahead=lookahead, poison=poison)
    torch.cuda.synchronize()
    gpu = {"o": to_np(out["o"]), "lse": to_np(ca.lse_full(out)), "dq": to_np(out["dq"]),
           "dk": to_np(out["dk"]), "dv": to_np(out["dv"])}
    ca.close()
    scale = softmax_scale or 1.0 / math.sqrt(D)
    ref = oracle.attention(host["q"], host["k"], host["v"], host["do"], scale)
    return gpu, ref, offsets


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_fp32_config_seq1024_4chunks(seed):
    # fp32, batch 1, 1 head, head_dim 64, seq 1024 in 4 chunks of 256.
    gpu, ref, off = run_case(1, 1024, 1, 1, 64, "f32", N=4, seed=seed)
    check_all(gpu, ref, "f32", off)


@pytest.mark.parametrize("D", [64, 128])
def test_fp32_ragged_gqa(D):
    gpu, ref, off = run_case(1, 700, 4, 2, D, "f32", offsets=[0, 100, 101, 450, 700], seed=3)
    check_all(gpu, ref, "f32", off)


def test_bf16_mha_medium():
    gpu, ref, off = run_case(1, 2048, 4, 4, 128, "bf16", N=4, seed=0)
    check_all(gpu, ref, "bf16", off)


def test_bf16_gqa_medium():
    gpu, ref, off = run_case(1, 1536, 8, 2, 128, "bf16", N=3, seed=1)
    check_all(gpu, ref, "bf16", off)


@pytest.mark.parametrize("D", [64, 128])
def test_bf16_ragged_offsets(D):
    # Chunk lengths 77, 223, 1, 699: tails inside every tile size, a
    # one-row chunk, and chunk boundaries off the tile grid.
    gpu, ref, off = run_case(1, 1000, 2, 1, D, "bf16", offsets=[0, 77, 300, 301, 1000], seed=2)
    check_all(gpu, ref, "bf16", off)


def test_bf16_balanced_partition_partial_offload():
    """FLOPs-balanced boundaries (long chunks first, c_k = S sqrt(k/N) on a
    64-row grid) with a sequence-aware partial offload: only a row prefix
    of each chunk leaves the device (and is poisoned there)."""
    S, N = 3072, 6
    offsets = L.sppo_balanced_offsets(S, N, 64)
    lens = [b - a for a, b in zip(offsets, offsets[1:])]
    rows = [lens[0] // 3, lens[1] - 5, 0, 64, lens[4], 0]
    gpu, ref, off = run_case(1, S, 4, 2, 128, "bf16", offsets=offsets, seed=11, offload="qkvol",
                             poison=True, rows=rows)
    check_all(gpu, ref, "bf16", off)


def test_bf16_batch2():
    gpu, ref, off = run_case(2, 640, 2, 2, 64, "bf16", N=5, seed=4)
    check_all(gpu, ref, "bf16", off)


def test_bf16_single_row_sequence():
    gpu, ref, off = run_case(1, 1, 2, 1, 128, "bf16", N=1, seed=5)
    check_all(gpu, ref, "bf16", off)


@pytest.mark.parametrize("kind", ["sharp_self", "sharp_future", "zero_q"])
def test_bf16_structured(kind):
    """Structured inputs that random ones cannot exercise.  A diagonal mask
    that drops a row's own key (sharp_self) or admits the next key
    (sharp_future) moves O, LSE and dV by O(1), forward or backward.

    The gates are parity.check_structured's, derived from the bf16 recipe
    emulated on the CPU (tests/test_structured_gates_cpu.py): max-abs
    scaled by max(1, max|ref|), and for sharp_self absolute gates only on
    dQ and dK."""
    gpu, ref, off = run_case(1, 2048, 2, 1, 128, "bf16", N=4, seed=6, kind=kind)
    check_structured(gpu, ref, kind, off)


def test_chunked_matches_unchunked_on_gpu():
    """Chunking is an exact rewrite: with chunk boundaries on the tile grid
    the forward and dQ are bitwise identical to one chunk; dK/dV differ only
    by the order of fp32 accumulation across chunks."""
    B, S, Hq, Hkv, D = 1, 2048, 4, 2, 128
    res = {}
    for N in (1, 4):
        announce(f"chunked-vs-unchunked N={N}")
        inp = make_inputs(B, S, Hq, Hkv, D, torch.bfloat16, seed=7, device="cuda")
        ca = ChunkedAttention(B, S, N, Hq, Hkv, D, dtype="bf16")
        out = ca.alloc_outputs()
        ca.step(inp, out)
        torch.cuda.synchronize()
        res[N] = {"o": out["o"].clone(), "lse": ca.lse_full(out).clone(), "dq": out["dq"].clone(),
                  "dk": out["dk"].clone(), "dv": out["dv"].clone()}
        ca.close()
    for n in ("o", "lse", "dq"):
        assert torch.equal(res[1][n], res[4][n]), n
    for n in ("dk", "dv"):
        a, b = res[1][n].double(), res[4][n].double()
        assert ((a - b).norm() / a.norm()).item() < 1e-5, n


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_finalize_rounds_each_chunk_after_its_backward(dtype):
    """Finalize: right after bwd(i), rows [c_i, c_{i+1}) of dK/dV are final
    and are written in the problem's dtype -- bit for bit the fp32
    accumulators rounded to nearest even (bf16) or copied (fp32) -- and
    within the gates of the oracle.  Before its backward a chunk cannot be
    finalized."""
    B, S, Hq, Hkv, D = 2, 1000, 4, 2, 64
    offsets = [0, 77, 300, 301, 1000]
    announce(f"finalize {dtype}")
    tdt = TORCH_DT[dtype]
    inp = make_inputs(B, S, Hq, Hkv, D, tdt, seed=17, device="cuda")
    host = {n: to_np(t) for n, t in inp.items()}
    ca = ChunkedAttention(B, S, 4, Hq, Hkv, D, dtype=dtype, offsets=offsets, offload="qkvol")
    out = ca.alloc_outputs()
    fin = {n: torch.full((B, S, Hkv, D), float("nan"), dtype=tdt, device="cuda") for n in ("dk", "dv")}
    with pytest.raises(L.SppoError) as ei:
        L.sppo_attn_finalize_chunk(ca.ctx, 0, out["dk"], out["dv"], fin["dk"], fin["dv"])
    assert ei.value.status == L.SPPO_ERR_STATE
    ca.step(inp, out, finalize=fin)
    torch.cuda.synchronize()
    for n in ("dk", "dv"):
        assert torch.equal(fin[n], out[n].to(tdt)), n
    ref = oracle.attention(host["q"], host["k"], host["v"], host["do"], 1.0 / math.sqrt(D))
    check_all({"dk": to_np(fin["dk"]), "dv": to_np(fin["dv"])}, ref, dtype, offsets)
    with pytest.raises(L.SppoError) as ei:
        L.sppo_attn_finalize_chunk(ca.ctx, 1, out["dk"], out["dv"], fin["dk"], fin["dk"])
    assert ei.value.status == L.SPPO_ERR_INVALID_ARG
    ca.close()


@pytest.mark.parametrize("D", [64, 128])
def test_bf16_mqa_ragged_offload(D):
    """Multi-query attention (8 query heads share one KV head: the dK/dV
    kernel sums over the whole group), ragged chunks off the tile grid, the
    full offload set with poisoned dead buffers, and a row-prefix plan with
    keep buffers on two chunks."""
    S = 1800
    offsets = [0, 333, 700, 701, 1500, 1800]
    lens = [b - a for a, b in zip(offsets, offsets[1:])]
    rows = [lens[0] // 2, lens[1], 0, lens[3] - 7, 0]
    gpu, ref, off = run_case(1, S, 8, 1, D, "bf16", offsets=offsets, seed=23, offload="qkvol", poison=True,
                             rows=rows)
    check_all(gpu, ref, "bf16", off)


def test_bf16_head_dim64_batch3_evict():
    """head_dim 64, three batch entries, GQA 6/2, the K/V-evicting mode with
    poisoned cache rows."""
    gpu, ref, off = run_case(3, 1280, 6, 2, 64, "bf16", N=5, seed=29, offload="qkvol_evict", poison=True)
    check_all(gpu, ref, "bf16", off)


@pytest.mark.parametrize("offload", ["qkvol", "qkvol_evict"])
def test_bf16_every_chunk_one_row(offload):
    """N = S: every chunk is one query row (a 31-row padded sub-block in
    every kernel, one-row copies of each tensor), offloaded and poisoned,
    over a walk of 48 chunks."""
    gpu, ref, off = run_case(1, 48, 4, 2, 128, "bf16", N=48, seed=31, offload=offload, poison=True)
    check_all(gpu, ref, "bf16", off)


@pytest.mark.parametrize("offload", ["qkvol", "qkvol_evict"])
def test_fp32_offload_row_prefix_batch2(offload):
    """The fp32 path through the offload engine (4-byte elements in every
    copy, keep buffer and arena region): batch 2, GQA, ragged chunks, a
    row-prefix plan with keep buffers, poisoned dead buffers."""
    offsets = [0, 97, 300, 301, 640]
    lens = [b - a for a, b in zip(offsets, offsets[1:])]
    rows = [lens[0] - 10, 0, 1, lens[3]]
    gpu, ref, off = run_case(2, 640, 4, 2, 64, "f32", offsets=offsets, seed=37, offload=offload, poison=True,
                             rows=rows)
    check_all(gpu, ref, "f32", off)


@pytest.mark.parametrize("dtype,scale", [("bf16", 0.15), ("f32", 0.2)])
def test_explicit_softmax_scale(dtype, scale):
    """A softmax scale other than 1/sqrt(D) (0.088 at D = 128) reaches every
    kernel: the forward's exponent, the backward's recomputed P, and the
    scale on dQ and dK.  Ragged GQA chunks, offloaded and poisoned.  (The
    fp32 LSE gate, 1e-5 absolute, is sized for logits of the default scale:
    the fp32 rounding of a 128-term dot product grows with the scale, and at
    0.5, logits around 20, it reaches 1.3e-5.)"""
    gpu, ref, off = run_case(1, 900, 4, 2, 128, dtype, offsets=[0, 200, 201, 555, 900], seed=41, offload="qkvol",
                             poison=True, softmax_scale=scale)
    check_all(gpu, ref, dtype, off)


@pytest.mark.parametrize("fwd_slots,lookahead", [(1, 0), (1, 2), (2, 1)])
def test_tight_arena(fwd_slots, lookahead):
    """The smallest device arenas: with fwd_slots = 1 every forward chunk
    reuses the region of the chunk just offloaded (the compute stream waits
    for that copy first), with 2 the one before it; the backward's prefetch
    reuses regions as they free up.  Ragged GQA chunks, offloaded and
    poisoned."""
    gpu, ref, off = run_case(1, 1500, 4, 2, 128, "bf16", offsets=[0, 300, 301, 700, 1100, 1500], seed=43,
                             offload="qkvol", poison=True, fwd_slots=fwd_slots, lookahead=lookahead)
    check_all(gpu, ref, "bf16", off)
