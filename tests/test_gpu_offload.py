"""Offload engine and C-ABI state machine on the GPU.

* Offload must not change a single bit of any result (on/off equality), for
  every offload mode, lookahead and offload set.
* Poison test: once a chunk's copy has landed on the host its device
  Q/O/LSE are overwritten with NaN; the backward must then read the
  prefetched copies, so results stay bitwise equal (a read of stale or
  not-yet-prefetched memory would surface as NaN).
* K/V eviction (qkvol_evict): the K/V cache rows of offloaded chunks are
  overwritten with NaN after the forward walk; the backward of the last
  chunk must consume the prefetched rows piece by piece, and every result
  stays bitwise equal to the run without offload.
* Order/state violations return the documented status and enqueue nothing.
"""
import gc
import sys

import pytest
import torch

from paper_2503_10377_amd import sppo as L
from paper_2503_10377_amd.chunked import ChunkedAttention
from paper_2503_10377_amd.inputs import make_inputs

pytestmark = pytest.mark.gpu

SHAPE = dict(B=1, S=4096, Hq=4, Hkv=2, D=128)
N = 8


def announce(msg):
    print(f"\n[case] {msg}", file=sys.stderr, flush=True)


def run(offload="none", offload_chunks=None, lookahead=2, poison=False, B=1, seed=0, dtype="bf16",
        offsets=None, shape=None, rows=None):
    S, Hq, Hkv, D = (shape or (SHAPE["S"], SHAPE["Hq"], SHAPE["Hkv"], SHAPE["D"]))
    n = N if offsets is None else len(offsets) - 1
    announce(f"offload={offload} chunks={offload_chunks} lookahead={lookahead} poison={poison} B={B} "
             f"dtype={dtype} offsets={offsets} shape={(S, Hq, Hkv, D)}")
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    inp = make_inputs(B, S, Hq, Hkv, D, tdt, seed=seed, device="cuda")
    ca = ChunkedAttention(B, S, n, Hq, Hkv, D, dtype=dtype, offload=offload, offsets=offsets)
    if rows is not None:
        ca.set_offload_rows(rows)
    out = ca.alloc_outputs()
    ca.step(inp, out, offload_chunks=offload_chunks, lookahead=lookahead, poison=poison)
    torch.cuda.synchronize()
    stats = L.sppo_copy_stats(ca.ctx) if offload != "none" else None
    res = {"o": out["o"].clone(), "lse": ca.lse_full(out).clone(), "dq": out["dq"].clone(),
           "dk": out["dk"].clone(), "dv": out["dv"].clone()}
    ca.close()
    return res, stats


@pytest.fixture(scope="module")
def baseline():
    return run("none")[0]


def assert_bitwise(a, b):
    for n in a:
        assert torch.equal(a[n], b[n]), n


@pytest.mark.parametrize("mode", ["qol", "qkvol"])
def test_offload_is_bitwise_invisible(baseline, mode):
    res, stats = run(mode)
    assert_bitwise(baseline, res)
    assert stats["n_d2h"] == N - 1 and stats["n_h2d"] == N - 1
    assert stats["ms_d2h"] > 0 and stats["ms_h2d"] > 0


@pytest.mark.parametrize("lookahead", [0, 1, 3, 8])
def test_poison_after_evict(baseline, lookahead):
    res, _ = run("qkvol", offload_chunks=list(range(N)), lookahead=lookahead, poison=True)
    assert_bitwise(baseline, res)


def test_poison_batch2():
    ref, _ = run("none", B=2, seed=3)
    res, _ = run("qkvol", poison=True, B=2, seed=3)
    assert_bitwise(ref, res)


def test_evict_is_bitwise_invisible(baseline):
    res, stats = run("qkvol_evict")
    assert_bitwise(baseline, res)
    S, Hq, Hkv, D = SHAPE["S"], SHAPE["Hq"], SHAPE["Hkv"], SHAPE["D"]
    s = S // N
    per_chunk_h2d = 2 * s * Hq * D * 2 + Hq * s * 4 + 2 * s * Hkv * D * 2
    assert stats["bytes_h2d"] == (N - 1) * per_chunk_h2d
    assert stats["n_d2h"] == N - 1 and stats["n_h2d"] == N - 1


@pytest.mark.parametrize("lookahead", [0, 2])
def test_evict_poison_all_chunks(baseline, lookahead):
    res, _ = run("qkvol_evict", offload_chunks=list(range(N)), lookahead=lookahead, poison=True)
    assert_bitwise(baseline, res)


def test_evict_poison_subset_batch2():
    ref, _ = run("none", B=2, seed=5)
    res, _ = run("qkvol_evict", offload_chunks=[0, 2, 3, 6], poison=True, B=2, seed=5)
    assert_bitwise(ref, res)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_evict_poison_ragged(dtype):
    """Chunk boundaries off the 128-key block grid: the per-chunk dK/dV
    launches of the last backward start their key blocks at c_j."""
    offsets = [0, 77, 300, 301, 1000]
    shape = (1000, 4, 2, 64)
    ref, _ = run("none", dtype=dtype, offsets=offsets, shape=shape, seed=7)
    res, _ = run("qkvol_evict", offload_chunks=[0, 1, 2, 3], dtype=dtype, offsets=offsets, shape=shape,
                 seed=7, poison=True)
    assert_bitwise(ref, res)


def test_evict_state_errors():
    S, Hq, Hkv, D = 1024, 2, 2, 64
    announce("evict state errors")
    inp = make_inputs(1, S, Hq, Hkv, D, torch.bfloat16, seed=0, device="cuda")
    q, k, v, do = inp["q"], inp["k"], inp["v"], inp["do"]

    def status_of(fn, *a):
        try:
            fn(*a)
        except L.SppoError as e:
            return e.status
        return L.SPPO_OK

    # K/V prefetch on a context that does not evict.
    ca = ChunkedAttention(1, S, 4, Hq, Hkv, D, dtype="bf16", offload="qkvol")
    assert status_of(L.sppo_prefetch_kv, ca.ctx, 0, k, v) == L.SPPO_ERR_STATE
    ca.close()

    ca = ChunkedAttention(1, S, 4, Hq, Hkv, D, dtype="bf16", offload="qkvol_evict")
    out = ca.alloc_outputs()
    ctx = ca.ctx
    qc = [ca.chunk_view(q, i) for i in range(4)]
    oc = [ca.chunk_view(out["o"], i) for i in range(4)]
    dc = [ca.chunk_view(do, i) for i in range(4)]
    dqc = [ca.chunk_view(out["dq"], i) for i in range(4)]
    lse = out["lse"]
    bufs = lambda i: L.chunk_bufs(q=qc[i], o=oc[i], lse=lse[i], k=k, v=v)  # noqa: E731
    bwd = lambda i: L.sppo_attn_bwd_chunk(ctx, i, qc[i], k, v, oc[i], lse[i], dc[i], dqc[i],  # noqa: E731
                                          out["dk"], out["dv"])
    for i in range(4):
        L.sppo_attn_fwd_chunk(ctx, i, qc[i], k, v, oc[i], lse[i])
        if i < 3:
            L.sppo_offload_issue(ctx, i, bufs(i))
        if i == 1:
            # the forward walk is not over yet
            assert status_of(L.sppo_prefetch_kv, ctx, 0, k, v) == L.SPPO_ERR_STATE
    assert status_of(L.sppo_prefetch_kv, ctx, 3, k, v) == L.SPPO_ERR_STATE  # never offloaded
    L.sppo_prefetch_kv(ctx, 2, k, v)
    L.sppo_prefetch_kv(ctx, 1, k, v)
    assert status_of(L.sppo_prefetch_kv, ctx, 1, k, v) == L.SPPO_ERR_STATE  # twice
    assert status_of(bwd, 3) == L.SPPO_ERR_STATE                              # chunk 0's K/V missing
    L.sppo_prefetch_kv(ctx, 0, k, v)
    bwd(3)
    assert status_of(L.sppo_prefetch_kv, ctx, 0, k, v) == L.SPPO_ERR_STATE  # backward started
    for i in (2, 1, 0):
        L.sppo_prefetch(ctx, i, bufs(i))
        bwd(i)
    torch.cuda.synchronize()
    ref, _ = run("none", shape=(S, Hq, Hkv, D), offsets=[0, 256, 512, 768, 1024], seed=0)
    assert torch.equal(out["dk"], ref["dk"]) and torch.equal(out["dq"], ref["dq"])
    ca.close()


@pytest.mark.parametrize("mode,B", [("qol", 1), ("qkvol", 1), ("qkvol_evict", 1), ("qkvol_evict", 2)])
def test_partial_offload_rows(mode, B):
    """Sequence-aware offloading: only a row prefix of each chunk leaves the
    device (poisoned after its copy lands); the rest stays resident."""
    S, Hq, Hkv, D = SHAPE["S"], SHAPE["Hq"], SHAPE["Hkv"], SHAPE["D"]
    s = S // N
    rows = [s // 2, 0, 100, s, 37, s - 1, 1, 64]
    ref = run("none", B=B, seed=9)[0]
    res, stats = run(mode, offload_chunks=list(range(N)), poison=True, B=B, seed=9, rows=rows)
    assert_bitwise(ref, res)
    per_row = 2 * Hq * D * 2 + 4 * Hq + (2 * Hkv * D * 2 if mode != "qol" else 0)
    assert stats["bytes_d2h"] == B * sum(rows) * per_row
    assert stats["bytes_h2d"] == B * sum(rows) * per_row - (0 if mode == "qkvol_evict" else
                                                            B * sum(rows) * (per_row - 2 * Hq * D * 2 - 4 * Hq))


def test_offload_rows_errors():
    announce("offload rows errors")
    S, Hq, Hkv, D = 1024, 2, 2, 64
    inp = make_inputs(1, S, Hq, Hkv, D, torch.bfloat16, seed=0, device="cuda")
    ca = ChunkedAttention(1, S, 4, Hq, Hkv, D, dtype="bf16", offload="qol")
    for i, r in ((0, -1), (0, 257), (4, 0)):
        with pytest.raises(L.SppoError) as ei:
            L.sppo_set_offload_rows(ca.ctx, i, r)
        assert ei.value.status == L.SPPO_ERR_INVALID_ARG
    L.sppo_set_offload_rows(ca.ctx, 1, 256)
    out = ca.alloc_outputs()
    L.sppo_attn_fwd_chunk(ca.ctx, 0, ca.chunk_view(inp["q"], 0), inp["k"], inp["v"], ca.chunk_view(out["o"], 0),
                          out["lse"][0])
    with pytest.raises(L.SppoError) as ei:
        L.sppo_set_offload_rows(ca.ctx, 1, 128)  # mid-walk
    assert ei.value.status == L.SPPO_ERR_STATE
    L.sppo_reset(ca.ctx)
    L.sppo_set_offload_rows(ca.ctx, 1, 128)
    assert ca.offload_rows() == [256, 128, 256, 256]
    torch.cuda.synchronize()
    ca.close()


def test_copy_bytes_match_the_offload_set():
    S, Hq, Hkv, D = SHAPE["S"], SHAPE["Hq"], SHAPE["Hkv"], SHAPE["D"]
    s = S // N
    q_bytes = s * Hq * D * 2
    lse_bytes = Hq * s * 4
    kv_bytes = s * Hkv * D * 2
    for mode, per_chunk_d2h in (("qol", 2 * q_bytes + lse_bytes),
                                ("qkvol", 2 * q_bytes + lse_bytes + 2 * kv_bytes)):
        _, stats = run(mode, offload_chunks=[0, 3, 5])
        assert stats["bytes_d2h"] == 3 * per_chunk_d2h, mode
        assert stats["bytes_h2d"] == 3 * (2 * q_bytes + lse_bytes), mode


def test_order_and_state_errors():
    S, Hq, Hkv, D = SHAPE["S"], SHAPE["Hq"], SHAPE["Hkv"], SHAPE["D"]
    announce("order and state errors")
    inp = make_inputs(1, S, Hq, Hkv, D, torch.bfloat16, seed=0, device="cuda")
    ca = ChunkedAttention(1, S, 4, Hq, Hkv, D, dtype="bf16", offload="qol")
    out = ca.alloc_outputs()
    q, k, v, do = inp["q"], inp["k"], inp["v"], inp["do"]
    qc = [ca.chunk_view(q, i) for i in range(4)]
    oc = [ca.chunk_view(out["o"], i) for i in range(4)]
    dc = [ca.chunk_view(do, i) for i in range(4)]
    dqc = [ca.chunk_view(out["dq"], i) for i in range(4)]
    lse = out["lse"]
    ctx = ca.ctx

    def status_of(fn, *a):
        try:
            fn(*a)
        except L.SppoError as e:
            return e.status
        return L.SPPO_OK

    bufs = lambda i: L.chunk_bufs(q=qc[i], o=oc[i], lse=lse[i], k=k, v=v)  # noqa: E731
    assert status_of(L.sppo_attn_fwd_chunk, ctx, 1, qc[1], k, v, oc[1], lse[1]) == L.SPPO_ERR_ORDER
    assert status_of(L.sppo_attn_bwd_chunk, ctx, 3, qc[3], k, v, oc[3], lse[3], dc[3], dqc[3],
                     out["dk"], out["dv"]) == L.SPPO_ERR_ORDER
    # dK and dV must be distinct accumulators (checked before the order)
    assert status_of(L.sppo_attn_bwd_chunk, ctx, 3, qc[3], k, v, oc[3], lse[3], dc[3], dqc[3],
                     out["dk"], out["dk"]) == L.SPPO_ERR_INVALID_ARG
    assert status_of(L.sppo_offload_issue, ctx, 0, bufs(0)) == L.SPPO_ERR_STATE  # before its fwd
    assert status_of(L.sppo_prefetch, ctx, 0, bufs(0)) == L.SPPO_ERR_STATE       # never offloaded
    assert status_of(L.sppo_offload_wait, ctx, 0) == L.SPPO_ERR_STATE
    assert status_of(L.sppo_attn_fwd_chunk, ctx, 7, qc[0], k, v, oc[0], lse[0]) == L.SPPO_ERR_INVALID_ARG
    misaligned = qc[0].data_ptr() + 2
    assert status_of(L.sppo_attn_fwd_chunk, ctx, 0, misaligned, k, v, oc[0], lse[0]) == L.SPPO_ERR_INVALID_ARG
    assert L.sppo_last_error(ctx)
    # A failed call leaves the context usable.
    for i in range(4):
        L.sppo_attn_fwd_chunk(ctx, i, qc[i], k, v, oc[i], lse[i])
        if i < 2:
            L.sppo_offload_issue(ctx, i, bufs(i))
    assert status_of(L.sppo_offload_issue, ctx, 1, bufs(1)) == L.SPPO_ERR_STATE  # twice
    assert status_of(L.sppo_attn_fwd_chunk, ctx, 0, qc[0], k, v, oc[0], lse[0]) == L.SPPO_ERR_ORDER
    for i in (3, 2):
        L.sppo_attn_bwd_chunk(ctx, i, qc[i], k, v, oc[i], lse[i], dc[i], dqc[i], out["dk"], out["dv"])
    # chunk 1 was offloaded and not prefetched: its backward must refuse.
    assert status_of(L.sppo_attn_bwd_chunk, ctx, 1, qc[1], k, v, oc[1], lse[1], dc[1], dqc[1],
                     out["dk"], out["dv"]) == L.SPPO_ERR_STATE
    L.sppo_prefetch(ctx, 1, bufs(1))
    assert status_of(L.sppo_prefetch, ctx, 1, bufs(1)) == L.SPPO_ERR_STATE  # twice
    L.sppo_attn_bwd_chunk(ctx, 1, qc[1], k, v, oc[1], lse[1], dc[1], dqc[1], out["dk"], out["dv"])
    L.sppo_prefetch(ctx, 0, bufs(0))
    L.sppo_attn_bwd_chunk(ctx, 0, qc[0], k, v, oc[0], lse[0], dc[0], dqc[0], out["dk"], out["dv"])
    torch.cuda.synchronize()
    assert torch.isfinite(out["dk"]).all() and torch.isfinite(out["dq"]).all()
    # A new walk starts at fwd(0); reset abandons a partial walk.
    L.sppo_attn_fwd_chunk(ctx, 0, qc[0], k, v, oc[0], lse[0])
    L.sppo_reset(ctx)
    L.sppo_attn_fwd_chunk(ctx, 0, qc[0], k, v, oc[0], lse[0])
    L.sppo_sync(ctx)
    torch.cuda.synchronize()
    ca.close()


def test_offload_on_context_without_offload_is_rejected():
    S, Hq, Hkv, D = 256, 2, 2, 64
    inp = make_inputs(1, S, Hq, Hkv, D, torch.bfloat16, seed=0, device="cuda")
    ca = ChunkedAttention(1, S, 2, Hq, Hkv, D, dtype="bf16", offload="none")
    out = ca.alloc_outputs()
    L.sppo_attn_fwd_chunk(ca.ctx, 0, ca.chunk_view(inp["q"], 0), inp["k"], inp["v"],
                          ca.chunk_view(out["o"], 0), out["lse"][0])
    with pytest.raises(L.SppoError) as ei:
        L.sppo_offload_issue(ca.ctx, 0, L.chunk_bufs(q=inp["q"], o=out["o"], lse=out["lse"][0]))
    assert ei.value.status == L.SPPO_ERR_STATE
    torch.cuda.synchronize()
    ca.close()


def test_arena_frees_offloaded_chunks():
    """Device staging arena (Sec. 5.2: an offloaded chunk's device memory is
    given back once its copy has landed).  With every chunk but the last
    offloaded, the walk holds its saved activations in an arena of 4 chunks
    instead of all 16, gives the bits of the walk without offload,
    and torch's peak of allocated device memory over a walk drops by the
    difference; a second walk allocates nothing."""
    B, S, Hq, Hkv, D = 1, 8192, 8, 2, 128
    n = 16
    res, peak, arena = {}, {}, {}
    for mode in ("none", "qkvol"):
        announce(f"arena memory, offload={mode}")
        inp = make_inputs(B, S, Hq, Hkv, D, torch.bfloat16, seed=21, device="cuda")
        ca = ChunkedAttention(B, S, n, Hq, Hkv, D, dtype="bf16", offload=mode)
        out = ca.alloc_outputs(export=False)
        gc.collect()  # tensors of earlier tests freed now, not in the middle of the measured step
        torch.cuda.synchronize()
        base = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        ca.step(inp, out, poison=(mode != "none"))
        torch.cuda.synchronize()
        peak[mode] = torch.cuda.max_memory_allocated() - base
        arena[mode] = ca.arena.nbytes
        region = ca._planes[0][1]
        inp = make_inputs(B, S, Hq, Hkv, D, torch.bfloat16, seed=21, device="cuda")
        gc.collect()
        torch.cuda.synchronize()
        base = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        ca.step(inp, out)
        torch.cuda.synchronize()
        assert torch.cuda.max_memory_allocated() - base <= 1 << 20, "a walk allocated device memory"
        res[mode] = {k: out[k].clone() for k in ("dq", "dk", "dv")}
        ca.close()
        del inp, out
    for k in res["none"]:
        assert torch.equal(res["none"][k], res["qkvol"][k]), k
    assert arena["none"] == n * region and arena["qkvol"] == 4 * region
    assert peak["none"] - peak["qkvol"] >= 0.9 * (arena["none"] - arena["qkvol"]), (peak, arena)


def test_reset_orders_outstanding_copies():
    """A walk abandoned with offloads and prefetches still in flight, then
    reset: the next walk on the same context and buffers must give exactly
    the bits of a clean run (reset waits for the abandoned copies)."""
    S, Hq, Hkv, D, n = 4096, 4, 2, 128, 8
    announce("reset with copies in flight")
    inp = make_inputs(1, S, Hq, Hkv, D, torch.bfloat16, seed=13, device="cuda")
    clean = ChunkedAttention(1, S, n, Hq, Hkv, D, dtype="bf16", offload="qkvol")
    ref = clean.alloc_outputs()
    clean.step(inp, ref)
    torch.cuda.synchronize()
    clean.close()
    # The abandoned walk runs on other inputs, into the buffers the next walk
    # fills, so a copy of it landing late would change the next walk's bits.
    old = make_inputs(1, S, Hq, Hkv, D, torch.bfloat16, seed=99, device="cuda")
    ca = ChunkedAttention(1, S, n, Hq, Hkv, D, dtype="bf16", offload="qkvol")
    out = ca.alloc_outputs()
    ctx, k, v = ca.ctx, old["k"], old["v"]
    qc = [ca.chunk_view(old["q"], i) for i in range(n)]
    oc = [ca.chunk_view(out["o"], i) for i in range(n)]
    dc = [ca.chunk_view(old["do"], i) for i in range(n)]
    dqc = [ca.chunk_view(out["dq"], i) for i in range(n)]
    lse = out["lse"]
    bufs = lambda i: L.chunk_bufs(q=qc[i], o=oc[i], lse=lse[i], k=k, v=v)  # noqa: E731
    for i in range(n):
        L.sppo_attn_fwd_chunk(ctx, i, qc[i], k, v, oc[i], lse[i])
        L.sppo_offload_issue(ctx, i, bufs(i))
    for i in (n - 1, n - 2, n - 3):
        L.sppo_prefetch(ctx, i, bufs(i))
    L.sppo_attn_bwd_chunk(ctx, n - 1, qc[n - 1], k, v, oc[n - 1], lse[n - 1], dc[n - 1], dqc[n - 1],
                          out["dk"], out["dv"])
    L.sppo_reset(ctx)  # no host synchronisation before it
    ca.step(inp, out)
    torch.cuda.synchronize()
    for name in ("o", "dq", "dk", "dv"):
        assert torch.equal(out[name], ref[name]), name
    assert torch.equal(ca.lse_full(out), torch.cat(ref["lse"], dim=2))
    ca.close()


def test_contexts_of_a_device_share_the_copy_streams():
    """Two contexts (two layers of a model, say) whose walks interleave
    chunk by chunk on one stream: both forward walks, then both backward
    walks in reverse, every offloaded chunk's Q/O/LSE poisoned once its copy
    has landed.  The contexts' copies run on the device's one pair of copy
    streams; each context must still give the bits of its own walk without
    offload."""
    S, Hq, Hkv, D, n = SHAPE["S"], SHAPE["Hq"], SHAPE["Hkv"], SHAPE["D"], N
    seeds = (31, 32)
    refs = [run("none", seed=sd)[0] for sd in seeds]
    announce("two contexts, interleaved walks on shared copy streams")
    inps = [make_inputs(1, S, Hq, Hkv, D, torch.bfloat16, seed=sd, device="cuda") for sd in seeds]
    cas = [ChunkedAttention(1, S, n, Hq, Hkv, D, dtype="bf16", offload="qkvol") for _ in seeds]
    outs = [ca.alloc_outputs() for ca in cas]
    qc = [[ca.chunk_view(inp["q"], i) for i in range(n)] for ca, inp in zip(cas, inps)]
    oc = [[ca.chunk_view(out["o"], i) for i in range(n)] for ca, out in zip(cas, outs)]
    dc = [[ca.chunk_view(inp["do"], i) for i in range(n)] for ca, inp in zip(cas, inps)]
    dqc = [[ca.chunk_view(out["dq"], i) for i in range(n)] for ca, out in zip(cas, outs)]

    def bufs(c, i):
        return L.chunk_bufs(q=qc[c][i], o=oc[c][i], lse=outs[c]["lse"][i], k=inps[c]["k"], v=inps[c]["v"])

    for i in range(n):
        for c in (0, 1):
            L.sppo_attn_fwd_chunk(cas[c].ctx, i, qc[c][i], inps[c]["k"], inps[c]["v"], oc[c][i], outs[c]["lse"][i])
            if i < n - 1:
                L.sppo_offload_issue(cas[c].ctx, i, bufs(c, i))
        for c in (0, 1):
            if i < n - 1:
                L.sppo_offload_wait(cas[c].ctx, i)
                qc[c][i].fill_(float("nan"))
                oc[c][i].fill_(float("nan"))
                outs[c]["lse"][i].fill_(float("nan"))
    for i in reversed(range(n)):
        for c in (1, 0):
            if 0 <= i - 1 <= n - 2:
                L.sppo_prefetch(cas[c].ctx, i - 1, bufs(c, i - 1))
            L.sppo_attn_bwd_chunk(cas[c].ctx, i, qc[c][i], inps[c]["k"], inps[c]["v"], oc[c][i],
                                  outs[c]["lse"][i], dc[c][i], dqc[c][i], outs[c]["dk"], outs[c]["dv"])
    torch.cuda.synchronize()
    for c in (0, 1):
        got = {"o": outs[c]["o"], "lse": cas[c].lse_full(outs[c]), "dq": outs[c]["dq"],
               "dk": outs[c]["dk"], "dv": outs[c]["dv"]}
        assert_bitwise(refs[c], got)
        cas[c].close()


class _Serializer:
    """Stands in for the walk's host pacer: at every chunk boundary the host
    waits until the device, the copy streams included, is idle."""

    def __init__(self, ctx):
        self.ctx = ctx

    def boundary(self, stream):
        torch.cuda.synchronize()
        L.sppo_sync(self.ctx)


@pytest.mark.parametrize("mode", ["qkvol", "qkvol_evict"])
def test_serialized_walk_matches_the_overlapped_one(mode):
    """The same offloading walk with every chunk's work finished (kernels and
    copies) before the next chunk's calls are made, against the walk where
    copies overlap compute: bitwise equal, so no result depends on how the
    copies interleave with the kernels."""
    announce(f"serialized vs overlapped walk, {mode}")
    res = {}
    for name in ("overlapped", "serialized"):
        inp = make_inputs(1, SHAPE["S"], SHAPE["Hq"], SHAPE["Hkv"], SHAPE["D"], torch.bfloat16, seed=23,
                          device="cuda")
        ca = ChunkedAttention(1, SHAPE["S"], N, SHAPE["Hq"], SHAPE["Hkv"], SHAPE["D"], dtype="bf16", offload=mode)
        if name == "serialized":
            ca.pacer = _Serializer(ca.ctx)
        out = ca.alloc_outputs()
        ca.step(inp, out, poison=True)
        torch.cuda.synchronize()
        res[name] = {"o": out["o"].clone(), "lse": ca.lse_full(out).clone(), "dq": out["dq"].clone(),
                     "dk": out["dk"].clone(), "dv": out["dv"].clone()}
        ca.close()
    assert_bitwise(res["overlapped"], res["serialized"])


def test_competing_link_traffic_leaves_results_unchanged():
    """The walk's copies share the host link with large copies of another
    stream, so they land later than they would alone: the backward still
    waits for each prefetch (poisoned dead buffers) and every result stays
    bitwise equal to the walk without offload."""
    announce("walk beside 1 GiB copies on another stream")
    ref, _ = run("none", seed=29)
    nbytes = 1 << 30
    dev = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    host = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    bg = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(bg):
        for _ in range(3):
            host.copy_(dev, non_blocking=True)
            dev.copy_(host, non_blocking=True)
    res, _ = run("qkvol", seed=29, poison=True, lookahead=1)
    torch.cuda.synchronize()
    assert_bitwise(ref, res)
    del dev, host


def test_contexts_on_two_streams_run_concurrently():
    """Two contexts' offloading walks, each on its own stream and enqueued
    back to back with the host unpaced, so their kernels and copies run on
    the device at the same time (each dK/dV launch with its own context's
    tile queues): each gives the bits of its walk run alone."""
    seeds = (41, 42)
    shape = (32768, 8, 2, 128)  # a few ms of device time per walk, so the walks overlap
    refs = [run("qkvol", seed=sd, shape=shape)[0] for sd in seeds]
    announce("two contexts on two streams at once")
    S, Hq, Hkv, D = shape
    inps = [make_inputs(1, S, Hq, Hkv, D, torch.bfloat16, seed=sd, device="cuda") for sd in seeds]
    cas = [ChunkedAttention(1, S, N, Hq, Hkv, D, dtype="bf16", offload="qkvol", host_ahead=0) for _ in seeds]
    outs = [ca.alloc_outputs() for ca in cas]
    for ca in cas:
        ca.prepare()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for ca, inp, out, st in zip(cas, inps, outs, streams):
        ca.step(inp, out, poison=True, stream=st)
    torch.cuda.synchronize()
    for ref, ca, out in zip(refs, cas, outs):
        got = {"o": out["o"], "lse": ca.lse_full(out), "dq": out["dq"], "dk": out["dk"], "dv": out["dv"]}
        assert_bitwise(ref, got)
        ca.close()


def test_contexts_from_two_host_threads():
    """Two host threads each create a context, run an offloading walk with
    poison on a stream of their own and destroy it, twice over (the library
    calls release the interpreter lock, so creation, the shared copy
    streams' reference counts, the walks and destruction interleave): every
    walk gives the bits of the same walk run alone."""
    import threading

    seeds, modes = (51, 52), ("qkvol", "qkvol_evict")
    refs = [run(m, seed=sd)[0] for m, sd in zip(modes, seeds)]
    announce("two host threads, two contexts each")
    S, Hq, Hkv, D = SHAPE["S"], SHAPE["Hq"], SHAPE["Hkv"], SHAPE["D"]
    inps = [make_inputs(1, S, Hq, Hkv, D, torch.bfloat16, seed=sd, device="cuda") for sd in seeds]
    torch.cuda.synchronize()
    results, errors = [[], []], []

    def worker(t):
        try:
            torch.cuda.set_device(0)
            st = torch.cuda.Stream()
            for _ in range(2):
                with torch.cuda.stream(st):
                    ca = ChunkedAttention(1, S, N, Hq, Hkv, D, dtype="bf16", offload=modes[t], host_ahead=1)
                    out = ca.alloc_outputs()
                    inp = {n: x.clone() for n, x in inps[t].items()}  # poison overwrites the offloaded rows of q
                    ca.step(inp, out, poison=True, stream=st)
                    st.synchronize()
                    results[t].append({"o": out["o"].clone(), "lse": ca.lse_full(out).clone(),
                                       "dq": out["dq"].clone(), "dk": out["dk"].clone(), "dv": out["dv"].clone()})
                    st.synchronize()
                    ca.close()
        except Exception as e:  # reported by the main thread
            errors.append(repr(e))

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(2)]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=90)
    assert not any(th.is_alive() for th in threads), "a worker did not finish"
    assert not errors, errors
    for t in range(2):
        assert len(results[t]) == 2
        for got in results[t]:
            assert_bitwise(refs[t], got)
