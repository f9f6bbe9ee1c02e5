"""The backward entry point that allocates nothing
(sppo_attn_bwd_chunk_noalloc) against sppo_attn_bwd_chunk, through the C
ABI: the same reverse walk of chunk backwards on the same inputs, once with
a context and once with the static-workspace variant, must give the same
bits -- a larger problem first, then a smaller one right after it on the
same GPU (the workspace keeps the previous call's contents), in bf16 and
fp32.  Also: no device memory is allocated by the variant's calls."""
import sys

import pytest
import torch

from paper_2503_10377_amd import sppo as L
from paper_2503_10377_amd.chunked import ChunkedAttention
from paper_2503_10377_amd.inputs import make_inputs

pytestmark = pytest.mark.gpu


def announce(msg):
    print(f"\n[case] {msg}", file=sys.stderr, flush=True)


def walk_both(B, S, Hq, Hkv, D, dtype, offsets, seed, scale=0.0):
    """dq, dk, dv of the reverse walk N-1..0 with the context's backward and
    with the allocation-free one (chunk N-1 overwrites dK/dV, the rest add);
    scale 0 is 1/sqrt(D)."""
    announce(f"no-alloc walk B={B} S={S} Hq={Hq} Hkv={Hkv} D={D} {dtype} offsets={offsets} scale={scale}")
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    inp = make_inputs(B, S, Hq, Hkv, D, tdt, seed=seed, device="cuda")
    ca = ChunkedAttention(B, S, len(offsets) - 1, Hq, Hkv, D, dtype=dtype, offsets=offsets, scale=scale)
    N = ca.N
    out = ca.alloc_outputs()
    qc = [ca.chunk_view(inp["q"], i) for i in range(N)]
    dc = [ca.chunk_view(inp["do"], i) for i in range(N)]
    oc = [ca.chunk_view(out["o"], i) for i in range(N)]
    for i in range(N):
        L.sppo_attn_fwd_chunk(ca.ctx, i, qc[i], inp["k"], inp["v"], oc[i], out["lse"][i])
    res = {}
    for name in ("ctx", "noalloc"):
        dq = [torch.empty_like(qc[i]) for i in range(N)]
        dk = torch.full((B, S, Hkv, D), float("nan"), dtype=torch.float32, device="cuda")
        dv = torch.full_like(dk, float("nan"))
        torch.cuda.synchronize()
        before = torch.cuda.memory_allocated()
        for i in reversed(range(N)):
            if name == "ctx":
                L.sppo_attn_bwd_chunk(ca.ctx, i, qc[i], inp["k"], inp["v"], oc[i], out["lse"][i], dc[i], dq[i],
                                      dk, dv)
            else:
                L.sppo_attn_bwd_chunk_noalloc(B, S, ca.offsets[i], ca.offsets[i + 1], Hq, Hkv, D, dtype, scale,
                                              0 if i == N - 1 else 1, qc[i], inp["k"], inp["v"], oc[i],
                                              out["lse"][i], dc[i], dq[i], dk, dv)
        torch.cuda.synchronize()
        assert torch.cuda.memory_allocated() <= before  # the variant allocated nothing
        res[name] = (dq, dk, dv)
    ca.close()
    return res


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_backward_matches_the_context_backward(dtype):
    big = walk_both(1, 4096, 8, 2, 128, dtype, [0, 1024, 2048, 3072, 4096], seed=31)
    small = walk_both(2, 1000, 2, 1, 64, dtype, [0, 77, 300, 301, 1000], seed=32)
    scaled = walk_both(2, 1000, 2, 1, 64, dtype, [0, 77, 300, 301, 1000], seed=32, scale=0.15)
    for res in (big, small, scaled):
        (dq_a, dk_a, dv_a), (dq_b, dk_b, dv_b) = res["ctx"], res["noalloc"]
        for a, b in zip(dq_a, dq_b):
            assert torch.equal(a, b)
        assert torch.equal(dk_a, dk_b) and torch.equal(dv_a, dv_b)
        assert torch.isfinite(dk_b).all()
    # the explicit scale reached the kernels (the walks differ only in it)
    assert not torch.equal(small["noalloc"][1], scaled["noalloc"][1])


def test_noalloc_rejects_a_chunk_beyond_the_workspace():
    t = torch.empty(16, dtype=torch.float32, device="cuda")
    with pytest.raises(L.SppoError) as ei:
        L.sppo_attn_bwd_chunk_noalloc(1, 65536, 0, 65536, 32, 32, 128, "bf16", 0.0, 0, t, t, t, t, t, t, t, t,
                                      t.data_ptr() + 16)
    assert ei.value.status == L.SPPO_ERR_UNSUPPORTED
    assert "workspace" in L.sppo_last_error(None)
