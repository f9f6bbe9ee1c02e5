"""GPU parity of the full-layer chunk walk (LayerNorm, QKV projection,
chunked attention, output projection, MLP; forward 0..N-1, backward N-1..0)
against the fp64 layer oracle on the same seeded bf16 inputs, plus bitwise
invisibility of the two-level activation management (everything but K/V
offloaded, the device copies poisoned) and the GEMM epilogues on their own.

Gates (bf16 path vs fp64, the layer's activations rounded to bf16 at every
step): per tensor, relative Frobenius error <= 1.2e-2 and max |err| <= 1.5e-2
of max |ref|.  A bf16 rounding per step gives ~0.2-0.4% per element; measured
errors are 3e-3..5.6e-3 on every output (dW_qkv and dgamma_1, at the end of
the backward chain, are the largest), so the gates leave about 2x headroom.
Dropping any term of the backward (a residual path, a LayerNorm gradient, a
projection) moves its outputs by O(1) relative, far above these gates.
"""
import math
import sys

import numpy as np
import pytest
import torch

from oracle import transformer_layer as T
from paper_2503_10377_amd import sppo as L
from paper_2503_10377_amd.chunked_layer import ChunkedLayer
from paper_2503_10377_amd.inputs import make_layer_inputs
from parity import to_np

pytestmark = pytest.mark.gpu

REL, MAXREL = 1.2e-2, 1.5e-2
KEYS = ("y", "dx", "dw_qkv", "dw_o", "dw_1", "dw_2", "dg1", "db1", "dg2", "db2")


def announce(msg):
    print(f"\n[case] {msg}", file=sys.stderr, flush=True)


def run_layer(S, Hq, Hkv, D, offsets, seed=0, offload="none", poison=False, lookahead=2, rows=None, fwd_slots=4):
    announce(f"layer S={S} Hq={Hq} Hkv={Hkv} D={D} offsets={offsets} seed={seed} offload={offload} "
             f"poison={poison} rows={rows}")
    inp, p = make_layer_inputs(S, Hq, Hkv, D, seed, device="cpu")
    host = {k: to_np(v) for k, v in {**inp, **p}.items()}
    dinp = {k: v.cuda() for k, v in inp.items()}
    dp = {k: v.cuda() for k, v in p.items()}
    lay = ChunkedLayer(S, len(offsets) - 1, Hq, Hkv, D, offsets=offsets, offload=offload, fwd_slots=fwd_slots)
    if rows is not None:
        lay.set_offload_rows(rows)
    out = lay.alloc_outputs()
    lay.step(dinp, dp, out, lookahead=lookahead, poison=poison)
    torch.cuda.synchronize()
    got = {k: to_np(out[k]) for k in KEYS}
    lay.close()
    return got, host


def oracle_layer(host, Hq, Hkv, D):
    p = {k: host[k] for k in ("w_qkv", "w_o", "w_1", "w_2", "g1", "b1", "g2", "b2")}
    return T.layer(host["x"], host["dy"], p, Hq, Hkv, D)


def check(got, ref):
    for k in KEYS:
        g, r = got[k], ref[k]
        assert np.isfinite(g).all(), k
        rel = np.linalg.norm(g - r) / np.linalg.norm(r)
        mx = np.abs(g - r).max() / np.abs(r).max()
        print(f"  {k:7s} rel_fro {rel:.2e} max_rel {mx:.2e}", file=sys.stderr, flush=True)
        assert rel <= REL and mx <= MAXREL, (k, rel, mx)


@pytest.mark.parametrize("Hq,Hkv,D,offsets", [
    (2, 2, 128, [0, 128, 256, 384, 512]),
    (4, 2, 64, [0, 100, 101, 300, 512]),     # GQA, ragged chunks incl. a one-row chunk
])
def test_layer_matches_oracle(Hq, Hkv, D, offsets):
    S = offsets[-1]
    got, host = run_layer(S, Hq, Hkv, D, offsets, seed=1)
    check(got, oracle_layer(host, Hq, Hkv, D))


@pytest.mark.parametrize("offload,rows", [("qol", None), ("qkvol", [200, 0, 1, 512]), ("qkvol_evict", None),
                                          ("qkvol_evict", [200, 0, 1, 512])])
def test_layer_offload_is_bitwise_invisible(offload, rows):
    # Q/O/LSE and the extra planes (x, h, a, LayerNorm statistics) of the
    # offloaded chunks are poisoned on the device once copied out; with
    # qkvol_evict so are their K/V cache rows after the forward walk.
    offsets = [0, 256, 512, 768, 1024]
    if rows is not None:
        rows = [min(r, offsets[i + 1] - offsets[i]) for i, r in enumerate(rows)]
    base, host = run_layer(1024, 2, 2, 128, offsets, seed=2)
    got, _ = run_layer(1024, 2, 2, 128, offsets, seed=2, offload=offload, poison=True, lookahead=1, rows=rows)
    for k in KEYS:
        assert np.array_equal(got[k], base[k]), k


def test_layer_tight_arena_is_bitwise_invisible():
    """The smallest arena (fwd_slots 1: each forward chunk reuses the region
    of the chunk just offloaded, after its copy) with lookahead 0, K/V
    evicted, everything dead poisoned."""
    offsets = [0, 200, 201, 600, 1024]
    base, _ = run_layer(1024, 2, 2, 128, offsets, seed=4)
    got, _ = run_layer(1024, 2, 2, 128, offsets, seed=4, offload="qkvol_evict", poison=True, lookahead=0,
                       fwd_slots=1)
    for k in KEYS:
        assert np.array_equal(got[k], base[k]), k


def test_gemm_epilogues_match_numpy():
    # Each epilogue on ragged M (NT) and ragged K (TN) against fp64 NumPy on
    # the same bf16 operands.
    g = torch.Generator().manual_seed(5)
    bf = torch.bfloat16
    M, N, K = 300, 512, 192
    a, b = torch.randn(M, K, generator=g).to(bf), torch.randn(N, K, generator=g).to(bf)
    aux = torch.randn(M, N, generator=g).to(bf)
    ref = to_np(a) @ to_np(b).T
    da, db, dx = a.cuda(), b.cuda(), aux.cuda()
    s = torch.cuda.current_stream().cuda_stream
    cases = {"bf16": ref, "add_bf16": ref + to_np(aux), "f32": ref}
    for epi, r in cases.items():
        c = torch.empty(M, N, device="cuda", dtype=torch.float32 if epi == "f32" else bf)
        L.sppo_gemm_bf16("nt", M, N, K, da, K, db, K, c, N, epi, dx, N, stream=s)
        torch.cuda.synchronize()
        tol = 1e-5 if epi == "f32" else 8e-3
        assert np.abs(to_np(c) - r).max() <= tol * np.abs(r).max(), epi
    pre = torch.empty(M, N, device="cuda", dtype=bf)
    c = torch.empty(M, N, device="cuda", dtype=bf)
    L.sppo_gemm_bf16("nt", M, N, K, da, K, db, K, c, N, "gelu", pre, N, stream=s)
    torch.cuda.synchronize()
    assert np.abs(to_np(pre) - ref).max() <= 8e-3 * np.abs(ref).max()
    assert np.abs(to_np(c) - T.gelu(to_np(pre))).max() <= 8e-3 * np.abs(ref).max()
    L.sppo_gemm_bf16("nt", M, N, K, da, K, db, K, c, N, "dgelu", dx, N, stream=s)
    torch.cuda.synchronize()
    r = ref * T.gelu_grad(to_np(aux))
    assert np.abs(to_np(c) - r).max() <= 8e-3 * np.abs(r).max()
    # TN with K ragged, accumulating onto ones
    Mt, Nt, Kt = 256, 512, 301
    at, bt = torch.randn(Kt, Mt, generator=g).to(bf), torch.randn(Kt, Nt, generator=g).to(bf)
    c = torch.ones(Mt, Nt, device="cuda")
    L.sppo_gemm_bf16("tn", Mt, Nt, Kt, at.cuda(), Mt, bt.cuda(), Nt, c, Nt, "acc_f32", stream=s)
    torch.cuda.synchronize()
    r = to_np(at).T @ to_np(bt) + 1.0
    assert np.abs(to_np(c) - r).max() <= 1e-5 * np.abs(r).max()
