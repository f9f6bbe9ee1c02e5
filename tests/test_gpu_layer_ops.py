"""The full-layer building blocks on their own, through the C ABI, at the
shapes the layer tests do not reach: LayerNorm widths that take each of the
kernel's register layouts (up to 8192), ragged row counts and strides, both
gradient modes (overwrite, accumulate); GEMMs with ragged M, N and K and
leading dimensions larger than the width; the transpose on ragged shapes; the
dQKV packing.  References: the fp64 oracle's LayerNorm and GELU, NumPy
products on the same bf16 operands.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import transformer_layer as T
from paper_2503_10377_amd import sppo as L
from parity import to_np

pytestmark = pytest.mark.gpu
bf = torch.bfloat16


def announce(msg):
    print(f"\n[case] {msg}", file=sys.stderr, flush=True)


def stream():
    return torch.cuda.current_stream().cuda_stream


@pytest.mark.parametrize("rows,H,ld", [(1, 8, 8), (33, 256, 264), (300, 2056, 2056), (65, 4096, 4104),
                                       (17, 6144, 6144), (40, 8192, 8192)])
def test_layernorm_fwd_bwd(rows, H, ld):
    announce(f"layernorm rows={rows} H={H} ld={ld}")
    g = torch.Generator().manual_seed(rows + H)
    x = (torch.randn(rows, ld, generator=g) * 2 + 0.5).to(bf)
    dy = torch.randn(rows, ld, generator=g).to(bf)
    dres = torch.randn(rows, ld, generator=g).to(bf)
    gamma, beta = 1 + 0.1 * torch.randn(H, generator=g), 0.1 * torch.randn(H, generator=g)
    xd, dyd, dresd = x.cuda(), dy.cuda(), dres.cuda()
    gd, bd = gamma.cuda(), beta.cuda()
    y = torch.full((rows, ld), float("nan"), device="cuda", dtype=bf)
    mean, rstd = torch.empty(rows, device="cuda"), torch.empty(rows, device="cuda")
    L.sppo_layernorm_fwd(rows, H, xd, ld, gd, bd, 1e-5, y, ld, mean, rstd, stream=stream())
    ws_bytes = L.sppo_layernorm_bwd_workspace(rows, H)
    ws = torch.empty(ws_bytes // 4, device="cuda")
    dx = torch.empty(rows, ld, device="cuda", dtype=bf)
    dg, db = torch.full((H,), 0.25, device="cuda"), torch.full((H,), -0.5, device="cuda")
    L.sppo_layernorm_bwd(rows, H, xd, ld, gd, mean, rstd, dyd, ld, dresd, ld, dx, ld, dg, db, ws, ws_bytes,
                         accumulate=1, stream=stream())
    torch.cuda.synchronize()
    xh, dyh, dresh = to_np(x)[:, :H], to_np(dy)[:, :H], to_np(dres)[:, :H]
    ref_y, ref_m, ref_r = T.layer_norm(xh, to_np(gamma), to_np(beta))
    assert torch.isnan(y[:, H:]).all(), "columns past H written"
    got_y = to_np(y[:, :H])
    assert np.abs(got_y - ref_y).max() <= 8e-3 * np.abs(ref_y).max()
    np.testing.assert_allclose(to_np(mean), ref_m, rtol=1e-5, atol=1e-5)
    np.testing.assert_allclose(to_np(rstd), ref_r, rtol=1e-4)
    ref_dx, ref_dg, ref_db = T.layer_norm_bwd(xh, to_np(gamma), ref_m, ref_r, dyh)
    ref_dx = ref_dx + dresh
    assert np.abs(to_np(dx[:, :H]) - ref_dx).max() <= 1e-2 * np.abs(ref_dx).max()
    np.testing.assert_allclose(to_np(dg), ref_dg + 0.25, rtol=2e-4, atol=2e-4 * np.abs(ref_dg).max())
    np.testing.assert_allclose(to_np(db), ref_db - 0.5, rtol=2e-4, atol=2e-4 * np.abs(ref_db).max())
    # overwrite mode, twice in a row: the same bits each time
    outs = []
    for _ in range(2):
        L.sppo_layernorm_bwd(rows, H, xd, ld, gd, mean, rstd, dyd, ld, dresd, ld, dx, ld, dg, db, ws, ws_bytes,
                             accumulate=0, stream=stream())
        torch.cuda.synchronize()
        outs.append((dg.clone(), db.clone()))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
    np.testing.assert_allclose(to_np(dg), ref_dg, rtol=2e-4, atol=2e-4 * np.abs(ref_dg).max())


@pytest.mark.parametrize("M,N,K,ldx", [(1, 8, 64, 0), (255, 200, 128, 8), (257, 264, 192, 0), (3000, 1032, 64, 64)])
def test_gemm_nt_ragged(M, N, K, ldx):
    announce(f"gemm nt M={M} N={N} K={K} ld extra={ldx}")
    g = torch.Generator().manual_seed(M + N + K)
    lda, ldb, ldc = K + ldx, K + ldx, N + ldx
    a, b = torch.randn(M, lda, generator=g).to(bf), torch.randn(N, ldb, generator=g).to(bf)
    c = torch.full((M, ldc), 7.0, device="cuda", dtype=bf)
    L.sppo_gemm_bf16("nt", M, N, K, a.cuda(), lda, b.cuda(), ldb, c, ldc, stream=stream())
    torch.cuda.synchronize()
    ref = to_np(a)[:, :K] @ to_np(b)[:, :K].T
    got = to_np(c)
    assert np.abs(got[:, :N] - ref).max() <= 8e-3 * np.abs(ref).max()
    assert np.all(got[:, N:] == 7.0), "columns past N written"


@pytest.mark.parametrize("M,N,K", [(256, 256, 1), (512, 768, 77), (256, 1024, 4097)])
def test_gemm_tn_ragged_k(M, N, K):
    announce(f"gemm tn M={M} N={N} K={K}")
    g = torch.Generator().manual_seed(M + N + K)
    a, b = torch.randn(K, M, generator=g).to(bf), torch.randn(K, N, generator=g).to(bf)
    c = torch.zeros(M, N, device="cuda")
    L.sppo_gemm_bf16("tn", M, N, K, a.cuda(), M, b.cuda(), N, c, N, "f32", stream=stream())
    torch.cuda.synchronize()
    ref = to_np(a).T @ to_np(b)
    assert np.abs(to_np(c) - ref).max() <= 1e-5 * np.abs(ref).max() + 1e-6


@pytest.mark.parametrize("R,C", [(1, 1), (63, 65), (130, 70), (4096, 12288)])
def test_transpose(R, C):
    announce(f"transpose {R}x{C}")
    x = torch.randn(R, C).to(bf)
    y = torch.empty(C, R, device="cuda", dtype=bf)
    L.sppo_transpose_bf16(x.cuda(), y, R, C, stream=stream())
    torch.cuda.synchronize()
    assert torch.equal(y.cpu(), x.t().contiguous())


def test_gelu_and_pack():
    announce("gelu and dqkv pack")
    x = (torch.randn(1000, 24) * 3).to(bf)
    y = torch.empty_like(x, device="cuda")
    L.sppo_gelu_bf16(x.cuda(), y, x.numel(), stream=stream())
    torch.cuda.synchronize()
    ref = T.gelu(to_np(x))
    assert np.abs(to_np(y) - ref).max() <= 8e-3 * np.abs(ref).max()
    rows, wq, wkv, S, c0 = 37, 64, 32, 100, 50
    dq = torch.randn(rows, wq).to(bf)
    dk, dv = torch.randn(S, wkv), torch.randn(S, wkv)
    out = torch.empty(rows, wq + 2 * wkv, device="cuda", dtype=bf)
    L.sppo_pack_qkv_grad(rows, wq, wkv, dq.cuda(), dk.cuda(), dv.cuda(), c0, out, stream=stream())
    torch.cuda.synchronize()
    ref = torch.cat([dq, dk[c0:c0 + rows].to(bf), dv[c0:c0 + rows].to(bf)], dim=1)
    assert torch.equal(out.cpu(), ref)


def test_layernorm_epsilon_reaches_the_kernel():
    """Rows of small variance (std 0.02) with eps = 1e-3 against the oracle's
    LayerNorm at the same eps: there 1/sqrt(var + eps) is 27% below
    1/sqrt(var), so a kernel that kept its own eps would miss by far more
    than the gate."""
    rows, H = 9, 256
    announce(f"layernorm eps rows={rows} H={H}")
    g = torch.Generator().manual_seed(5)
    x = (0.02 * torch.randn(rows, H, generator=g) + 0.3).to(bf)
    dy = torch.randn(rows, H, generator=g).to(bf)
    gamma, beta = 1 + 0.1 * torch.randn(H, generator=g), 0.1 * torch.randn(H, generator=g)
    eps = 1e-3
    y = torch.empty(rows, H, device="cuda", dtype=bf)
    mean, rstd = torch.empty(rows, device="cuda"), torch.empty(rows, device="cuda")
    xd, gd = x.cuda(), gamma.cuda()
    L.sppo_layernorm_fwd(rows, H, xd, H, gd, beta.cuda(), eps, y, H, mean, rstd, stream=stream())
    ws_bytes = L.sppo_layernorm_bwd_workspace(rows, H)
    ws = torch.empty(ws_bytes // 4, device="cuda")
    dx = torch.empty(rows, H, device="cuda", dtype=bf)
    zeros = torch.zeros(rows, H, device="cuda", dtype=bf)
    dg, db = torch.empty(H, device="cuda"), torch.empty(H, device="cuda")
    L.sppo_layernorm_bwd(rows, H, xd, H, gd, mean, rstd, dy.cuda(), H, zeros, H, dx, H, dg, db, ws, ws_bytes,
                         accumulate=0, stream=stream())
    torch.cuda.synchronize()
    xh = to_np(x)
    ref_y, ref_m, ref_r = T.layer_norm(xh, to_np(gamma), to_np(beta), eps=eps)
    assert np.abs(1 / np.sqrt(xh.var(axis=1) + eps) * np.sqrt(xh.var(axis=1)) - 1).min() > 0.2  # eps matters
    np.testing.assert_allclose(to_np(rstd), ref_r, rtol=1e-4)
    assert np.abs(to_np(y) - ref_y).max() <= 8e-3 * np.abs(ref_y).max()
    ref_dx, ref_dg, ref_db = T.layer_norm_bwd(xh, to_np(gamma), ref_m, ref_r, to_np(dy))
    assert np.abs(to_np(dx) - ref_dx).max() <= 1e-2 * np.abs(ref_dx).max()
    np.testing.assert_allclose(to_np(dg), ref_dg, rtol=2e-4, atol=2e-4 * np.abs(ref_dg).max())
