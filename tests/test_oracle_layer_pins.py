"""Pins of the full-layer oracle (oracle/transformer_layer.py) to things
other than itself: central finite differences of L = sum(dy * y) for every
input and parameter, LayerNorm moments, GELU identities, the closed form with
zero output projections, and the subsequence walk == the unchunked layer."""
import math

import numpy as np
import pytest

from oracle import transformer_layer as T

HQ, HKV, D = 2, 1, 4
H = HQ * D


def params(rng, h=H, hq=HQ, hkv=HKV, d=D, scale=0.5):
    wt = (hq + 2 * hkv) * d
    return dict(w_qkv=rng.normal(0, scale, (h, wt)), w_o=rng.normal(0, scale, (hq * d, h)),
                w_1=rng.normal(0, scale, (h, 4 * h)), w_2=rng.normal(0, scale, (4 * h, h)),
                g1=rng.normal(1, 0.2, h), b1=rng.normal(0, 0.2, h), g2=rng.normal(1, 0.2, h), b2=rng.normal(0, 0.2, h))


def loss(x, dy, p):
    return float((T.layer_forward(x, p, HQ, HKV, D)["y"] * dy).sum())


def test_layer_norm_moments():
    rng = np.random.default_rng(0)
    x = rng.normal(3.0, 2.0, (6, 16))
    y, mean, rstd = T.layer_norm(x, np.ones(16), np.zeros(16))
    var = x.var(axis=1)
    np.testing.assert_allclose(mean, x.mean(axis=1), rtol=0, atol=1e-12)
    np.testing.assert_allclose(y.mean(axis=1), 0.0, atol=1e-12)
    np.testing.assert_allclose((y * y).mean(axis=1), var / (var + T.EPS), rtol=1e-12)
    np.testing.assert_allclose(rstd, 1 / np.sqrt(var + T.EPS), rtol=1e-12)


def test_layer_norm_bwd_matches_finite_differences():
    rng = np.random.default_rng(1)
    x, g, b, dy = rng.normal(size=(3, 8)), rng.normal(size=8), rng.normal(size=8), rng.normal(size=(3, 8))
    _, mean, rstd = T.layer_norm(x, g, b)
    dx, dg, db = T.layer_norm_bwd(x, g, mean, rstd, dy)
    f = lambda x_, g_, b_: float((T.layer_norm(x_, g_, b_)[0] * dy).sum())
    e = 1e-6
    for idx in np.ndindex(x.shape):
        xp, xm = x.copy(), x.copy()
        xp[idx] += e
        xm[idx] -= e
        assert abs((f(xp, g, b) - f(xm, g, b)) / (2 * e) - dx[idx]) < 1e-7
    for j in range(8):
        gp, gm, bp, bm = g.copy(), g.copy(), b.copy(), b.copy()
        gp[j] += e; gm[j] -= e; bp[j] += e; bm[j] -= e
        assert abs((f(x, gp, b) - f(x, gm, b)) / (2 * e) - dg[j]) < 1e-7
        assert abs((f(x, g, bp) - f(x, g, bm)) / (2 * e) - db[j]) < 1e-7


def test_gelu_identities():
    a = np.linspace(-6, 6, 97)
    np.testing.assert_allclose(T.gelu(a) - T.gelu(-a), a, atol=1e-14)
    assert T.gelu(0.0) == 0.0 and T.gelu_grad(0.0) == 0.5
    np.testing.assert_allclose(T.gelu(np.array([10.0, -10.0])), [10.0, 0.0], atol=1e-12)
    e = 1e-6
    np.testing.assert_allclose(T.gelu_grad(a), (T.gelu(a + e) - T.gelu(a - e)) / (2 * e), atol=1e-8)
    # the tanh form at a = 1: 0.5 (1 + tanh(sqrt(2/pi) * 1.044715))
    assert abs(T.gelu(1.0) - 0.5 * (1 + math.tanh(math.sqrt(2 / math.pi) * 1.044715))) < 1e-15


def test_layer_gradients_match_finite_differences():
    rng = np.random.default_rng(2)
    S = 5
    p = params(rng)
    x, dy = rng.normal(size=(S, H)), rng.normal(size=(S, H))
    f = T.layer_forward(x, p, HQ, HKV, D)
    g = T.layer_backward(x, dy, p, f, HQ, HKV, D)
    e = 1e-6

    def fd_x(idx):
        xp, xm = x.copy(), x.copy()
        xp[idx] += e
        xm[idx] -= e
        return (loss(xp, dy, p) - loss(xm, dy, p)) / (2 * e)

    for idx in np.ndindex(x.shape):
        assert abs(fd_x(idx) - g["dx"][idx]) < 1e-6 * max(1.0, abs(g["dx"][idx]))
    name_of = dict(w_qkv="dw_qkv", w_o="dw_o", w_1="dw_1", w_2="dw_2", g1="dg1", b1="db1", g2="dg2", b2="db2")
    for name, gname in name_of.items():
        w = p[name]
        picks = [np.unravel_index(k, w.shape) for k in rng.choice(w.size, size=min(6, w.size), replace=False)]
        for idx in picks:
            pp = {k: v.copy() for k, v in p.items()}
            pm = {k: v.copy() for k, v in p.items()}
            pp[name][idx] += e
            pm[name][idx] -= e
            num = (loss(x, dy, pp) - loss(x, dy, pm)) / (2 * e)
            assert abs(num - g[gname][idx]) < 1e-6 * max(1.0, abs(num)), (name, idx)


def test_zero_output_projections_make_the_layer_the_identity():
    rng = np.random.default_rng(3)
    p = params(rng)
    p["w_o"][:] = 0.0
    p["w_2"][:] = 0.0
    x, dy = rng.normal(size=(7, H)), rng.normal(size=(7, H))
    out = T.layer(x, dy, p, HQ, HKV, D)
    np.testing.assert_array_equal(out["y"], x)
    np.testing.assert_allclose(out["dx"], dy, atol=1e-14)
    np.testing.assert_array_equal(out["dw_qkv"], 0.0)
    np.testing.assert_array_equal(out["dw_1"], 0.0)
    assert np.abs(out["dw_2"]).max() > 0 and np.abs(out["dw_o"]).max() > 0


@pytest.mark.parametrize("offsets", [[0, 3, 4, 9, 12], [0, 12], [0, 1, 2, 3, 12]])
def test_chunked_walk_equals_unchunked_layer(offsets):
    rng = np.random.default_rng(4)
    hq, hkv, d = 4, 2, 4
    h = hq * d
    p = params(rng, h=h, hq=hq, hkv=hkv, d=d)
    x, dy = rng.normal(size=(12, h)), rng.normal(size=(12, h))
    ref = T.layer(x, dy, p, hq, hkv, d)
    got = T.chunked_layer(x, dy, p, hq, hkv, d, offsets)
    for key, val in ref.items():
        np.testing.assert_allclose(got[key], val, rtol=1e-10, atol=1e-11, err_msg=key)


def test_gelu_tanh_form_is_within_its_error_of_the_exact_gelu():
    # The tanh form approximates x Phi(x) to within 4.8e-4 everywhere; a wrong
    # constant (0.04715 for 0.044715, or sqrt(1/pi)) is off by 1e-3 or more.
    a = np.linspace(-8, 8, 20001)
    exact = a * 0.5 * (1 + np.array([math.erf(v / math.sqrt(2)) for v in a]))
    err = np.abs(T.gelu(a) - exact)
    assert err.max() < 4.8e-4
    assert err.max() > 4.6e-4  # the approximation's own error, not a fit to the exact one


def test_layer_norm_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(5)
    x = rng.normal(1.0, 3.0, (9, 24))
    g, b = rng.normal(1, 0.2, 24), rng.normal(0, 0.2, 24)
    y, mean, rstd = T.layer_norm(x, g, b)
    ref = torch.nn.functional.layer_norm(torch.tensor(x), (24,), torch.tensor(g), torch.tensor(b), eps=T.EPS)
    np.testing.assert_allclose(y, ref.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("hq,hkv", [(2, 2), (4, 2)])
def test_layer_matches_torch_autograd(hq, hkv):
    # The pre-LayerNorm GPT block built from torch's own LayerNorm, tanh GELU
    # and causal scaled-dot-product attention in fp64, differentiated by
    # autograd: an implementation and a gradient derived independently of
    # the oracle's hand-written chain rule.
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    rng = np.random.default_rng(6)
    d, S = 4, 11
    h = hq * d
    p = params(rng, h=h, hq=hq, hkv=hkv, d=d)
    x, dy = rng.normal(size=(S, h)), rng.normal(size=(S, h))
    tp = {k: torch.tensor(v, requires_grad=True) for k, v in p.items()}
    tx = torch.tensor(x, requires_grad=True)
    u = F.layer_norm(tx, (h,), tp["g1"], tp["b1"], eps=T.EPS)
    qkv = u @ tp["w_qkv"]
    q = qkv[:, :hq * d].reshape(S, hq, d).transpose(0, 1)
    k = qkv[:, hq * d:(hq + hkv) * d].reshape(S, hkv, d).transpose(0, 1)
    v = qkv[:, (hq + hkv) * d:].reshape(S, hkv, d).transpose(0, 1)
    k, v = k.repeat_interleave(hq // hkv, dim=0), v.repeat_interleave(hq // hkv, dim=0)
    o = F.scaled_dot_product_attention(q[None], k[None], v[None], is_causal=True)[0]
    hh = tx + o.transpose(0, 1).reshape(S, hq * d) @ tp["w_o"]
    z = F.layer_norm(hh, (h,), tp["g2"], tp["b2"], eps=T.EPS)
    y = hh + F.gelu(z @ tp["w_1"], approximate="tanh") @ tp["w_2"]
    (y * torch.tensor(dy)).sum().backward()
    got = T.layer(x, dy, p, hq, hkv, d)
    np.testing.assert_allclose(got["y"], y.detach().numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(got["dx"], tx.grad.numpy(), rtol=1e-10, atol=1e-11)
    for name in ("w_qkv", "w_o", "w_1", "w_2"):
        np.testing.assert_allclose(got["d" + name], tp[name].grad.numpy(), rtol=1e-10, atol=1e-11, err_msg=name)
    for name, key in (("g1", "dg1"), ("b1", "db1"), ("g2", "dg2"), ("b2", "db2")):
        np.testing.assert_allclose(got[key], tp[name].grad.numpy(), rtol=1e-10, atol=1e-11, err_msg=name)


@pytest.mark.parametrize("hq,hkv", [(2, 1), (4, 2)])
def test_sampled_rows_equal_the_full_forward(hq, hkv):
    # y at chosen rows, from a longer prefix, equals those rows of the full
    # forward (causality: later rows of the prefix do not matter).
    rng = np.random.default_rng(7)
    d, S = 4, 13
    h = hq * d
    p = params(rng, h=h, hq=hq, hkv=hkv, d=d)
    x = rng.normal(size=(S, h))
    full = T.layer_forward(x, p, hq, hkv, d)["y"]
    rows = [0, 1, 5, 11]
    got = T.layer_forward_rows(x, p, rows, hq, hkv, d)
    np.testing.assert_allclose(got, full[rows], rtol=1e-12, atol=1e-12)
    got_short = T.layer_forward_rows(x[:12], p, rows, hq, hkv, d)
    np.testing.assert_allclose(got_short, full[rows], rtol=1e-12, atol=1e-12)
