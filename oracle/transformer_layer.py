"""fp64 oracle: one full transformer layer over a causal sequence, its
analytic gradient, and the subsequence (chunk) walk of both.

TEST INFRASTRUCTURE ONLY -- never imported by the product path.

The paper trains models of the "GPT architecture" (Sec. 7) and counts a
subsequence's per-layer tensors -- the attention's Q, K, V, its output, the
projections and the MLP -- as the activations that two-level management
keeps (K/V) or offloads (the rest) (Sec. 5.1).  It does not write the
block's algebra out; the reading here is the standard pre-LayerNorm GPT
block with no biases on the projections and an MLP of width 4H:

    u = LN1(x)                         LN(x) = (x - mean) / sqrt(var + eps) * gamma + beta
    q, k, v = u Wq, u Wk, u Wv         [Wq | Wk | Wv] = W_qkv, [H, (Hq + 2 Hkv) D]
    O = causal attention(q, k, v)      (oracle.causal_attention; GQA by head groups)
    h = x + O Wo
    z = LN2(h)
    a = z W1,  g = gelu(a)             gelu(a) = a/2 (1 + tanh(sqrt(2/pi)(a + 0.044715 a^3)))
    y = h + g W2

with x, y [S, H] (batch 1, H = Hq D), biased variance, eps = 1e-5.  The
backward is the gradient of L = sum(dy * y) for a given dy; every step is
the chain rule of the line above it, written out below.

The chunked walk follows the paper's subsequence schedule: the forward of
chunk i (rows [c_i, c_{i+1})) appends its K/V rows to the cache and attends
to rows [0, c_{i+1}) (Sec. 5.1); the backward runs i = N-1..0, accumulating
dK/dV across chunks and the weight gradients across chunks (Sec. 5.2).
Everything but attention acts row by row, so the walk is an exact rewrite of
the unchunked layer (up to the order of fp64 sums).

Pins (tests/test_oracle_layer_pins.py): central finite differences of L for
every input and parameter; the LayerNorm's moments; gelu's identities
gelu(x) - gelu(-x) = x, gelu'(0) = 1/2 and its finite difference; the closed
form Wo = W2 = 0 (then y = x and dx = dy); the walk equals the unchunked
layer; y at sampled rows from a prefix equals those rows of the full forward.
"""
from __future__ import annotations

import math

import numpy as np

from .causal_attention import attention_bwd, attention_fwd, chunked_attention_bwd, chunked_attention_fwd

EPS = 1e-5
_K0 = math.sqrt(2.0 / math.pi)
_K1 = 0.044715


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def layer_norm(x, gamma, beta, eps=EPS):
    """Row-wise LayerNorm with the biased variance.  Returns (y, mean, rstd)."""
    x = _f64(x)
    mean = x.mean(axis=1)
    var = ((x - mean[:, None]) ** 2).mean(axis=1)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mean[:, None]) * rstd[:, None]
    return xhat * _f64(gamma) + _f64(beta), mean, rstd


def layer_norm_bwd(x, gamma, mean, rstd, dy):
    """Gradient of sum(dy * LN(x)).  With xhat = (x - mean) rstd and
    g = dy gamma: dx = rstd (g - mean_j g - xhat mean_j(g xhat)); dgamma =
    sum_rows dy xhat; dbeta = sum_rows dy.  Returns (dx, dgamma, dbeta)."""
    x, dy = _f64(x), _f64(dy)
    xhat = (x - _f64(mean)[:, None]) * _f64(rstd)[:, None]
    g = dy * _f64(gamma)
    dx = _f64(rstd)[:, None] * (g - g.mean(axis=1, keepdims=True) - xhat * (g * xhat).mean(axis=1, keepdims=True))
    return dx, (dy * xhat).sum(axis=0), dy.sum(axis=0)


def gelu(a):
    a = _f64(a)
    return 0.5 * a * (1.0 + np.tanh(_K0 * (a + _K1 * a ** 3)))


def gelu_grad(a):
    """d gelu / da = (1 + t)/2 + a (1 - t^2) K0 (1 + 3 K1 a^2) / 2, t = tanh(K0 (a + K1 a^3))."""
    a = _f64(a)
    t = np.tanh(_K0 * (a + _K1 * a ** 3))
    return 0.5 * (1.0 + t) + 0.5 * a * (1.0 - t * t) * _K0 * (1.0 + 3.0 * _K1 * a * a)


def _split_qkv(qkv, hq, hkv, d):
    s = qkv.shape[0]
    q = qkv[:, : hq * d].reshape(1, s, hq, d)
    k = qkv[:, hq * d: (hq + hkv) * d].reshape(1, s, hkv, d)
    v = qkv[:, (hq + hkv) * d:].reshape(1, s, hkv, d)
    return q, k, v


def layer_forward(x, p, hq, hkv, d, scale=None):
    """Unchunked layer.  p: dict with w_qkv, w_o, w_1, w_2, g1, b1, g2, b2.
    Returns a dict with y and the intermediates the backward uses."""
    x = _f64(x)
    S, H = x.shape
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    u, m1, r1 = layer_norm(x, p["g1"], p["b1"])
    q, k, v = _split_qkv(u @ _f64(p["w_qkv"]), hq, hkv, d)
    o4, lse = attention_fwd(q, k, v, scale)
    o = o4.reshape(S, hq * d)
    h = x + o @ _f64(p["w_o"])
    z, m2, r2 = layer_norm(h, p["g2"], p["b2"])
    a = z @ _f64(p["w_1"])
    g = gelu(a)
    y = h + g @ _f64(p["w_2"])
    return dict(y=y, u=u, q=q, k=k, v=v, o=o, o4=o4, lse=lse, h=h, z=z, a=a, g=g, m1=m1, r1=r1, m2=m2, r2=r2,
                scale=scale)


def layer_backward(x, dy, p, f, hq, hkv, d):
    """Gradient of L = sum(dy * y) given the forward intermediates f.
    Returns dx, dw_qkv, dw_o, dw_1, dw_2, dg1, db1, dg2, db2."""
    x, dy = _f64(x), _f64(dy)
    S, H = x.shape
    # y = h + g W2
    dw_2 = f["g"].T @ dy
    da = (dy @ _f64(p["w_2"]).T) * gelu_grad(f["a"])
    # a = z W1
    dw_1 = f["z"].T @ da
    dz = da @ _f64(p["w_1"]).T
    # z = LN2(h); h also feeds y directly
    dh_ln, dg2, db2 = layer_norm_bwd(f["h"], p["g2"], f["m2"], f["r2"], dz)
    dh = dy + dh_ln
    # h = x + O Wo
    dw_o = f["o"].T @ dh
    do4 = (dh @ _f64(p["w_o"]).T).reshape(1, S, hq, d)
    dq, dk, dv = attention_bwd(f["q"], f["k"], f["v"], do4, f["scale"], f["o4"], f["lse"])
    dqkv = np.concatenate([dq.reshape(S, -1), dk.reshape(S, -1), dv.reshape(S, -1)], axis=1)
    # q, k, v = u W_qkv
    dw_qkv = f["u"].T @ dqkv
    du = dqkv @ _f64(p["w_qkv"]).T
    # u = LN1(x); x also feeds h directly
    dx_ln, dg1, db1 = layer_norm_bwd(x, p["g1"], f["m1"], f["r1"], du)
    return dict(dx=dh + dx_ln, dw_qkv=dw_qkv, dw_o=dw_o, dw_1=dw_1, dw_2=dw_2, dg1=dg1, db1=db1, dg2=dg2, db2=db2)


def layer_forward_rows(x, p, rows, hq, hkv, d, scale=None):
    """y at the given rows only, from the prefix x [R, H] (R > max(rows)):
    the causal layer's row r depends on rows 0..r alone, so this needs the
    K/V projections of the prefix and, per sampled row, its own query, one
    softmax per head over its visible keys, and the row-wise rest of the
    block.  Returns [len(rows), H]."""
    x = _f64(x)
    H = x.shape[1]
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    G = hq // hkv
    w = _f64(p["w_qkv"])
    u, _, _ = layer_norm(x, p["g1"], p["b1"])
    k = u @ w[:, hq * d:(hq + hkv) * d]
    v = u @ w[:, (hq + hkv) * d:]
    out = np.empty((len(rows), H))
    for i, r in enumerate(rows):
        q = u[r] @ w[:, :hq * d]
        o = np.empty(hq * d)
        for h in range(hq):
            kv = slice((h // G) * d, (h // G + 1) * d)
            s = (k[:r + 1, kv] @ q[h * d:(h + 1) * d]) * scale
            e = np.exp(s - s.max())
            o[h * d:(h + 1) * d] = (e / e.sum()) @ v[:r + 1, kv]
        hr = x[r] + o @ _f64(p["w_o"])
        z, _, _ = layer_norm(hr[None, :], p["g2"], p["b2"])
        out[i] = hr + gelu(z[0] @ _f64(p["w_1"])) @ _f64(p["w_2"])
    return out


def layer(x, dy, p, hq, hkv, d, scale=None):
    """Forward and backward of the unchunked layer as one dict."""
    f = layer_forward(x, p, hq, hkv, d, scale)
    out = layer_backward(x, dy, p, f, hq, hkv, d)
    out["y"] = f["y"]
    return out


def chunked_layer(x, dy, p, hq, hkv, d, offsets, scale=None):
    """The subsequence walk: forward chunk by chunk with a growing K/V cache,
    then the backward in reverse order with dK/dV and the weight gradients
    accumulated across chunks.  Returns the same dict as ``layer``."""
    x, dy = _f64(x), _f64(dy)
    S, H = x.shape
    c = np.asarray(offsets, dtype=np.int64)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    n = len(c) - 1
    y = np.zeros_like(x)
    kc = np.zeros((1, S, hkv, d))
    vc = np.zeros((1, S, hkv, d))
    saved = []
    for i in range(n):
        r = slice(c[i], c[i + 1])
        u, m1, r1 = layer_norm(x[r], p["g1"], p["b1"])
        q, k, v = _split_qkv(u @ _f64(p["w_qkv"]), hq, hkv, d)
        kc[:, r], vc[:, r] = k, v
        # rows [c_i, c_{i+1}) of the causal attention over keys [0, c_{i+1}):
        # the last chunk of a two-chunk split of the prefix
        pre = c[i + 1]
        qq = np.zeros((1, pre, hq, d))
        qq[:, c[i]:pre] = q
        offs = [0, c[i], pre] if c[i] > 0 else [0, pre]
        oo, ll = chunked_attention_fwd(qq, kc[:, :pre], vc[:, :pre], scale, offs)
        o4, lse = oo[:, c[i]:pre], ll[:, :, c[i]:pre]
        o = o4.reshape(pre - c[i], hq * d)
        h = x[r] + o @ _f64(p["w_o"])
        z, m2, r2 = layer_norm(h, p["g2"], p["b2"])
        a = z @ _f64(p["w_1"])
        y[r] = h + gelu(a) @ _f64(p["w_2"])
        saved.append(dict(u=u, q=q, o=o, o4=o4, lse=lse, h=h, z=z, a=a, m1=m1, r1=r1, m2=m2, r2=r2))
    dx = np.zeros_like(x)
    acc = {key: 0.0 for key in ("dw_qkv", "dw_o", "dw_1", "dw_2", "dg1", "db1", "dg2", "db2")}
    dk_acc = np.zeros((1, S, hkv, d))
    dv_acc = np.zeros((1, S, hkv, d))
    for i in reversed(range(n)):
        r = slice(c[i], c[i + 1])
        f = saved[i]
        dyi = dy[r]
        acc["dw_2"] = acc["dw_2"] + gelu(f["a"]).T @ dyi
        da = (dyi @ _f64(p["w_2"]).T) * gelu_grad(f["a"])
        acc["dw_1"] = acc["dw_1"] + f["z"].T @ da
        dz = da @ _f64(p["w_1"]).T
        dh_ln, dg2, db2 = layer_norm_bwd(f["h"], p["g2"], f["m2"], f["r2"], dz)
        acc["dg2"], acc["db2"] = acc["dg2"] + dg2, acc["db2"] + db2
        dh = dyi + dh_ln
        acc["dw_o"] = acc["dw_o"] + f["o"].T @ dh
        do4 = (dh @ _f64(p["w_o"]).T).reshape(1, -1, hq, d)
        pre = c[i + 1]
        qq = np.zeros((1, pre, hq, d))
        dd = np.zeros((1, pre, hq, d))
        oo = np.zeros((1, pre, hq, d))
        ll = np.zeros((1, hq, pre))
        qq[:, c[i]:pre], dd[:, c[i]:pre], oo[:, c[i]:pre], ll[:, :, c[i]:pre] = f["q"], do4, f["o4"], f["lse"]
        offs = [0, c[i], pre] if c[i] > 0 else [0, pre]
        dq, dk, dv = chunked_attention_bwd(qq, kc[:, :pre], vc[:, :pre], dd, scale, offs, oo, ll)
        dk_acc[:, :pre] += dk
        dv_acc[:, :pre] += dv
        # chunk i's K/V rows have received every later chunk's contribution
        dqkv = np.concatenate([dq[0, c[i]:pre].reshape(pre - c[i], -1),
                               dk_acc[0, r].reshape(pre - c[i], -1),
                               dv_acc[0, r].reshape(pre - c[i], -1)], axis=1)
        acc["dw_qkv"] = acc["dw_qkv"] + f["u"].T @ dqkv
        du = dqkv @ _f64(p["w_qkv"]).T
        dx_ln, dg1, db1 = layer_norm_bwd(x[r], p["g1"], f["m1"], f["r1"], du)
        acc["dg1"], acc["db1"] = acc["dg1"] + dg1, acc["db1"] + db1
        dx[r] = dh + dx_ln
    out = dict(acc)
    out["dx"], out["y"] = dx, y
    return out
