"""fp64 oracle: causal softmax attention, its analytic gradient, and the
subsequence (chunk) decomposition of both.

TEST INFRASTRUCTURE ONLY -- never imported by the product path.

What is computed (the paper never writes the attention formula out; this is
standard scaled dot-product causal attention, the operation whose activations
the paper's two-level activation management (Sec. 5.1) splits into a resident
K/V cache and offloaded per-subsequence tensors).  For batch b, query head h,
KV head g = h // (Hq // Hkv), global query row r and key j:

    s_rj   = scale * <Q[b,r,h], K[b,j,g]>                       visible iff j <= r
    LSE_r  = log sum_{j<=r} exp(s_rj)                           (natural log)
    P_rj   = exp(s_rj - LSE_r) for j <= r, else 0
    O_r    = sum_j P_rj V[b,j,g]

Backward for the loss L = sum(dO * O) with a given upstream gradient dO:

    Delta_r = <dO_r, O_r>
    dP_rj   = <dO_r, V_j>
    dS_rj   = P_rj (dP_rj - Delta_r)
    dQ_r    = scale * sum_j dS_rj K_j
    dK_j    = scale * sum_{h in group g} sum_{r>=j} dS_rj Q_r
    dV_j    =         sum_{h in group g} sum_{r>=j} P_rj dO_r

The chunked variant follows the paper's subsequence decomposition (Sec. 5.1:
a query of subsequence i attends to the K/V of subsequences 0..i, so only the
diagonal block carries the causal mask; Sec. 5.2: the backward of subsequences
runs in reverse order).  It exists to check that chunking is an exact rewrite.

Pins (tests/test_oracle_pins.py): brute-force Python loops on tiny inputs
(forward); central finite differences of L (gradients); closed forms at S=1
and Q=0; invariants sum_j dK_j = 0, sum_j dV_j = sum_r dO_r, sum q.dQ = sum
k.dK, sum_j dS_rj = 0; the LSE bounds; chunked == unchunked; GQA == MHA with
repeated K/V; a hand-derived worked example (tests/golden/).

Blocking over query rows (``row_block``) only bounds memory: every row's
formula is unchanged, and only the order of fp64 summation of the dK/dV
contributions differs.
"""
from __future__ import annotations

import numpy as np


def _group(hq: int, hkv: int) -> int:
    if hkv <= 0 or hq % hkv != 0:
        raise ValueError(f"n_q_heads={hq} must be a multiple of n_kv_heads={hkv}")
    return hq // hkv


def equal_offsets(seq_len: int, n_chunks: int) -> np.ndarray:
    """Chunk offsets c_0=0 < ... < c_N=S for N equal-length subsequences
    (the length-based partition of Sec. 3.2)."""
    if n_chunks <= 0 or seq_len % n_chunks != 0:
        raise ValueError("equal partition needs S % N == 0")
    return np.arange(n_chunks + 1, dtype=np.int64) * (seq_len // n_chunks)


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def _masked_scores(qb, kb, scale, rows, keys):
    """scale * qb @ kb.T with -inf where key index > query index."""
    s = scale * (qb @ kb.T)
    s[keys[None, :] > rows[:, None]] = -np.inf
    return s


def _row_lse(s):
    m = s.max(axis=1, keepdims=True)
    return m + np.log(np.exp(s - m).sum(axis=1, keepdims=True))


def attention_fwd(q, k, v, scale, row_block=512):
    """Unchunked causal attention forward. Returns (o [B,S,Hq,D], lse [B,Hq,S])."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, S, Hq, D = q.shape
    G = _group(Hq, k.shape[2])
    o = np.zeros_like(q)
    lse = np.empty((B, Hq, S))
    for b in range(B):
        for h in range(Hq):
            kg, vg = k[b, :, h // G, :], v[b, :, h // G, :]
            for r0 in range(0, S, row_block):
                r1 = min(S, r0 + row_block)
                rows, keys = np.arange(r0, r1), np.arange(r1)
                s = _masked_scores(q[b, r0:r1, h, :], kg[:r1], scale, rows, keys)
                l_ = _row_lse(s)
                p = np.exp(s - l_)
                o[b, r0:r1, h, :] = p @ vg[:r1]
                lse[b, h, r0:r1] = l_[:, 0]
    return o, lse


def attention_bwd(q, k, v, do, scale, o=None, lse=None, row_block=512):
    """Unchunked causal attention backward for L = sum(dO * O).

    Returns (dq, dk, dv).  ``o``/``lse`` default to this module's own forward;
    Delta is always formed from the fp64 O."""
    q, k, v, do = _f64(q), _f64(k), _f64(v), _f64(do)
    if o is None or lse is None:
        o, lse = attention_fwd(q, k, v, scale, row_block)
    B, S, Hq, D = q.shape
    G = _group(Hq, k.shape[2])
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for b in range(B):
        for h in range(Hq):
            g = h // G
            kg, vg = k[b, :, g, :], v[b, :, g, :]
            for r0 in range(0, S, row_block):
                r1 = min(S, r0 + row_block)
                rows, keys = np.arange(r0, r1), np.arange(r1)
                qb, dob, ob = q[b, r0:r1, h, :], do[b, r0:r1, h, :], o[b, r0:r1, h, :]
                s = _masked_scores(qb, kg[:r1], scale, rows, keys)
                p = np.exp(s - lse[b, h, r0:r1][:, None])
                delta = (dob * ob).sum(axis=1)
                dp = dob @ vg[:r1].T
                ds = p * (dp - delta[:, None])
                dq[b, r0:r1, h, :] = scale * (ds @ kg[:r1])
                dk[b, :r1, g, :] += scale * (ds.T @ qb)
                dv[b, :r1, g, :] += p.T @ dob
    return dq, dk, dv


def attention(q, k, v, do, scale, row_block=512):
    """Forward and backward of unchunked causal attention as a dict."""
    o, lse = attention_fwd(q, k, v, scale, row_block)
    dq, dk, dv = attention_bwd(q, k, v, do, scale, o, lse, row_block)
    return {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv}


def _check_offsets(offsets, S):
    c = np.asarray(offsets, dtype=np.int64)
    if c.ndim != 1 or len(c) < 2 or c[0] != 0 or c[-1] != S or np.any(np.diff(c) <= 0):
        raise ValueError("offsets must be strictly increasing from 0 to S")
    return c


def chunked_attention_fwd(q, k, v, scale, offsets):
    """Forward over subsequences (Sec. 5.1).

    For chunk i (rows [c_i, c_{i+1})) and every KV subsequence j <= i, form the
    partial result over block j alone -- fully visible for j < i, causally
    masked for j == i -- as (O_ij, LSE_ij); then merge them:
        LSE_i = log sum_j exp(LSE_ij),   O_i = sum_j exp(LSE_ij - LSE_i) O_ij.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, S, Hq, D = q.shape
    G = _group(Hq, k.shape[2])
    c = _check_offsets(offsets, S)
    o = np.zeros_like(q)
    lse = np.empty((B, Hq, S))
    for b in range(B):
        for h in range(Hq):
            kg, vg = k[b, :, h // G, :], v[b, :, h // G, :]
            for i in range(len(c) - 1):
                rows = np.arange(c[i], c[i + 1])
                qb = q[b, c[i]:c[i + 1], h, :]
                parts_o, parts_l = [], []
                for j in range(i + 1):
                    keys = np.arange(c[j], c[j + 1])
                    s = _masked_scores(qb, kg[c[j]:c[j + 1]], scale, rows, keys)
                    l_ = _row_lse(s)
                    parts_l.append(l_[:, 0])
                    parts_o.append(np.exp(s - l_) @ vg[c[j]:c[j + 1]])
                L = np.stack(parts_l)                    # [i+1, rows]
                m = L.max(axis=0)
                tot = m + np.log(np.exp(L - m).sum(axis=0))
                w = np.exp(L - tot)                      # merge weights
                o[b, c[i]:c[i + 1], h, :] = sum(w[j][:, None] * parts_o[j] for j in range(i + 1))
                lse[b, h, c[i]:c[i + 1]] = tot
    return o, lse


def chunked_attention_bwd(q, k, v, do, scale, offsets, o, lse):
    """Backward over subsequences in reverse order (Sec. 5.2), accumulating
    dK/dV of every KV subsequence j <= i into running sums while chunk i's dQ
    is formed from its own blocks.  ``o``/``lse`` are the forward results."""
    q, k, v, do, o, lse = map(_f64, (q, k, v, do, o, lse))
    B, S, Hq, D = q.shape
    G = _group(Hq, k.shape[2])
    c = _check_offsets(offsets, S)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for i in reversed(range(len(c) - 1)):
        rows = np.arange(c[i], c[i + 1])
        for b in range(B):
            for h in range(Hq):
                g = h // G
                qb, dob = q[b, c[i]:c[i + 1], h, :], do[b, c[i]:c[i + 1], h, :]
                delta = (dob * o[b, c[i]:c[i + 1], h, :]).sum(axis=1)
                lrow = lse[b, h, c[i]:c[i + 1]][:, None]
                for j in range(i + 1):
                    keys = np.arange(c[j], c[j + 1])
                    kj, vj = k[b, c[j]:c[j + 1], g, :], v[b, c[j]:c[j + 1], g, :]
                    p = np.exp(_masked_scores(qb, kj, scale, rows, keys) - lrow)
                    ds = p * (dob @ vj.T - delta[:, None])
                    dq[b, c[i]:c[i + 1], h, :] += scale * (ds @ kj)
                    dk[b, c[j]:c[j + 1], g, :] += scale * (ds.T @ qb)
                    dv[b, c[j]:c[j + 1], g, :] += p.T @ dob
    return dq, dk, dv


def rows_fwd_bwd(q_rows, do_rows, rows, k, v, scale):
    """O, LSE, Delta and dQ of selected global query rows only.

    q_rows, do_rows : [B, R, Hq, D] -- Q and dO at global positions ``rows``
    k, v            : [B, S, Hkv, D] -- the full K/V (any float dtype)
    Returns dict o [B,R,Hq,D], lse [B,Hq,R], delta [B,Hq,R], dq [B,R,Hq,D].
    Each row uses the same formulas as ``attention_fwd``/``attention_bwd``
    over keys 0..r; rows are independent, so a subset is exact."""
    q_rows, do_rows = _f64(q_rows), _f64(do_rows)
    rows = np.asarray(rows, dtype=np.int64)
    B, R, Hq, D = q_rows.shape
    Hkv = k.shape[2]
    G = _group(Hq, Hkv)
    out = {
        "o": np.zeros((B, R, Hq, D)), "dq": np.zeros((B, R, Hq, D)),
        "lse": np.zeros((B, Hq, R)), "delta": np.zeros((B, Hq, R)),
    }
    rmax = int(rows.max()) + 1
    for b in range(B):
        for g in range(Hkv):
            kg, vg = _f64(k[b, :rmax, g, :]), _f64(v[b, :rmax, g, :])
            keys = np.arange(rmax)
            for h in range(g * G, (g + 1) * G):
                qb, dob = q_rows[b, :, h, :], do_rows[b, :, h, :]
                s = _masked_scores(qb, kg, scale, rows, keys)
                l_ = _row_lse(s)
                p = np.exp(s - l_)
                ob = p @ vg
                delta = (dob * ob).sum(axis=1)
                ds = p * (dob @ vg.T - delta[:, None])
                out["o"][b, :, h, :] = ob
                out["lse"][b, h, :] = l_[:, 0]
                out["delta"][b, h, :] = delta
                out["dq"][b, :, h, :] = scale * (ds @ kg)
    return out


def tail_keys_bwd(q_tail, do_tail, k, v, scale, t0, row_block=256):
    """dK/dV of the keys j >= t0 of a length-S sequence.

    Key j only receives gradient from rows r >= j, so keys j >= t0 need just
    rows [t0, S): their full forward over all keys (for LSE and Delta) and
    their dS restricted to keys >= t0.  q_tail/do_tail are Q/dO rows [t0, S)
    as [B, S-t0, Hq, D]; k, v are full [B, S, Hkv, D] (any float dtype).
    Returns (dk_tail, dv_tail) as [B, S-t0, Hkv, D]."""
    q_tail, do_tail = _f64(q_tail), _f64(do_tail)
    B, T, Hq, D = q_tail.shape
    S = k.shape[1]
    Hkv = k.shape[2]
    G = _group(Hq, Hkv)
    if T != S - t0:
        raise ValueError("q_tail must hold rows [t0, S)")
    dk = np.zeros((B, T, Hkv, D))
    dv = np.zeros((B, T, Hkv, D))
    keys = np.arange(S)
    for b in range(B):
        for g in range(Hkv):
            kg, vg = _f64(k[b, :, g, :]), _f64(v[b, :, g, :])
            for h in range(g * G, (g + 1) * G):
                for a0 in range(0, T, row_block):
                    a1 = min(T, a0 + row_block)
                    rows = np.arange(t0 + a0, t0 + a1)
                    qb, dob = q_tail[b, a0:a1, h, :], do_tail[b, a0:a1, h, :]
                    s = _masked_scores(qb, kg, scale, rows, keys)
                    l_ = _row_lse(s)
                    p = np.exp(s - l_)
                    delta = (dob * (p @ vg)).sum(axis=1)
                    pt = p[:, t0:]
                    ds = pt * (dob @ vg[t0:].T - delta[:, None])
                    dk[b, :, g, :] += scale * (ds.T @ qb)
                    dv[b, :, g, :] += pt.T @ dob
    return dk, dv


def keys_bwd_rows(q_rows, do_rows, row0, k, v, scale, keys, row_block=256):
    """Contributions of the query rows [row0, row0 + R) to dK/dV at selected
    keys.

    dK_j and dV_j are sums over the rows r >= j (the backward formulas in the
    module docstring), and each row's terms need only that row's own LSE and
    Delta, formed here from all of its keys 0..r exactly as in
    ``attention_fwd`` / ``attention_bwd``.  Rows are independent, so summing
    this function over a partition of the rows [min(keys), S) gives the
    exact dK/dV at ``keys``: the chunked backward walk (Sec. 5.2) adds the
    same terms, chunk by chunk in reverse order, for the early keys that
    accumulate over many backward calls.

    q_rows, do_rows : Q and dO rows [row0, row0 + R) as [B, R, Hq, D]
    k, v            : the full [B, S, Hkv, D] (any float dtype)
    keys            : global key indices (any order, may repeat)
    Returns (dk, dv) as [B, len(keys), Hkv, D]."""
    q_rows, do_rows = _f64(q_rows), _f64(do_rows)
    keys = np.asarray(keys, dtype=np.int64)
    B, R, Hq, D = q_rows.shape
    Hkv = k.shape[2]
    G = _group(Hq, Hkv)
    dk = np.zeros((B, len(keys), Hkv, D))
    dv = np.zeros((B, len(keys), Hkv, D))
    rmax = row0 + R
    for b in range(B):
        for g in range(Hkv):
            kg, vg = _f64(k[b, :rmax, g, :]), _f64(v[b, :rmax, g, :])
            k_sel, v_sel = kg[np.minimum(keys, rmax - 1)], vg[np.minimum(keys, rmax - 1)]
            for h in range(g * G, (g + 1) * G):
                for a0 in range(0, R, row_block):
                    a1 = min(R, a0 + row_block)
                    rows = np.arange(row0 + a0, row0 + a1)
                    r_end = row0 + a1
                    qb, dob = q_rows[b, a0:a1, h, :], do_rows[b, a0:a1, h, :]
                    s = _masked_scores(qb, kg[:r_end], scale, rows, np.arange(r_end))
                    l_ = _row_lse(s)
                    delta = (dob * (np.exp(s - l_) @ vg[:r_end])).sum(axis=1)
                    # the selected keys' columns: s_rj and P_rj, zero where j > r
                    s_sel = scale * (qb @ k_sel.T)
                    p_sel = np.where(keys[None, :] <= rows[:, None], np.exp(s_sel - l_), 0.0)
                    ds = p_sel * (dob @ v_sel.T - delta[:, None])
                    dk[b, :, g, :] += scale * (ds.T @ qb)
                    dv[b, :, g, :] += p_sel.T @ dob
    return dk, dv
