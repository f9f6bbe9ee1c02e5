"""Pins of the fp64 oracle against things other than itself (CPU only).

* forward: brute-force pure-Python loops (math.exp, explicit sums)
* gradients: central finite differences of L = sum(dO * O)
* closed forms: S=1, Q=0 (prefix mean of V, LSE=ln(r+1), dK=0, dV reverse sums)
* invariants: sum_j dK_j = 0, sum_j dV_j = sum_r dO_r, sum q.dQ = sum k.dK,
  sum_j dS_rj = 0, max_j s_rj <= LSE_r <= max_j s_rj + ln(r+1)
* the subsequence decomposition (Sec. 5.1) equals the unchunked result
* GQA equals MHA on K/V repeated per group
* hand-derived worked examples (tests/golden/worked_examples.json)
* source mutations planted in the oracle (wrong mask, dropped term, wrong
  index, wrong log base, missing scale) each fail at least one pin.
"""
import json
import math
import os
import types

import numpy as np
import pytest

import oracle
from oracle import causal_attention as oracle_mod

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")


def rand_inputs(seed, B, S, Hq, Hkv, D, scale_q=1.0):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, S, Hq, D)) * scale_q
    k = rng.standard_normal((B, S, Hkv, D))
    v = rng.standard_normal((B, S, Hkv, D))
    do = rng.standard_normal((B, S, Hq, D))
    return q, k, v, do


# ---------------------------------------------------------------- brute force
def brute_fwd(q, k, v, scale):
    """Causal attention with explicit Python loops (no NumPy arithmetic)."""
    B, S, Hq, D = q.shape
    Hkv = k.shape[2]
    G = Hq // Hkv
    o = np.zeros((B, S, Hq, D))
    lse = np.zeros((B, Hq, S))
    for b in range(B):
        for h in range(Hq):
            g = h // G
            for r in range(S):
                logits = []
                for j in range(r + 1):
                    acc = 0.0
                    for d in range(D):
                        acc += float(q[b, r, h, d]) * float(k[b, j, g, d])
                    logits.append(scale * acc)
                m = max(logits)
                z = sum(math.exp(x - m) for x in logits)
                lse[b, h, r] = m + math.log(z)
                for d in range(D):
                    o[b, r, h, d] = sum(math.exp(logits[j] - m) / z * float(v[b, j, g, d])
                                        for j in range(r + 1))
    return o, lse


def loss(mod, q, k, v, do, scale):
    o, _ = mod.attention_fwd(q, k, v, scale)
    return float((o * do).sum())


def fd_grads(mod, q, k, v, do, scale, h=1e-6):
    """Central finite differences of L = sum(dO * O) w.r.t. q, k, v."""
    out = []
    for which in range(3):
        args = [q.copy(), k.copy(), v.copy()]
        x = args[which]
        g = np.zeros_like(x)
        it = np.nditer(x, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            x0 = x[idx]
            x[idx] = x0 + h
            lp = loss(mod, *args, do, scale)
            x[idx] = x0 - h
            lm = loss(mod, *args, do, scale)
            x[idx] = x0
            g[idx] = (lp - lm) / (2 * h)
        out.append(g)
    return out


SHAPES = [  # B, S, Hq, Hkv, D
    (1, 1, 1, 1, 2),
    (1, 5, 1, 1, 3),
    (2, 7, 2, 1, 2),
    (1, 6, 4, 2, 3),
]


@pytest.mark.parametrize("shape", SHAPES)
def test_forward_matches_brute_force(shape):
    B, S, Hq, Hkv, D = shape
    q, k, v, _ = rand_inputs(1, B, S, Hq, Hkv, D, scale_q=1.5)
    scale = 1 / math.sqrt(D)
    o, lse = oracle.attention_fwd(q, k, v, scale)
    ob, lb = brute_fwd(q, k, v, scale)
    np.testing.assert_allclose(o, ob, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lb, rtol=0, atol=1e-12)


@pytest.mark.parametrize("shape", SHAPES[1:])
def test_gradients_match_finite_differences(shape):
    B, S, Hq, Hkv, D = shape
    q, k, v, do = rand_inputs(2, B, S, Hq, Hkv, D)
    scale = 0.7
    dq, dk, dv = oracle.attention_bwd(q, k, v, do, scale)
    fq, fk, fv = fd_grads(oracle_mod, q, k, v, do, scale)
    for a, f in ((dq, fq), (dk, fk), (dv, fv)):
        np.testing.assert_allclose(a, f, rtol=0, atol=2e-7 * max(1.0, np.abs(f).max()))


def test_single_token_closed_form():
    q, k, v, do = rand_inputs(3, 2, 1, 2, 2, 4)
    o, lse = oracle.attention_fwd(q, k, v, 0.5)
    np.testing.assert_allclose(o, v, atol=1e-15)
    np.testing.assert_allclose(lse, 0.5 * np.einsum("bshd,bshd->bhs", q, k), atol=1e-14)
    dq, dk, dv = oracle.attention_bwd(q, k, v, do, 0.5)
    # P = 1 for the only key: dS = dP - Delta = 0, so dQ = dK = 0 and dV = dO.
    assert np.abs(dq).max() < 1e-14 and np.abs(dk).max() < 1e-14
    np.testing.assert_allclose(dv, do, atol=1e-15)


def test_zero_query_closed_form():
    B, S, Hq, Hkv, D = 1, 9, 2, 1, 3
    _, k, v, do = rand_inputs(4, B, S, Hq, Hkv, D)
    q = np.zeros((B, S, Hq, D))
    r = np.arange(1, S + 1)
    o, lse = oracle.attention_fwd(q, k, v, 0.3)
    prefix_mean = np.cumsum(v, axis=1) / r[None, :, None, None]
    np.testing.assert_allclose(o, np.repeat(prefix_mean, Hq, axis=2), atol=1e-14)
    np.testing.assert_allclose(lse, np.broadcast_to(np.log(r), (B, Hq, S)), atol=1e-14)
    dq, dk, dv = oracle.attention_bwd(q, k, v, do, 0.3)
    assert np.abs(dk).max() < 1e-14
    # dV_j = sum_{h} sum_{r>=j} dO_r / (r+1): a reverse cumulative sum.
    w = do.sum(axis=2, keepdims=True) / r[None, :, None, None]
    expect = np.flip(np.cumsum(np.flip(w, axis=1), axis=1), axis=1)
    np.testing.assert_allclose(dv, expect, atol=1e-13)


def test_equal_keys_give_prefix_mean():
    B, S, Hq, Hkv, D = 1, 6, 1, 1, 4
    q, _, v, _ = rand_inputs(5, B, S, Hq, Hkv, D)
    k = np.broadcast_to(np.array([0.3, -1.0, 2.0, 0.5]), (B, S, Hkv, D)).copy()
    o, _ = oracle.attention_fwd(q, k, v, 1.0)
    prefix_mean = np.cumsum(v, axis=1) / np.arange(1, S + 1)[None, :, None, None]
    np.testing.assert_allclose(o, prefix_mean, atol=1e-13)


def test_one_hot_values_give_probabilities():
    B, S, D = 1, 5, 5
    q, k, _, _ = rand_inputs(6, B, S, 1, 1, D)
    v = np.eye(S).reshape(B, S, 1, D)
    o, lse = oracle.attention_fwd(q, k, v, 0.8)
    s = 0.8 * q[0, :, 0] @ k[0, :, 0].T
    p = np.where(np.tril(np.ones((S, S))) > 0, np.exp(s - lse[0, 0][:, None]), 0.0)
    np.testing.assert_allclose(o[0, :, 0], p, atol=1e-14)
    np.testing.assert_allclose(o.sum(axis=-1), 1.0, atol=1e-14)


@pytest.mark.parametrize("shape", [(1, 40, 2, 2, 8), (2, 33, 4, 1, 5), (1, 64, 8, 2, 16)])
def test_gradient_invariants(shape):
    B, S, Hq, Hkv, D = shape
    q, k, v, do = rand_inputs(7, B, S, Hq, Hkv, D, scale_q=2.0)
    scale = 1 / math.sqrt(D)
    o, lse = oracle.attention_fwd(q, k, v, scale)
    dq, dk, dv = oracle.attention_bwd(q, k, v, do, scale, o, lse)
    G = Hq // Hkv
    # key-shift invariance: adding c to every key leaves softmax unchanged.
    assert np.abs(dk.sum(axis=1)).max() < 1e-12 * max(1, np.abs(dk).max()) * S
    # value-shift invariance: adding c to every value adds c to every output.
    do_grouped = do.reshape(B, S, Hkv, G, D).sum(axis=3)
    np.testing.assert_allclose(dv.sum(axis=1), do_grouped.sum(axis=1), atol=1e-11)
    # q <-> k rescaling invariance: scores depend on q.k only.
    qdq = (q * dq).reshape(B, S, Hkv, G, D).sum(axis=(1, 3, 4))
    kdk = (k * dk).sum(axis=(1, 3))
    np.testing.assert_allclose(qdq, kdk, atol=1e-11)
    # LSE bounds.
    for b in range(B):
        for h in range(Hq):
            s = scale * q[b, :, h] @ k[b, :, h // G].T
            s = np.where(np.tril(np.ones((S, S))) > 0, s, -np.inf)
            mx = s.max(axis=1)
            assert np.all(lse[b, h] >= mx - 1e-12)
            assert np.all(lse[b, h] <= mx + np.log(np.arange(1, S + 1)) + 1e-12)


def test_ds_rows_sum_to_zero():
    B, S, Hq, Hkv, D = 1, 12, 1, 1, 4
    q, k, v, do = rand_inputs(8, B, S, Hq, Hkv, D)
    o, lse = oracle.attention_fwd(q, k, v, 0.5)
    s = 0.5 * q[0, :, 0] @ k[0, :, 0].T
    p = np.where(np.tril(np.ones((S, S))) > 0, np.exp(s - lse[0, 0][:, None]), 0.0)
    delta = (do[0, :, 0] * o[0, :, 0]).sum(-1)
    ds = p * (do[0, :, 0] @ v[0, :, 0].T - delta[:, None])
    np.testing.assert_allclose(ds.sum(axis=1), 0.0, atol=1e-13)


@pytest.mark.parametrize("offsets", [[0, 48], [0, 24, 48], [0, 16, 32, 48],
                                     [0, 1, 2, 3, 20, 30, 47, 48], [0, 5, 6, 30, 48]])
def test_chunked_equals_unchunked(offsets):
    B, S, Hq, Hkv, D = 2, 48, 4, 2, 8
    q, k, v, do = rand_inputs(9, B, S, Hq, Hkv, D, scale_q=1.5)
    scale = 1 / math.sqrt(D)
    ref = oracle.attention(q, k, v, do, scale, row_block=7)
    o, lse = oracle.chunked_attention_fwd(q, k, v, scale, offsets)
    np.testing.assert_allclose(o, ref["o"], atol=1e-12)
    np.testing.assert_allclose(lse, ref["lse"], atol=1e-12)
    dq, dk, dv = oracle.chunked_attention_bwd(q, k, v, do, scale, offsets, o, lse)
    for a, n in ((dq, "dq"), (dk, "dk"), (dv, "dv")):
        np.testing.assert_allclose(a, ref[n], atol=1e-12)


def test_gqa_equals_mha_with_repeated_kv():
    B, S, Hq, Hkv, D = 1, 20, 8, 2, 6
    q, k, v, do = rand_inputs(10, B, S, Hq, Hkv, D)
    G = Hq // Hkv
    gqa = oracle.attention(q, k, v, do, 0.4)
    mha = oracle.attention(q, np.repeat(k, G, axis=2), np.repeat(v, G, axis=2), do, 0.4)
    for n in ("o", "lse", "dq"):
        np.testing.assert_allclose(gqa[n], mha[n], atol=1e-13)
    for n in ("dk", "dv"):
        summed = mha[n].reshape(B, S, Hkv, G, D).sum(axis=3)
        np.testing.assert_allclose(gqa[n], summed, atol=1e-13)


def test_row_subset_and_tail_keys_match_full():
    B, S, Hq, Hkv, D = 1, 70, 4, 2, 8
    q, k, v, do = rand_inputs(11, B, S, Hq, Hkv, D)
    ref = oracle.attention(q, k, v, do, 0.35)
    rows = np.array([0, 1, 17, 31, 32, 69])
    sub = oracle.rows_fwd_bwd(q[:, rows], do[:, rows], rows, k, v, 0.35)
    np.testing.assert_allclose(sub["o"], ref["o"][:, rows], atol=1e-13)
    np.testing.assert_allclose(sub["lse"], ref["lse"][:, :, rows], atol=1e-13)
    np.testing.assert_allclose(sub["dq"], ref["dq"][:, rows], atol=1e-13)
    t0 = 50
    dk, dv = oracle.tail_keys_bwd(q[:, t0:], do[:, t0:], k, v, 0.35, t0, row_block=6)
    np.testing.assert_allclose(dk, ref["dk"][:, t0:], atol=1e-13)
    np.testing.assert_allclose(dv, ref["dv"][:, t0:], atol=1e-13)


def test_early_keys_from_row_blocks_match_full():
    """keys_bwd_rows: the contributions of any partition of the rows
    [min(keys), S) add up to the full oracle's dK/dV at those keys (early
    keys included, GQA, repeated and unsorted keys), and rows before a key
    contribute exactly nothing to it."""
    B, S, Hq, Hkv, D = 2, 90, 4, 2, 8
    q, k, v, do = rand_inputs(12, B, S, Hq, Hkv, D)
    ref = oracle.attention(q, k, v, do, 0.3)
    keys = np.array([40, 3, 89, 17, 40, 64, 65])
    lo = int(keys.min())
    dk = np.zeros((B, len(keys), Hkv, D))
    dv = np.zeros_like(dk)
    for r0, r1 in ((lo, 20), (20, 21), (21, 64), (64, S)):
        a, b = oracle.keys_bwd_rows(q[:, r0:r1], do[:, r0:r1], r0, k, v, 0.3, keys, row_block=7)
        dk += a
        dv += b
    np.testing.assert_allclose(dk, ref["dk"][:, keys], atol=1e-13)
    np.testing.assert_allclose(dv, ref["dv"][:, keys], atol=1e-13)
    a, b = oracle.keys_bwd_rows(q[:, :lo], do[:, :lo], 0, k, v, 0.3, keys)
    assert not a.any() and not b.any()


def _golden_value(x):
    if isinstance(x, list):
        return [_golden_value(y) for y in x]
    if isinstance(x, str):
        coef, _, arg = x.partition("ln")
        c = {"": 1.0, "-": -1.0}.get(coef, None)
        c = float(coef) if c is None else c
        return c * math.log(float(arg))
    return float(x)


def test_hand_derived_worked_examples():
    with open(GOLDEN) as f:
        data = json.load(f)
    for ex in data["examples"]:
        arr = {n: np.array(_golden_value(ex[n])) for n in ex
               if n not in ("name", "derivation", "scale")}
        S, D = arr["q"].shape
        q = arr["q"].reshape(1, S, 1, D)
        k = arr["k"].reshape(1, S, 1, D)
        v = arr["v"].reshape(1, S, 1, D)
        o, lse = oracle.attention_fwd(q, k, v, ex["scale"])
        np.testing.assert_allclose(o[0, :, 0], arr["o"], atol=1e-13, err_msg=ex["name"])
        np.testing.assert_allclose(lse[0, 0], arr["lse"], atol=1e-13, err_msg=ex["name"])
        if "dq" in arr:
            do = arr["do"].reshape(1, S, 1, D)
            dq, dk, dv = oracle.attention_bwd(q, k, v, do, ex["scale"])
            for n, a in (("dq", dq), ("dk", dk), ("dv", dv)):
                np.testing.assert_allclose(a[0, :, 0], arr[n], atol=1e-13, err_msg=ex["name"])


def test_row_blocking_does_not_change_results():
    q, k, v, do = rand_inputs(12, 1, 37, 2, 1, 4)
    a = oracle.attention(q, k, v, do, 0.5, row_block=512)
    b = oracle.attention(q, k, v, do, 0.5, row_block=5)
    for n in a:
        np.testing.assert_allclose(a[n], b[n], atol=1e-13)


# ------------------------------------------------------------ planted mistakes
MUTATIONS = {
    "mask_admits_next_key": ("keys[None, :] > rows[:, None]", "keys[None, :] > rows[:, None] + 1"),
    "mask_excludes_self": ("keys[None, :] > rows[:, None]", "keys[None, :] >= rows[:, None]"),
    "dropped_delta_term": ("ds = p * (dp - delta[:, None])", "ds = p * dp"),
    "dq_missing_scale": ("dq[b, r0:r1, h, :] = scale * (ds @ kg[:r1])",
                         "dq[b, r0:r1, h, :] = (ds @ kg[:r1])"),
    "wrong_kv_head_index": ("kg, vg = k[b, :, h // G, :], v[b, :, h // G, :]",
                            "kg, vg = k[b, :, h % G, :], v[b, :, h % G, :]"),
    "log2_lse": ("np.log(np.exp(s - m)", "np.log2(np.exp(s - m)"),
    "dv_uses_dq_weights": ("dv[b, :r1, g, :] += p.T @ dob", "dv[b, :r1, g, :] += ds.T @ dob"),
}


def _mutant(src_old, src_new):
    with open(oracle_mod.__file__) as f:
        src = f.read()
    assert src_old in src, src_old
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src.replace(src_old, src_new), "oracle_mutant", "exec"), mod.__dict__)
    return mod


def _pins_pass(mod):
    """Run a compact version of the pins above against module ``mod``."""
    try:
        with np.errstate(all="ignore"):
            q, k, v, do = rand_inputs(13, 1, 5, 4, 2, 2, scale_q=1.5)
            o, lse = mod.attention_fwd(q, k, v, 0.6)
            ob, lb = brute_fwd(q, k, v, 0.6)
            if not (np.allclose(o, ob, atol=1e-12) and np.allclose(lse, lb, atol=1e-12)):
                return False
            dq, dk, dv = mod.attention_bwd(q, k, v, do, 0.6)
            fq, fk, fv = fd_grads(mod, q, k, v, do, 0.6)
            return all(np.allclose(a, f, atol=1e-6) for a, f in ((dq, fq), (dk, fk), (dv, fv)))
    except (ValueError, IndexError, FloatingPointError):
        return False


def test_pins_accept_the_oracle():
    assert _pins_pass(oracle_mod)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_reject_planted_mistakes(name):
    assert not _pins_pass(_mutant(*MUTATIONS[name])), name
