"""Negative controls for the parity gates (CPU only): results corrupted the
ways a broken kernel would corrupt them must fail the gates, and the exact
result rounded to bf16 must pass.  Corruptions come from the oracle (planted
mistakes or post-hoc edits of its output), never from altered GPU code."""
import math
import types

import numpy as np
import pytest

import oracle
from oracle import causal_attention as oracle_mod
from parity import GateError, check_all

S, H, D, N = 4096, 1, 64, 8


def bf16_round(x):
    """Round float64 values to bf16 (nearest-even) and back, for a realistic
    'correct but bf16' result."""
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


@pytest.fixture(scope="module")
def case():
    rng = np.random.default_rng(0)
    q, k, v, do = (bf16_round(rng.standard_normal((1, S, H, D))) for _ in range(4))
    scale = 1 / math.sqrt(D)
    ref = oracle.attention(q, k, v, do, scale)
    return q, k, v, do, scale, ref, list(oracle.equal_offsets(S, N))


def rounded(ref):
    out = {n: bf16_round(ref[n]) for n in ("o", "dq")}
    out.update({n: ref[n].astype(np.float32).astype(np.float64) for n in ("dk", "dv", "lse")})
    return out


def test_bf16_rounded_exact_result_passes(case):
    *_, ref, off = case
    check_all(rounded(ref), ref, "bf16", off)


def test_zeroed_last_chunk_fails(case):
    *_, ref, off = case
    bad = rounded(ref)
    bad["o"][:, off[-2]:] = 0.0
    with pytest.raises(GateError):
        check_all(bad, ref, "bf16", off)


def test_dropped_first_block_of_last_chunk_fails(case):
    q, k, v, do, scale, ref, off = case
    c = off[1]
    rows = np.arange(off[-2], S)
    # The last chunk attending to keys [c_1, r] only: block 0 dropped.
    sub = oracle.rows_fwd_bwd(q[:, rows], do[:, rows], rows - c, k[:, c:], v[:, c:], scale)
    bad = rounded(ref)
    bad["o"][:, rows] = bf16_round(sub["o"])
    bad["lse"][:, :, rows] = sub["lse"]
    with pytest.raises(GateError):
        check_all(bad, ref, "bf16", off)


@pytest.mark.parametrize("mutation", [
    ("keys[None, :] > rows[:, None]", "keys[None, :] > rows[:, None] + 1"),   # admits key r+1
    ("keys[None, :] > rows[:, None]", "keys[None, :] > rows[:, None] - 1"),   # off by one the other way
])
def test_diagonal_mask_off_by_one_fails(case, mutation):
    q, k, v, do, scale, ref, off = case
    with open(oracle_mod.__file__) as f:
        src = f.read()
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src.replace(*mutation), "oracle_mutant", "exec"), mod.__dict__)
    with np.errstate(all="ignore"):
        bad = mod.attention(q, k, v, do, scale)
    with pytest.raises(GateError):
        check_all(rounded(bad), ref, "bf16", off)


def test_dropped_delta_fails(case):
    *_, ref, off = case
    bad = rounded(ref)
    bad["dq"] = bad["dq"] * 0.9
    with pytest.raises(GateError):
        check_all(bad, ref, "bf16", off)
