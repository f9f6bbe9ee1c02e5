"""Host-side offload policy of libsppo, no GPU needed.

* FLOPs-balanced partition (c_k = S sqrt(k/N)): structure, hand-computed
  offsets, and the property it exists for -- every chunk holds about the
  same number of visible (query, key) pairs of the causal triangle.
* Sequence-aware offload plan: rows_i = min(s_i, floor(bw * t_i / bytes_per_row)),
  aligned down when partial, 0 for the last chunk; hand-computed cases.
"""
import pytest

from paper_2503_10377_amd import sppo as L


def pairs(offsets):
    """Visible (query, key) pairs of each chunk of a causal sequence."""
    out = []
    for i in range(len(offsets) - 1):
        c, s = offsets[i], offsets[i + 1] - offsets[i]
        out.append(s * c + s * (s + 1) // 2)
    return out


def test_balanced_offsets_hand_values():
    # S = 1600, N = 4: c_k = 800 sqrt(k) -> 800, 1131.37, 1385.64, 1600
    assert L.sppo_balanced_offsets(1600, 4, 1) == [0, 800, 1131, 1386, 1600]
    # same with 64-row alignment: 768 (12.5 -> 12 or 13? 800/64 = 12.5 rounds to 13 -> 832)
    got = L.sppo_balanced_offsets(1600, 4, 64)
    assert got == [0, 832, 1152, 1408, 1600]
    assert L.sppo_balanced_offsets(777, 1, 1) == [0, 777]


@pytest.mark.parametrize("S,N,align", [(131072, 16, 128), (524288, 32, 128), (1048576, 64, 256), (32768, 8, 64)])
def test_balanced_offsets_balance_the_work(S, N, align):
    off = L.sppo_balanced_offsets(S, N, align)
    assert off[0] == 0 and off[-1] == S and len(off) == N + 1
    assert all(b - a >= align for a, b in zip(off, off[1:]))
    assert all(c % align == 0 for c in off[:-1])
    p = pairs(off)
    assert sum(p) == S * (S + 1) // 2
    # A chunk holds (c_{k+1}^2 - c_k^2 + s_k) / 2 pairs; the ideal
    # boundaries give S^2 / (2N) each.  Rounding moves a boundary c by at
    # most align/2, which changes a neighbour's pairs by at most c*align/2
    # <= S*align/2, i.e. by align*N/S of the ideal share -- two boundaries
    # per chunk, plus the small diagonal term s_k/2.
    mean = sum(p) / N
    bound = 2.0 * align * N / S + 1e-3
    assert max(abs(x - mean) / mean for x in p) <= bound
    # Equal-length chunks are far less balanced: the last has about 2N-1
    # times the first's pairs.
    eq = pairs([S // N * k for k in range(N + 1)])
    assert max(eq) / min(eq) > 2 * N - 2
    # Long chunks first (up to one alignment step of rounding).
    lens = [b - a for a, b in zip(off, off[1:])]
    assert all(n1 <= n0 + align for n0, n1 in zip(lens, lens[1:]))
    assert lens[0] > 2 * lens[-1]


def test_balanced_offsets_degenerate_and_errors():
    assert L.sppo_balanced_offsets(10, 10, 1) == list(range(11))  # every chunk one row
    assert L.sppo_balanced_offsets(8, 2, 4) == [0, 4, 8]          # sqrt(1/2)*8 = 5.66 -> 4 (alignment)
    for args in [(10, 11, 1), (100, 4, 32), (0, 1, 1), (10, 0, 1), (10, 2, 0)]:
        with pytest.raises(L.SppoError):
            L.sppo_balanced_offsets(*args)


def test_offload_plan_hand_values():
    off = [0, 1000, 2000, 3000]
    # 1 GB/s = 1e6 bytes per ms; 1000 bytes per row -> 1000 rows per ms
    assert L.sppo_plan_offload_rows(off, 1000.0, 1.0, [0.5, 2.0, 9.0], 1) == [500, 1000, 0]
    assert L.sppo_plan_offload_rows(off, 1000.0, 1.0, [0.5, 2.0, 9.0], 128) == [384, 1000, 0]
    assert L.sppo_plan_offload_rows(off, 1000.0, 1.0, [0.0, 0.9999, 1.0], 1) == [0, 999, 0]
    # exactly the chunk: not aligned down
    assert L.sppo_plan_offload_rows([0, 1000, 1100], 1000.0, 1.0, [1.0, 5.0], 128) == [1000, 0]
    assert L.sppo_plan_offload_rows([0, 5], 10.0, 1.0, [3.0], 1) == [0]  # single chunk: nothing to overlap


def test_offload_plan_bounds_copy_time():
    """alpha_i * A_i never needs more than t_i at the given rate."""
    off = L.sppo_balanced_offsets(131072, 16, 128)
    bpr = 2 * 32 * 128 * 2 + 4 * 32 + 2 * 32 * 128 * 2
    t = [9.8] * 16
    rows = L.sppo_plan_offload_rows(off, bpr, 55.0, t, 128)
    for i, r in enumerate(rows[:-1]):
        s = off[i + 1] - off[i]
        assert 0 <= r <= s
        assert r * bpr / (55.0 * 1e6) <= t[i] + 1e-9
        if r < s:  # limited by the link: within one alignment step of the budget
            assert (r + 128) * bpr / (55.0 * 1e6) > t[i]
    assert rows[-1] == 0


def test_offload_plan_errors():
    with pytest.raises(L.SppoError):
        L.sppo_plan_offload_rows([0, 10], 0.0, 1.0, [1.0], 1)
    with pytest.raises(L.SppoError):
        L.sppo_plan_offload_rows([0, 10], 10.0, -1.0, [1.0], 1)
    with pytest.raises(L.SppoError):
        L.sppo_plan_offload_rows([0, 10, 10], 10.0, 1.0, [1.0, 1.0], 1)  # empty chunk
    with pytest.raises(L.SppoError):
        L.sppo_plan_offload_rows([0, 10], 10.0, 1.0, [float("nan")], 1)
