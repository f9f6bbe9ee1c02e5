"""The device staging arena's bookkeeping, on the CPU: the circular
allocator (placement, reuse order, the wait before reusing an offloaded
chunk's memory), the walk schedule it is planned from, and the planned
capacities: max(quarantine, lookahead) + 1 chunks for equal chunks with all but the last
offloaded, every chunk without offload, and a replay of every schedule at
its planned capacity that never needs a region that is still live."""
import pytest
import torch

from paper_2503_10377_amd import ring as R
from paper_2503_10377_amd import sppo as L


def test_circular_allocation_and_reuse(monkeypatch):
    waits = []
    monkeypatch.setattr(L, "sppo_offload_wait", lambda ctx, i, stream=None: waits.append(i))
    a = R.DeviceArena(3 * 256, "cpu", quarantine=1)
    o0 = a.acquire(None, None, 256, 0)
    o1 = a.acquire(None, None, 200, 1)
    assert (o0, o1) == (0, 256)
    a.release(o0, after_offload=True)
    o2 = a.acquire(None, None, 256, 2)   # the tail first, no wait
    assert o2 == 512 and waits == []
    o3 = a.acquire(None, None, 256, 3)   # wraps onto chunk 0's region: waits for its offload
    assert o3 == 0 and waits == [0]
    with pytest.raises(RuntimeError):
        a.acquire(None, None, 256, 4)    # everything live
    a.release(o1)                        # freed in stream order: no wait
    assert a.acquire(None, None, 256, 5) == 256 and waits == [0]
    v = a.view(o2, (4, 8), torch.float32)
    v.fill_(1.0)
    assert a.buf[o2:o2 + 128].view(torch.float32).sum() == 32


def test_quarantine_skips_fresh_offloads():
    for q, third in ((1, 0), (2, None)):
        a = R.CircularAllocator(2 * 256)
        x = a.alloc(256, 0, lambda r: True)
        a.release(x, after_offload=True)
        assert a.alloc(256, 1, lambda r: a.count - r.released_at >= q) == 256
        assert a.alloc(256, 2, lambda r: a.count - r.released_at >= q) == third


def test_walk_schedule_order():
    ev = R.walk_schedule(4, [0, 1, 2], lookahead=1)
    assert ev == [("alloc", 0), ("offload", 0), ("alloc", 1), ("offload", 1), ("alloc", 2), ("offload", 2),
                  ("alloc", 3), ("alloc", 2), ("free", 3), ("alloc", 1), ("free", 2), ("alloc", 0), ("free", 1),
                  ("free", 0)]


@pytest.mark.parametrize("q", [0, 1, 3])
@pytest.mark.parametrize("lookahead", [0, 2, 3])
def test_planned_capacities(q, lookahead):
    """Equal chunks, all but the last offloaded: the forward rotates over
    q + 1 chunks (a region is reused q + 1 chunks later, the last chunk
    included), the backward holds its chunk and `lookahead` prefetched ones.
    Without offload every chunk keeps its memory."""
    n, a = 16, 1024
    sizes = [a] * n
    assert R.plan_capacity(R.walk_schedule(n, range(n - 1), lookahead), sizes, q) == (max(q + 1, lookahead + 1) * a, q)
    assert R.plan_capacity(R.walk_schedule(n, [], lookahead), sizes, q)[0] == n * a


@pytest.mark.parametrize("N", [1, 2, 5, 16, 64])
@pytest.mark.parametrize("lookahead", [0, 1, 2, 8])
@pytest.mark.parametrize("which", ["none", "all_but_last", "all", "some"])
@pytest.mark.parametrize("sizes", ["equal", "balanced"])
def test_every_schedule_replays_at_its_capacity(N, lookahead, which, sizes):
    offl = {"none": set(), "all_but_last": set(range(N - 1)), "all": set(range(N)),
            "some": {i for i in range(N) if i % 3 == 1}}[which]
    sz = [4096] * N if sizes == "equal" else [4096 * (N - i) // N + 256 for i in range(N)]
    sch = R.walk_schedule(N, offl, lookahead)
    cap, q = R.plan_capacity(sch, sz, 3)
    assert R.replay(sch, sz, cap, q)
    total = sum(R._up(s) for s in sz)
    # circular first fit can fragment around chunks that stay resident
    assert cap <= (total if which != "some" else total + max(R._up(s) for s in sz))


# ---- property test: the circular allocator against an independent model ----
from hypothesis import given, settings, strategies as st


@settings(max_examples=300, deadline=None)
@given(cap_blocks=st.integers(1, 24), q=st.integers(0, 3),
       ops=st.lists(st.tuples(st.sampled_from(["alloc", "release"]), st.integers(1, 8 * R.ALIGN),
                              st.integers(0, 10 ** 6), st.booleans()), max_size=60))
def test_allocator_against_a_model(cap_blocks, q, ops):
    """Random allocations and releases.  A model of the byte ranges (live,
    released by an offload at allocation count t, or free) checks every
    answer: placements in bounds and aligned, never over a live range or an
    offloaded one inside its quarantine; every offloaded range a placement
    reuses is reported through ``take`` (the caller waits for its copy);
    a failed allocation means no aligned placement was possible; the bytes
    in use match the live ranges."""
    cap = cap_blocks * R.ALIGN
    a = R.CircularAllocator(cap)
    model = []  # [start, end, state, released_at]

    def usable(r, count):  # count: the allocations made before the one asking
        return r[2] == "free" or (r[2] == "offload" and count - r[3] >= q)

    for kind, nbytes, pick, offl in ops:
        if kind == "alloc":
            n = R._up(nbytes)
            before = a.count
            taken = []
            off = a.alloc(nbytes, 0, lambda reg: a.count - reg.released_at >= q, lambda reg: taken.append(reg.start))
            if off is None:
                for s in range(0, cap - n + 1, R.ALIGN):
                    assert any(m[0] < s + n and m[1] > s and not usable(m, before) for m in model), (s, n, model)
                assert a.count == before
                continue
            assert off % R.ALIGN == 0 and 0 <= off and off + n <= cap
            over = [m for m in model if m[0] < off + n and m[1] > off]
            assert all(usable(m, before) for m in over), (off, n, over)
            assert sorted(taken) == sorted(m[0] for m in over if m[2] == "offload")
            model = [m for m in model if m not in over] + [[off, off + n, "live", 0]]
        else:
            live = [m for m in model if m[2] == "live"]
            if not live:
                continue
            m = live[pick % len(live)]
            a.release(m[0], after_offload=offl)
            m[2], m[3] = ("offload" if offl else "free"), a.count
        assert a.in_use == sum(m[1] - m[0] for m in model if m[2] == "live")
        assert a.high_water >= a.in_use
