"""Device staging arena for the saved activations of a chunk walk.

Two-level activation management (Sec. 5.1) keeps only the K/V cache
resident; a chunk's other saved tensors leave the device after its forward
and must be back before its backward.  The device memory they occupied is
what the offload saves, so it must really be given back: the memory
recurrence of Sec. 5.2 (M_i = M_{i-1} + A_i - alpha_{i-1} A_{i-1}) assumes
an offloaded chunk's memory is released once its copy has landed.

The arena is one preallocated device buffer used as a circular allocator:
each chunk's saved tensors get one contiguous region (its planes inside it,
each on a 256-byte boundary), allocated when the chunk's forward produces
them or when its prefetch brings them back, and released
  * after the chunk's offload was issued: the next allocation that reuses
    any of its bytes first makes the compute stream wait for that offload's
    copies (``sppo_offload_wait``);
  * after the chunk's backward was enqueued: stream order alone protects it
    (a prefetch into it waits for everything enqueued before it).
Allocations walk around the buffer in order, so the forward walk reuses the
memory of the oldest offloaded chunks and the backward walk (prefetching a
few chunks ahead) that of the chunks whose backward is done; regions still
live are skipped.  Nothing is allocated or freed while a walk runs.

The capacity comes from replaying the walk's own allocation order
(``walk_schedule``) on the CPU: the smallest arena in which no allocation
needs a region that is still live, nor one released by an offload fewer
than ``quarantine`` allocations earlier (so a chunk's copy has the forward
of the next few chunks to land before its memory is written again).  With
equal chunks and everything but the last chunk offloaded this is
max(quarantine, lookahead) + 1 chunks; with no offload it is the sum of all
chunks.
"""
from __future__ import annotations

import torch

from . import sppo as L

ALIGN = 256


def _up(n: int) -> int:
    return (int(n) + ALIGN - 1) // ALIGN * ALIGN


class _Region:
    __slots__ = ("start", "end", "state", "chunk", "released_at")

    def __init__(self, start, end, chunk):
        self.start, self.end, self.chunk = start, end, chunk
        self.state = "live"  # "live", "offload" (reusable after its copy), "free"
        self.released_at = 0


class CircularAllocator:
    """Circular first-fit allocation over ``capacity`` bytes; pure
    bookkeeping (no device memory), shared by the arena and the planner.
    ``reuse(region)`` is asked whether a released region's bytes may be
    reused (False: treat it as live); ``take(region)`` is called for each
    released region whose bytes an allocation then does reuse."""

    def __init__(self, capacity: int):
        self.capacity = int(capacity)
        self.reset()

    def reset(self):
        self.regions = []  # allocation order
        self.head = 0
        self.count = 0
        self.in_use = 0
        self.high_water = 0

    def alloc(self, nbytes: int, chunk: int, reuse, take=None) -> int | None:
        n = _up(nbytes)
        if n > self.capacity:
            return None
        start, moved = self.head, 0
        while moved <= self.capacity + n:
            if start + n > self.capacity:
                moved += self.capacity - start
                start = 0
            end = start + n
            blockers = [r for r in self.regions if r.start < end and r.end > start]
            stuck = [r for r in blockers if r.state == "live"]
            if not stuck:  # ask about released regions only for a range that is otherwise free
                stuck = [r for r in blockers if r.state == "offload" and not reuse(r)]
            if stuck:
                nxt = max(r.end for r in stuck)
                moved += nxt - start
                start = nxt
                continue
            for r in blockers:
                if take is not None and r.state == "offload":
                    take(r)
                self.regions.remove(r)
            reg = _Region(start, end, chunk)
            self.regions.append(reg)
            self.head = end
            self.count += 1
            self.in_use += n
            self.high_water = max(self.high_water, self.in_use)
            return start
        return None

    def release(self, start: int, after_offload: bool):
        for r in self.regions:
            if r.start == start and r.state == "live":
                r.state = "offload" if after_offload else "free"
                r.released_at = self.count
                self.in_use -= r.end - r.start
                return
        raise KeyError(f"no live region at offset {start}")


def walk_schedule(n_chunks, offload_chunks, lookahead):
    """The allocation order of a chunk walk: ("alloc", i) when chunk i's
    forward starts, ("offload", i) when its offload is issued (its region is
    released), ("alloc", i) again when its prefetch is issued (the backward
    walks N-1..0 with prefetches ``lookahead`` chunks ahead), ("free", i)
    after its backward.  Chunks that are not offloaded keep their forward
    region until their backward."""
    offl = set(offload_chunks)
    ev = []
    for i in range(n_chunks):
        ev.append(("alloc", i))
        if i in offl:
            ev.append(("offload", i))
    pending, nxt = sorted(offl, reverse=True), 0
    for i in reversed(range(n_chunks)):
        while nxt < len(pending) and pending[nxt] >= i - lookahead:
            ev.append(("alloc", pending[nxt]))
            nxt += 1
        ev.append(("free", i))
    return ev


def replay(schedule, sizes, capacity, quarantine) -> bool:
    """Whether the schedule fits ``capacity`` bytes without reusing a live
    region or one released by an offload less than ``quarantine``
    allocations ago."""
    a = CircularAllocator(capacity)
    where = {}
    for kind, i in schedule:
        if kind == "alloc":
            off = a.alloc(sizes[i], i, lambda r: a.count - r.released_at >= quarantine)
            if off is None:
                return False
            where[i] = off
        else:
            a.release(where[i], after_offload=(kind == "offload"))
    return True


def _smallest_capacity(schedule, sizes, quarantine) -> int:
    """Smallest capacity (256-byte steps, by bisection from the largest
    region up) for which the schedule replays."""
    lo = max(_up(s) for s in sizes)
    if replay(schedule, sizes, lo, quarantine):
        return lo
    hi = sum(_up(s) for s in sizes)
    while not replay(schedule, sizes, hi, quarantine):
        hi += lo
    while hi - lo > ALIGN:
        mid = (lo + hi) // 2 // ALIGN * ALIGN
        if replay(schedule, sizes, mid, quarantine):
            hi = mid
        else:
            lo = mid
    return hi


def plan_capacity(schedule, sizes, quarantine) -> tuple:
    """(capacity, quarantine) for the arena: the smallest capacity at the
    given quarantine, unless that exceeds keeping every chunk resident (a
    short walk, where waiting for the offloads costs nothing), in which case
    the quarantine is lowered until it does not."""
    total = sum(_up(s) for s in sizes)
    for q in range(quarantine, -1, -1):
        cap = _smallest_capacity(schedule, sizes, q)
        if cap <= total or q == 0:
            return cap, q
    raise AssertionError("unreachable")


class DeviceArena:
    """The device buffer behind a CircularAllocator.  It takes the planner's
    decisions exactly (the same quarantine), so a walk that follows the
    planned schedule never runs out of room; reusing a region released by
    an offload first makes the stream wait for that offload."""

    def __init__(self, capacity: int, device, quarantine: int):
        self.quarantine = quarantine
        self.alloc_ = CircularAllocator(capacity)
        self.buf = torch.empty(max(_up(capacity), ALIGN), dtype=torch.uint8, device=device)

    @property
    def nbytes(self) -> int:
        return self.buf.numel()

    @property
    def high_water(self) -> int:
        return self.alloc_.high_water

    def reset(self):
        """Forget every region (between walks, once their work is ordered
        before whatever the next walk enqueues)."""
        self.alloc_.reset()

    def acquire(self, ctx, stream, nbytes, chunk) -> int:
        a = self.alloc_
        waited = set()

        def take(r):
            if r.chunk not in waited:
                L.sppo_offload_wait(ctx, r.chunk, stream)
                waited.add(r.chunk)

        off = a.alloc(nbytes, chunk, lambda r: a.count - r.released_at >= self.quarantine, take)
        if off is None:
            raise RuntimeError(f"device arena of {self.nbytes} bytes is too small for chunk {chunk}")
        return off

    def release(self, off: int, after_offload: bool = False):
        self.alloc_.release(off, after_offload)

    def view(self, off: int, shape, dtype) -> torch.Tensor:
        n = 1
        for d in shape:
            n *= int(d)
        nbytes = n * torch.empty((), dtype=dtype).element_size()
        return self.buf[off:off + nbytes].view(dtype).view(*shape)


def plane_layout(planes: dict) -> tuple:
    """Offsets of named planes (bytes) inside one region, and its size."""
    offsets, pos = {}, 0
    for name, nbytes in planes.items():
        offsets[name] = pos
        pos += _up(nbytes)
    return offsets, max(pos, ALIGN)


class KeepArena:
    """One device buffer holding the keep regions of the chunks whose offload
    moves only a row prefix (``sppo_keep_bytes``: the rows that stay on the
    device while the chunk's region is reused)."""

    def __init__(self, sizes: list, device):
        self.offsets, pos = [], 0
        for n in sizes:
            self.offsets.append(pos if n else None)
            pos += _up(int(n))
        self.buf = torch.empty(pos, dtype=torch.uint8, device=device) if pos else None

    @property
    def nbytes(self) -> int:
        return 0 if self.buf is None else self.buf.numel()

    def ptr(self, i: int):
        if self.buf is None or self.offsets[i] is None:
            return None
        return self.buf.data_ptr() + self.offsets[i]
