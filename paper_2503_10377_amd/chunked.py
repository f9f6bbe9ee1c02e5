"""The chunk loop over libsppo: forward 0..N-1 with per-chunk offload, then
the reverse backward walk with prefetch (Sec. 5.1-5.2 of SPPO).

Only C-ABI calls and torch allocations happen here; every arithmetic step of
the path runs in the library's kernels.  Device tensors:
    q, do      [B, S, Hq, D]    inputs (dtype of the problem)
    k, v       [B, S, Hkv, D]   the resident K/V cache
    dq         [B, S, Hq, D]    output
    dk, dv     [B, S, Hkv, D]   fp32 accumulators
    o, lse     full-length copies of O ([B, S, Hq, D]) and of the per-chunk
               LSE ([B, Hq, s_i] each), filled only when a walk is asked to
               export them (tests); the walk itself keeps O_i and LSE_i in
               its device arena.
For B = 1 every chunk of q, do and dq is a contiguous view of the full
tensor; for B > 1 the chunk-local tensors are separate contiguous buffers.

Device memory of the saved activations (ring.DeviceArena): O_i and LSE_i
are produced into a region of a preallocated device arena; Q_i is read from
the caller's q in the forward.  An offloaded chunk's region (and its rows of
the caller's q) are dead once its offload has landed, and later chunks reuse
that memory; its prefetch brings Q_i, O_i and LSE_i back into a free region
and its backward reads them there.  With a row-prefix offload
(sequence-aware offloading) the rows that stay on the device move to a keep
buffer (``sppo_chunk_bufs.keep``) and back.  A chunk that is not offloaded
keeps its region until its backward.  The arena's size is planned from the
walk's allocation order, so that the forward reuses a chunk's memory
``fwd_slots`` chunks later.

Offload policy (``offload_chunks``): by default every chunk except the last
is offloaded -- the last chunk's backward runs right after its forward, so
sending its activations away and back could only add time.  Prefetches run
``lookahead`` chunks ahead of the backward walk.  With ``qkvol_evict`` the
K/V cache rows of the offloaded chunks are given up once the forward walk is
over; their copies are queued on the host-to-device stream right before the
backward of the last chunk, whose dK/dV work consumes them chunk by chunk in
the order they arrive.

Host pacing: the host stays at most ``host_ahead`` chunk boundaries ahead of
the device (a HostPacer; 0 lets it run free).
"""
from __future__ import annotations

import torch

from . import sppo as L
from .pacing import HostPacer
from .ring import DeviceArena, KeepArena, plan_capacity, plane_layout, walk_schedule


class ChunkedAttention:
    def __init__(self, B, S, n_chunks, Hq, Hkv, D, dtype="bf16", offsets=None, scale=0.0,
                 offload="none", device="cuda", host_ahead=2, fwd_slots=4):
        self.ctx = L.sppo_create(B, S, n_chunks, Hq, Hkv, D, dtype=dtype, chunk_offsets=offsets,
                                 softmax_scale=scale, offload=offload)
        self.B, self.S, self.N, self.Hq, self.Hkv, self.D = B, S, n_chunks, Hq, Hkv, D
        self.offsets = L.sppo_get_offsets(self.ctx)
        self.torch_dtype = torch.bfloat16 if self.ctx.problem["dtype"] == L.SPPO_BF16 else torch.float32
        self.offload = L.OFFLOAD_MODES.get(offload, offload)
        self.device = device
        self.pacer = HostPacer(host_ahead)
        self.fwd_slots = fwd_slots
        self.arena = None
        self.keep = None
        self._layout = None

    def close(self):
        self.ctx.close()

    # ------------------------------------------------------------ buffers
    def chunk_len(self, i):
        return self.offsets[i + 1] - self.offsets[i]

    def chunk_view(self, full, i):
        """Chunk-local contiguous [B, s_i, H, D] buffer for a full tensor."""
        c0, c1 = self.offsets[i], self.offsets[i + 1]
        if self.B == 1:
            return full[:, c0:c1]
        return full[:, c0:c1].contiguous()

    def alloc_outputs(self, export=True):
        """dq, dk, dv; with ``export`` also the full-length o and per-chunk
        lse that a walk with export=True fills."""
        B, S, Hq, Hkv, D = self.B, self.S, self.Hq, self.Hkv, self.D
        dev, dt = self.device, self.torch_dtype
        if not export:
            return {
                "dq": torch.empty((B, S, Hq, D), dtype=dt, device=dev),
                "dk": torch.empty((B, S, Hkv, D), dtype=torch.float32, device=dev),
                "dv": torch.empty((B, S, Hkv, D), dtype=torch.float32, device=dev),
            }
        # Per-chunk LSE slots back to back, each starting on a 16-byte boundary.
        sizes = [B * Hq * self.chunk_len(i) for i in range(self.N)]
        lse_flat = torch.empty(sum((n + 3) // 4 * 4 for n in sizes), dtype=torch.float32, device=dev)
        lse, pos = [], 0
        for i, n in enumerate(sizes):
            lse.append(lse_flat[pos:pos + n].view(B, Hq, self.chunk_len(i)))
            pos += (n + 3) // 4 * 4
        return {
            "o": torch.empty((B, S, Hq, D), dtype=dt, device=dev),
            "dq": torch.empty((B, S, Hq, D), dtype=dt, device=dev),
            "lse": lse,
            "lse_flat": lse_flat,
            "dk": torch.empty((B, S, Hkv, D), dtype=torch.float32, device=dev),
            "dv": torch.empty((B, S, Hkv, D), dtype=torch.float32, device=dev),
        }

    def lse_full(self, out):
        """[B, Hq, S] view assembled from the per-chunk LSE buffers."""
        return torch.cat(out["lse"], dim=2)

    # ---------------------------------------------------------- the walk
    def set_offload_rows(self, rows):
        """Offloaded row prefix per chunk (sequence-aware offloading); the
        rest of each chunk stays resident."""
        for i, r in enumerate(rows):
            L.sppo_set_offload_rows(self.ctx, i, r)

    def offload_rows(self):
        return L.sppo_get_offload_rows(self.ctx)

    def offload_bytes_per_row(self):
        """Bytes of the offload set per token row (Q, O, LSE; plus K, V in
        the QKVOL modes), all batch entries."""
        elt = 2 if self.torch_dtype == torch.bfloat16 else 4
        b = 2 * self.Hq * self.D * elt + 4 * self.Hq
        if self.offload in (L.SPPO_OFFLOAD_QKVOL, L.SPPO_OFFLOAD_QKVOL_EVICT):
            b += 2 * self.Hkv * self.D * elt
        return self.B * b

    def default_offload_chunks(self):
        if self.offload == L.SPPO_OFFLOAD_NONE:
            return []
        return list(range(self.N - 1))

    def region_planes(self, i):
        """Byte sizes of chunk i's saved tensors in its arena region."""
        B, Hq, D, n = self.B, self.Hq, self.D, self.chunk_len(i)
        elt = 2 if self.torch_dtype == torch.bfloat16 else 4
        return {"q": B * n * Hq * D * elt, "o": B * n * Hq * D * elt, "lse": B * Hq * n * 4}

    def prepare(self, offload_chunks=None, lookahead=2):
        """Allocate the device arena and keep buffers for a walk with these
        settings (done again only when they change; a walk allocates
        nothing).  Returns the bytes they hold."""
        if offload_chunks is None:
            offload_chunks = self.default_offload_chunks()
        offl = tuple(sorted(set(offload_chunks)))
        rows = tuple(self.offload_rows())
        key = (offl, lookahead, rows)
        if self._layout != key:
            self._planes = [plane_layout(self.region_planes(i)) for i in range(self.N)]
            sizes = [size for _, size in self._planes]
            q = self.fwd_slots - 1  # a chunk's forward memory is reused fwd_slots chunks later
            cap, q = plan_capacity(walk_schedule(self.N, offl, lookahead), sizes, quarantine=q)
            self.arena = None
            self.keep = None
            self.arena = DeviceArena(cap, self.device, quarantine=q)
            self.keep = KeepArena([L.sppo_keep_bytes(self.ctx, i) if i in offl else 0 for i in range(self.N)],
                                  self.device)
            self._layout = key
        return self.arena.nbytes + self.keep.nbytes

    def _acquire(self, i, s):
        """Allocate chunk i's region; returns (offset, views of its planes)."""
        off = self.arena.acquire(self.ctx, s, self._planes[i][1], i)
        B, Hq, D, n = self.B, self.Hq, self.D, self.chunk_len(i)
        po, dt, a = self._planes[i][0], self.torch_dtype, self.arena
        return off, {"q": a.view(off + po["q"], (B, n, Hq, D), dt), "o": a.view(off + po["o"], (B, n, Hq, D), dt),
                     "lse": a.view(off + po["lse"], (B, Hq, n), torch.float32)}

    def step(self, inp, out, offload_chunks=None, lookahead=2, poison=False, stream=None, marks=None,
             export=None, finalize=None):
        """One forward + backward pass over all chunks.

        ``export`` (default: when ``out`` has "o") copies every O_i and LSE_i
        into out["o"] / out["lse"] after its forward, for checking.
        ``finalize`` (a dict with bf16/fp32 "dk" and "dv" [B, S, Hkv, D])
        receives each chunk's final dK/dV rows right after its backward.
        With ``marks`` (a list), timing events are recorded on the stream
        before each chunk's forward and backward and at the end, appended as
        (label, event).  ``poison`` (test hook) overwrites every device buffer
        an offload has made dead -- the chunk's arena region, its rows of the
        caller's q and, with K/V eviction, the evicted cache rows -- with NaN
        once the copy has landed."""
        if offload_chunks is None:
            offload_chunks = self.default_offload_chunks()
        if export is None:
            export = "o" in out
        offl = set(offload_chunks)
        self.prepare(sorted(offl), lookahead)
        arena, keep = self.arena, self.keep
        arena.reset()
        s = torch.cuda.current_stream() if stream is None else stream
        q, k, v, do = inp["q"], inp["k"], inp["v"], inp["do"]
        qc = [self.chunk_view(q, i) for i in range(self.N)]
        dc = [self.chunk_view(do, i) for i in range(self.N)]
        dqc = [self.chunk_view(out["dq"], i) for i in range(self.N)]
        rows = self.offload_rows()

        def mark(label):
            self.pacer.boundary(s)
            if marks is not None:
                e = torch.cuda.Event(enable_timing=True)
                e.record(s)
                marks.append((label, e))

        held = {}  # chunk -> (region, views) of chunks that stay on the device
        for i in range(self.N):
            mark(("fwd", i))
            slot, sv = self._acquire(i, s)
            L.sppo_attn_fwd_chunk(self.ctx, i, qc[i], k, v, sv["o"], sv["lse"], s)
            if export:
                c0, c1 = self.offsets[i], self.offsets[i + 1]
                with torch.cuda.stream(s):
                    out["o"][:, c0:c1].copy_(sv["o"])
                    out["lse"][i].copy_(sv["lse"])
            if i in offl:
                bufs = L.chunk_bufs(q=qc[i], o=sv["o"], lse=sv["lse"], k=k, v=v, keep=keep.ptr(i))
                L.sppo_offload_issue(self.ctx, i, bufs, s)
                arena.release(slot, after_offload=True)
                if poison:
                    L.sppo_offload_wait(self.ctx, i, s)
                    r = rows[i] if keep.ptr(i) is None else self.chunk_len(i)
                    with torch.cuda.stream(s):
                        qc[i][:, :r].fill_(float("nan"))
                        sv["o"].fill_(float("nan"))
                        sv["lse"].fill_(float("nan"))
            else:
                held[i] = (slot, sv)
        if self.offload == L.SPPO_OFFLOAD_QKVOL_EVICT:
            kv_chunks = sorted(offl, reverse=True)
            if poison:
                # The evicted K/V rows are dead once their copies have landed.
                for j in kv_chunks:
                    L.sppo_offload_wait(self.ctx, j, s)
                with torch.cuda.stream(s):
                    for j in kv_chunks:
                        c0 = self.offsets[j]
                        k[:, c0:c0 + rows[j]].fill_(float("nan"))
                        v[:, c0:c0 + rows[j]].fill_(float("nan"))
            for j in kv_chunks:
                L.sppo_prefetch_kv(self.ctx, j, k, v, s)
        pending = sorted(offl, reverse=True)
        back = {}  # chunk -> (region, views) of prefetched chunks
        nxt = 0
        for i in reversed(range(self.N)):
            while nxt < len(pending) and pending[nxt] >= i - lookahead:
                j = pending[nxt]
                slot, sv = self._acquire(j, s)
                L.sppo_prefetch(self.ctx, j, L.chunk_bufs(q=sv["q"], o=sv["o"], lse=sv["lse"], keep=keep.ptr(j)), s)
                back[j] = (slot, sv)
                nxt += 1
            mark(("bwd", i))
            slot, sv = back.pop(i) if i in offl else held.pop(i)
            qi = sv["q"] if i in offl else qc[i]
            L.sppo_attn_bwd_chunk(self.ctx, i, qi, k, v, sv["o"], sv["lse"], dc[i], dqc[i],
                                  out["dk"], out["dv"], s)
            arena.release(slot)
            if finalize is not None:
                L.sppo_attn_finalize_chunk(self.ctx, i, out["dk"], out["dv"], finalize["dk"], finalize["dv"], s)
        mark(("end", -1))
        if self.B > 1:
            with torch.cuda.stream(s):
                for i in range(self.N):
                    c0, c1 = self.offsets[i], self.offsets[i + 1]
                    out["dq"][:, c0:c1].copy_(dqc[i])

    def forward_only(self, inp, out, stream=None):
        """Forward over all chunks without offload; leaves the context ready
        for a new walk."""
        s = torch.cuda.current_stream() if stream is None else stream
        oc = [self.chunk_view(out["o"], i) for i in range(self.N)]
        for i in range(self.N):
            L.sppo_attn_fwd_chunk(self.ctx, i, self.chunk_view(inp["q"], i), inp["k"], inp["v"],
                                  oc[i], out["lse"][i], s)
        L.sppo_reset(self.ctx)
        if self.B > 1:
            for i in range(self.N):
                c0, c1 = self.offsets[i], self.offsets[i + 1]
                out["o"][:, c0:c1].copy_(oc[i])
