"""The chunk loop over libsppo: forward 0..N-1 with per-chunk offload, then
the reverse backward walk with prefetch (Sec. 5.1-5.2 of SPPO).

Only C-ABI calls and torch allocations happen here; every arithmetic step of
the path runs in the library's kernels.  Device tensors:
    q, do      [B, S, Hq, D]    inputs (dtype of the problem)
    k, v       [B, S, Hkv, D]   the resident K/V cache
    o, dq      [B, S, Hq, D]    outputs
    lse        per chunk [B, Hq, s_i] fp32, stored back to back
    dk, dv     [B, S, Hkv, D]   fp32 accumulators
For B = 1 every chunk tensor is a contiguous view of the full tensor; for
B > 1 the chunk-local tensors are separate contiguous buffers.

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


class ChunkedAttention:
    def __init__(self, B, S, n_chunks, Hq, Hkv, D, dtype="bf16", offsets=None, scale=0.0,
                 offload="none", device="cuda", host_ahead=2):
        self.ctx = L.sppo_create(B, S, n_chunks, Hq, Hkv, D, dtype=dtype, chunk_offsets=offsets,
                                 softmax_scale=scale, offload=offload)
        self.B, self.S, self.N, self.Hq, self.Hkv, self.D = B, S, n_chunks, Hq, Hkv, D
        self.offsets = L.sppo_get_offsets(self.ctx)
        self.torch_dtype = torch.bfloat16 if self.ctx.problem["dtype"] == L.SPPO_BF16 else torch.float32
        self.offload = L.OFFLOAD_MODES.get(offload, offload)
        self.device = device
        self.pacer = HostPacer(host_ahead)

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

    def alloc_outputs(self):
        B, S, Hq, Hkv, D = self.B, self.S, self.Hq, self.Hkv, self.D
        dev, dt = self.device, self.torch_dtype
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

    def step(self, inp, out, offload_chunks=None, lookahead=2, poison=False, stream=None, marks=None):
        """One forward + backward pass over all chunks.  With ``marks`` (a
        list), timing events are recorded on the stream before each chunk's
        forward and backward and at the end, appended as (label, event)."""
        if offload_chunks is None:
            offload_chunks = self.default_offload_chunks()
        offl = set(offload_chunks)
        s = torch.cuda.current_stream() if stream is None else stream
        q, k, v, do = inp["q"], inp["k"], inp["v"], inp["do"]
        qc = [self.chunk_view(q, i) for i in range(self.N)]
        dc = [self.chunk_view(do, i) for i in range(self.N)]
        oc = [self.chunk_view(out["o"], i) for i in range(self.N)]
        dqc = [self.chunk_view(out["dq"], i) for i in range(self.N)]
        lse = out["lse"]
        rows = self.offload_rows() if poison else None

        def mark(label):
            self.pacer.boundary(s)
            if marks is not None:
                e = torch.cuda.Event(enable_timing=True)
                e.record(s)
                marks.append((label, e))

        for i in range(self.N):
            mark(("fwd", i))
            L.sppo_attn_fwd_chunk(self.ctx, i, qc[i], k, v, oc[i], lse[i], s)
            if i in offl:
                bufs = L.chunk_bufs(q=qc[i], o=oc[i], lse=lse[i], k=k, v=v)
                L.sppo_offload_issue(self.ctx, i, bufs, s)
                if poison:
                    # Test hook: once the copy has landed on the host, the
                    # offloaded rows on the device are dead; overwrite them
                    # with NaN (the resident remainder stays intact).
                    L.sppo_offload_wait(self.ctx, i, s)
                    r = rows[i]
                    with torch.cuda.stream(s):
                        qc[i][:, :r].fill_(float("nan"))
                        oc[i][:, :r].fill_(float("nan"))
                        lse[i][:, :, :r].fill_(float("nan"))
        if self.offload == L.SPPO_OFFLOAD_QKVOL_EVICT:
            kv_chunks = sorted(offl, reverse=True)
            if poison:
                # Test hook: the evicted K/V rows are dead once their copies
                # have landed; overwrite them with NaN.
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
        nxt = 0
        for i in reversed(range(self.N)):
            while nxt < len(pending) and pending[nxt] >= i - lookahead:
                j = pending[nxt]
                L.sppo_prefetch(self.ctx, j, L.chunk_bufs(q=qc[j], o=oc[j], lse=lse[j]), s)
                nxt += 1
            mark(("bwd", i))
            L.sppo_attn_bwd_chunk(self.ctx, i, qc[i], k, v, oc[i], lse[i], dc[i], dqc[i],
                                  out["dk"], out["dv"], s)
        mark(("end", -1))
        if self.B > 1:
            for i in range(self.N):
                c0, c1 = self.offsets[i], self.offsets[i + 1]
                out["o"][:, c0:c1].copy_(oc[i])
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
