"""One full transformer layer over a chunked sequence, composed of libsppo
calls: the forward walks the chunks 0..N-1, the backward N-1..0 (Sec. 5.1-5.2
of SPPO), batch 1.

The layer (pre-LayerNorm GPT block, MLP width 4H, no projection biases):
    u = LN1(x); q, k, v = u W_qkv; O = causal attention; h = x + O W_o
    z = LN2(h); a = z W_1; y = h + gelu(a) W_2
Weights are bf16 [in, out] (W_qkv columns [q | k | v]); LayerNorm
parameters fp32.  The walk keeps the transposed weights for the forward
GEMMs (C = A B^T with B = W^T) and uses the weights as stored for the data
gradients.

Two-level activation management (Sec. 5.1): the K/V cache of the whole
sequence stays on the device; every other tensor a chunk's backward needs --
Q_i, O_i, LSE_i and the "extra planes" x_i, h_i, a_i and the two
LayerNorms' statistics -- is offloaded after the chunk's forward (all chunks
but the last by default) and prefetched before its backward.  u, z and
gelu(a) are recomputed in the backward from x, h and a.  With
``qkvol_evict`` the offloaded chunks' K/V cache rows are given up after the
forward walk as well and stream back under the last chunk's backward.

The saved tensors a chunk produces live in a region of a preallocated
device arena (ring.DeviceArena): an offloaded chunk's region is reused once
its copy has landed, and its prefetch lands in a free region.  x_i is read
from the caller's x in the forward (those rows of x are dead once
offloaded) and comes back into the chunk's region.

The host stays at most ``host_ahead`` chunk boundaries ahead of the device
(a HostPacer; 0 lets it run free).

Only C-ABI calls and torch allocations happen here; every arithmetic step
runs in the library's kernels.
"""
from __future__ import annotations

import torch

from . import sppo as L
from .pacing import HostPacer
from .ring import DeviceArena, KeepArena, plan_capacity, plane_layout, walk_schedule

PLANES = ("x", "h", "a", "m1", "r1", "m2", "r2")


class ChunkedLayer:
    def __init__(self, S, n_chunks, Hq, Hkv, D, offsets=None, offload="none", device="cuda", eps=1e-5,
                 host_ahead=2, fwd_slots=4):
        H = Hq * D
        wt = (Hq + 2 * Hkv) * D
        if H % 256 or wt % 256 or H > 8192:
            raise ValueError("the layer needs Hq*D and (Hq+2Hkv)*D multiples of 256 and Hq*D <= 8192")
        self.S, self.N, self.Hq, self.Hkv, self.D, self.H, self.Wt = S, n_chunks, Hq, Hkv, D, H, wt
        self.eps = eps
        self.device = device
        row_bytes = [2 * H, 2 * H, 8 * H, 4, 4, 4, 4]  # x, h, a bf16; mean/rstd of LN1, LN2 fp32
        self.ctx = L.sppo_create(1, S, n_chunks, Hq, Hkv, D, dtype="bf16", chunk_offsets=offsets,
                                 offload=offload, extra_row_bytes=row_bytes)
        self.offsets = L.sppo_get_offsets(self.ctx)
        self.offload = L.OFFLOAD_MODES.get(offload, offload)
        self.s_max = max(self.offsets[i + 1] - self.offsets[i] for i in range(n_chunks))
        self.pacer = HostPacer(host_ahead)
        self.fwd_slots = fwd_slots
        self.arena = None
        self.keep = None
        self._layout = None
        self._alloc()

    def close(self):
        self.ctx.close()

    def chunk_len(self, i):
        return self.offsets[i + 1] - self.offsets[i]

    def _alloc(self):
        S, H, Wt, dev = self.S, self.H, self.Wt, self.device
        bf, f32 = torch.bfloat16, torch.float32
        HqD, HkvD, sm = self.Hq * self.D, self.Hkv * self.D, self.s_max
        e = lambda *shape, dt=bf: torch.empty(*shape, dtype=dt, device=dev)
        # the K/V cache and its gradient accumulators (full length)
        self.k, self.v = e(S, HkvD), e(S, HkvD)
        self.dk, self.dv = e(S, HkvD, dt=f32), e(S, HkvD, dt=f32)
        # transposed weights for the forward GEMMs
        self.wT = {"w_qkv": e(Wt, H), "w_o": e(H, HqD), "w_1": e(4 * H, H), "w_2": e(H, 4 * H)}
        # chunk-sized scratch
        self.u, self.z, self.g = e(sm, H), e(sm, H), e(sm, 4 * H)
        self.da, self.dz, self.dh = e(sm, 4 * H), e(sm, H), e(sm, H)
        self.dO, self.dq, self.dqkv, self.du = e(sm, HqD), e(sm, HqD), e(sm, Wt), e(sm, H)
        wsb = max(L.sppo_layernorm_bwd_workspace(self.chunk_len(i), H) for i in range(self.N))
        self.ws = torch.empty(wsb // 4, dtype=f32, device=dev)
        self.ws_bytes = wsb

    def alloc_outputs(self):
        H, Wt, dev = self.H, self.Wt, self.device
        f32 = torch.float32
        return {"y": torch.empty(self.S, H, dtype=torch.bfloat16, device=dev),
                "dx": torch.empty(self.S, H, dtype=torch.bfloat16, device=dev),
                "dw_qkv": torch.empty(H, Wt, dtype=f32, device=dev),
                "dw_o": torch.empty(self.Hq * self.D, H, dtype=f32, device=dev),
                "dw_1": torch.empty(H, 4 * H, dtype=f32, device=dev),
                "dw_2": torch.empty(4 * H, H, dtype=f32, device=dev),
                **{k: torch.empty(H, dtype=f32, device=dev) for k in ("dg1", "db1", "dg2", "db2")}}

    def offload_bytes_per_row(self):
        """Bytes per token row of the offload set: Q, O, LSE, the extra planes
        (and K, V in the QKVOL modes)."""
        b = 2 * self.Hq * self.D * 2 + 4 * self.Hq + 12 * self.H + 16
        if self.offload in (L.SPPO_OFFLOAD_QKVOL, L.SPPO_OFFLOAD_QKVOL_EVICT):
            b += 2 * self.Hkv * self.D * 2
        return b

    def set_offload_rows(self, rows):
        for i, r in enumerate(rows):
            L.sppo_set_offload_rows(self.ctx, i, r)

    # ------------------------------------------------------------ the walk
    def region_planes(self, i):
        """Byte sizes of chunk i's saved tensors in its arena region."""
        n, H, HqD = self.chunk_len(i), self.H, self.Hq * self.D
        return {"q": 2 * n * HqD, "o": 2 * n * HqD, "lse": 4 * self.Hq * n, "x": 2 * n * H, "h": 2 * n * H,
                "a": 8 * n * H, "m1": 4 * n, "r1": 4 * n, "m2": 4 * n, "r2": 4 * n}

    def prepare(self, offload_chunks, lookahead):
        """Allocate the device arena and keep buffers for a walk with these
        settings (again only when they change; a walk allocates nothing).
        Returns the bytes they hold."""
        offl = tuple(sorted(set(offload_chunks)))
        key = (offl, lookahead, tuple(L.sppo_get_offload_rows(self.ctx)))
        if self._layout != key:
            self._planes = [plane_layout(self.region_planes(i)) for i in range(self.N)]
            q = self.fwd_slots - 1
            cap, q = plan_capacity(walk_schedule(self.N, offl, lookahead), [sz for _, sz in self._planes],
                                   quarantine=q)
            self.arena = None
            self.keep = None
            self.arena = DeviceArena(cap, self.device, quarantine=q)
            self.keep = KeepArena([L.sppo_keep_bytes(self.ctx, i) if i in offl else 0 for i in range(self.N)],
                                  self.device)
            self._layout = key
        return self.arena.nbytes + self.keep.nbytes

    def _acquire(self, i, s, x=None):
        """Allocate chunk i's region; returns (offset, views of its saved
        tensors).  x_i is the caller's rows when given, else the region's x
        plane (where a prefetch puts it)."""
        off = self.arena.acquire(self.ctx, s, self._planes[i][1], i)
        n, H, HqD = self.chunk_len(i), self.H, self.Hq * self.D
        bf, f32 = torch.bfloat16, torch.float32
        po = self._planes[i][0]
        pl = lambda name, shape, dt: self.arena.view(off + po[name], shape, dt)  # noqa: E731
        v = dict(q=pl("q", (n, HqD), bf), o=pl("o", (n, HqD), bf), lse=pl("lse", (self.Hq, n), f32),
                 h=pl("h", (n, H), bf), a=pl("a", (n, 4 * H), bf),
                 **{k: pl(k, (n,), f32) for k in ("m1", "r1", "m2", "r2")})
        v["x"] = x if x is not None else pl("x", (n, H), bf)
        return off, v

    def _bufs(self, v, keep):
        return L.chunk_bufs(q=v["q"], o=v["o"], lse=v["lse"], k=self.k, v=self.v,
                            extra=[v[name] for name in PLANES], keep=keep)

    def step(self, inp, p, out, offload_chunks=None, lookahead=2, poison=False, stream=None, marks=None,
             ops=None):
        """Forward and backward of the layer over all chunks.  inp: x, dy
        [S, H] bf16 (x's chunk rows are the x planes: offloading a chunk
        makes its rows of x dead, and the prefetch brings them back into the
        chunk's arena region; poison=True overwrites every dead buffer -- the
        rows of x and the chunk's region -- with NaN once copied).  p: the
        weights (w_qkv, w_o, w_1, w_2 bf16; g1, b1, g2, b2 fp32).  marks:
        list that receives ((phase, chunk), event) at every chunk boundary.
        ops: list that receives (category, algorithmic flop, start event,
        end event) around every library call on the compute stream."""
        s = torch.cuda.current_stream() if stream is None else stream
        H, Wt, HqD, HkvD = self.H, self.Wt, self.Hq * self.D, self.Hkv * self.D
        if offload_chunks is None:
            offload_chunks = [] if self.offload == L.SPPO_OFFLOAD_NONE else list(range(self.N - 1))
        offl = set(offload_chunks)
        self.prepare(offl, lookahead)
        arena, keep = self.arena, self.keep
        arena.reset()
        x, dy = inp["x"], inp["dy"]

        def mark(label):
            self.pacer.boundary(s)
            if marks is not None:
                ev = torch.cuda.Event(enable_timing=True)
                ev.record(s)
                marks.append((label, ev))

        def timed(cat, fn, flop=0):
            def call(*a, **kw):
                if ops is None:
                    return fn(*a, **kw)
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(s)
                r = fn(*a, **kw)
                e1.record(s)
                ops.append((cat(a) if callable(cat) else cat, flop(a) if callable(flop) else flop, e0, e1))
                return r
            return call

        gemm = timed(lambda a: "gemm_" + a[0] + ("_fwd" if fwd_phase[0] and a[0] == "nt" else
                                                 "_bwd" if a[0] == "nt" else ""),
                     L.sppo_gemm_bf16, lambda a: 2 * a[1] * a[2] * a[3])
        fwd_phase = [True]
        transpose = timed("transpose", L.sppo_transpose_bf16)
        ln_fwd = timed("layernorm", L.sppo_layernorm_fwd)
        ln_bwd = timed("layernorm", L.sppo_layernorm_bwd)
        gelu = timed("gelu", L.sppo_gelu_bf16)
        pack = timed("pack", L.sppo_pack_qkv_grad)
        pairs = lambda a: self.chunk_len(a[1]) * self.offsets[a[1]] + self.chunk_len(a[1]) * (self.chunk_len(a[1]) + 1) // 2
        attn_fwd = timed("attn_fwd", L.sppo_attn_fwd_chunk, lambda a: 4 * self.D * self.Hq * pairs(a))
        attn_bwd = timed("attn_bwd", L.sppo_attn_bwd_chunk, lambda a: 10 * self.D * self.Hq * pairs(a))

        mark(("wT", -1))
        transpose(p["w_qkv"], self.wT["w_qkv"], H, Wt, s)
        transpose(p["w_o"], self.wT["w_o"], HqD, H, s)
        transpose(p["w_1"], self.wT["w_1"], H, 4 * H, s)
        transpose(p["w_2"], self.wT["w_2"], 4 * H, H, s)
        held, back = {}, {}  # chunk -> (region, views): not offloaded / prefetched
        for i in range(self.N):
            mark(("fwd", i))
            n, c0 = self.chunk_len(i), self.offsets[i]
            slot, v = self._acquire(i, s, x=x[c0:c0 + n])
            u, z, g = self.u[:n], self.z[:n], self.g[:n]
            ln_fwd(n, H, v["x"], H, p["g1"], p["b1"], self.eps, u, H, v["m1"], v["r1"], s)
            wq = self.wT["w_qkv"]
            gemm("nt", n, HqD, H, u, H, wq, H, v["q"], HqD, stream=s)
            gemm("nt", n, HkvD, H, u, H, wq[HqD:], H, self.k[c0:], HkvD, stream=s)
            gemm("nt", n, HkvD, H, u, H, wq[HqD + HkvD:], H, self.v[c0:], HkvD, stream=s)
            attn_fwd(self.ctx, i, v["q"], self.k, self.v, v["o"], v["lse"], s)
            gemm("nt", n, H, HqD, v["o"], HqD, self.wT["w_o"], HqD, v["h"], H, "add_bf16", v["x"], H, stream=s)
            ln_fwd(n, H, v["h"], H, p["g2"], p["b2"], self.eps, z, H, v["m2"], v["r2"], s)
            gemm("nt", n, 4 * H, H, z, H, self.wT["w_1"], H, g, 4 * H, "gelu", v["a"], 4 * H, stream=s)
            gemm("nt", n, H, 4 * H, g, 4 * H, self.wT["w_2"], 4 * H, out["y"][c0:], H, "add_bf16", v["h"], H,
                 stream=s)
            if i in offl:
                L.sppo_offload_issue(self.ctx, i, self._bufs(v, keep.ptr(i)), s)
                arena.release(slot, after_offload=True)
                if poison:
                    # Test hook: once copied, the chunk's region and its rows of
                    # x are dead (the rows that stay went to the keep buffer).
                    L.sppo_offload_wait(self.ctx, i, s)
                    with torch.cuda.stream(s):
                        for t in v.values():
                            t.fill_(float("nan"))
            else:
                held[i] = (slot, v)
        fwd_phase[0] = False
        if self.offload == L.SPPO_OFFLOAD_QKVOL_EVICT:
            # The K/V cache rows of the offloaded chunks are given up here;
            # their copies come back on the host-to-device stream in the order
            # the last chunk's backward consumes them (chunk by chunk).
            rows = L.sppo_get_offload_rows(self.ctx)
            kv_chunks = sorted(offl, reverse=True)
            if poison:
                # Test hook: the evicted rows are dead once their copies have landed.
                for j in kv_chunks:
                    L.sppo_offload_wait(self.ctx, j, s)
                with torch.cuda.stream(s):
                    for j in kv_chunks:
                        c0 = self.offsets[j]
                        self.k[c0:c0 + rows[j]].fill_(float("nan"))
                        self.v[c0:c0 + rows[j]].fill_(float("nan"))
            for j in kv_chunks:
                L.sppo_prefetch_kv(self.ctx, j, self.k, self.v, s)
        pending = sorted(offl, reverse=True)
        nxt = 0
        for i in reversed(range(self.N)):
            while nxt < len(pending) and pending[nxt] >= i - lookahead:
                j = pending[nxt]
                slot, vj = self._acquire(j, s)
                L.sppo_prefetch(self.ctx, j, self._bufs(vj, keep.ptr(j)), s)
                back[j] = (slot, vj)
                nxt += 1
            mark(("bwd", i))
            n, c0 = self.chunk_len(i), self.offsets[i]
            slot, v = back.pop(i) if i in offl else held.pop(i)
            if i in offl:
                L.sppo_prefetch_wait(self.ctx, i, s)
            first = i == self.N - 1  # overwrite the weight gradients instead of adding
            wacc = "f32" if first else "acc_f32"
            u, z, g = self.u[:n], self.z[:n], self.g[:n]
            da, dz, dh, dO = self.da[:n], self.dz[:n], self.dh[:n], self.dO[:n]
            dyi = dy[c0:c0 + n]
            # y = h + gelu(a) W2
            gelu(v["a"], g, n * 4 * H, s)
            gemm("nt", n, 4 * H, H, dyi, H, p["w_2"], H, da, 4 * H, "dgelu", v["a"], 4 * H, stream=s)
            gemm("tn", 4 * H, H, n, g, 4 * H, dyi, H, out["dw_2"], H, wacc, stream=s)
            # a = z W1, z = LN2(h)
            ln_fwd(n, H, v["h"], H, p["g2"], p["b2"], self.eps, z, H, v["m2"], v["r2"], s)
            gemm("nt", n, H, 4 * H, da, 4 * H, p["w_1"], 4 * H, dz, H, stream=s)
            gemm("tn", H, 4 * H, n, z, H, da, 4 * H, out["dw_1"], 4 * H, wacc, stream=s)
            ln_bwd(n, H, v["h"], H, p["g2"], v["m2"], v["r2"], dz, H, dyi, H, dh, H, out["dg2"],
                                 out["db2"], self.ws, self.ws_bytes, accumulate=0 if first else 1, stream=s)
            # h = x + O Wo
            gemm("nt", n, HqD, H, dh, H, p["w_o"], H, dO, HqD, stream=s)
            gemm("tn", HqD, H, n, v["o"], HqD, dh, H, out["dw_o"], H, wacc, stream=s)
            attn_bwd(self.ctx, i, v["q"], self.k, self.v, v["o"], v["lse"], dO, self.dq[:n],
                                  self.dk, self.dv, s)
            # q, k, v = u W_qkv (chunk i's dK/dV rows are complete now)
            dqkv = self.dqkv[:n]
            pack(n, HqD, HkvD, self.dq[:n], self.dk, self.dv, c0, dqkv, s)
            ln_fwd(n, H, v["x"], H, p["g1"], p["b1"], self.eps, u, H, v["m1"], v["r1"], s)
            gemm("nt", n, H, Wt, dqkv, Wt, p["w_qkv"], Wt, self.du[:n], H, stream=s)
            gemm("tn", H, Wt, n, u, H, dqkv, Wt, out["dw_qkv"], Wt, wacc, stream=s)
            # u = LN1(x); x also reaches h
            ln_bwd(n, H, v["x"], H, p["g1"], v["m1"], v["r1"], self.du[:n], H, dh, H,
                                 out["dx"][c0:], H, out["dg1"], out["db1"], self.ws, self.ws_bytes,
                                 accumulate=0 if first else 1, stream=s)
            arena.release(slot)
        mark(("end", -1))

    @staticmethod
    def flops(S, offsets, Hq, Hkv, D):
        """Algorithmic flop of one forward + backward: the GEMMs (3 x 2 m n k
        per projection) plus attention (14 D per visible pair per head)."""
        H, wt = Hq * D, (Hq + 2 * Hkv) * D
        gemm = 3 * 2 * S * (H * wt + Hq * D * H + 2 * H * 4 * H)
        pairs = 0
        for i in range(len(offsets) - 1):
            s_i, c_i = offsets[i + 1] - offsets[i], offsets[i]
            pairs += s_i * c_i + s_i * (s_i + 1) // 2
        return gemm + 14 * D * Hq * pairs, gemm
