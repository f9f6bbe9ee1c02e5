"""Seeded synthetic inputs for the chunked-attention path.

Shared by the tests, ``__graft_entry__.smoke()`` and ``bench.py``; holds none
of the attention arithmetic.  Values are i.i.d. N(0, 1) drawn in fp32 on the
target device and rounded to the problem dtype (round-to-nearest-even for
bf16).  Every block of 4096 rows of every tensor has its own seed derived
from (seed, tensor, batch entry, block), so a tensor does not depend on how
the sequence is chunked, and a prefix of a longer sequence is identical to
the shorter one.

Structured kinds exercise what random inputs cannot:
    "randn"        Q, K, V, dO ~ N(0, 1)
    "sharp_self"   Q[:, r, h] = 2 K[:, r, h // G]  (each row's own key dominates)
    "sharp_future" Q[:, r, h] = 2 K[:, r+1, h // G] (the first invisible key
                   dominates if the mask admits it; the last row uses its own key)
    "zero_q"       Q = 0 (softmax is uniform over the visible keys)
Multiplying by 2 is exact in bf16, so the structure survives the rounding.
"""
from __future__ import annotations

import torch

TENSOR_IDS = {"q": 0, "k": 1, "v": 2, "do": 3}
BLOCK_ROWS = 4096
KINDS = ("randn", "sharp_self", "sharp_future", "zero_q")


_M32 = 0xFFFFFFFF


def _mix32(x: int) -> int:
    """An invertible mix of 32-bit integers (xor-shifts and odd multipliers,
    each a bijection), so distinct inputs give distinct outputs."""
    x ^= x >> 16
    x = (x * 0x7FEB352D) & _M32
    x ^= x >> 15
    x = (x * 0x846CA68B) & _M32
    return x ^ (x >> 16)


def _block_seed(seed: int, tid: int, b: int, blk: int) -> int:
    """64-bit generator seed of one block of one tensor.  (seed, tensor,
    batch entry, block) are packed into 32 bits and mixed bijectively into
    both halves: torch's CPU generator keeps only the low 32 bits of a seed
    (the device generator all 64), so the low half alone must already differ
    for every block, or on the CPU every tensor would draw the same values."""
    if not (0 <= seed < 256 and 0 <= tid < 32 and 0 <= b < 8 and 0 <= blk < 65536):
        raise ValueError(f"seed {seed}, tensor {tid}, batch entry {b} or block {blk} out of the generator's range "
                         "(seed < 256, batch < 8, sequence < 2^28 rows)")
    key = (seed << 24) | (tid << 19) | (b << 16) | blk
    return (_mix32(key ^ 0x5BD1E995) << 32) | _mix32(key)


def randn_bshd(shape, seed: int, tid: int, device, dtype) -> torch.Tensor:
    """[B, S, H, D] tensor of N(0,1) draws rounded to ``dtype``, block-seeded."""
    B, S, H, D = shape
    out = torch.empty(shape, dtype=dtype, device=device)
    gen = torch.Generator(device=device)
    for b in range(B):
        for r0 in range(0, S, BLOCK_ROWS):
            r1 = min(S, r0 + BLOCK_ROWS)
            gen.manual_seed(_block_seed(seed, tid, b, r0 // BLOCK_ROWS))
            blk = torch.randn((r1 - r0, H, D), generator=gen, device=device, dtype=torch.float32)
            out[b, r0:r1].copy_(blk.to(dtype))
            del blk
    return out


def make_inputs(B: int, S: int, Hq: int, Hkv: int, D: int, dtype=torch.bfloat16, seed: int = 0,
                device="cuda", kind: str = "randn") -> dict:
    """Q, dO [B,S,Hq,D] and K, V [B,S,Hkv,D] on ``device``."""
    if kind not in KINDS:
        raise ValueError(f"unknown input kind {kind!r}")
    G = Hq // Hkv
    k = randn_bshd((B, S, Hkv, D), seed, TENSOR_IDS["k"], device, dtype)
    v = randn_bshd((B, S, Hkv, D), seed, TENSOR_IDS["v"], device, dtype)
    do = randn_bshd((B, S, Hq, D), seed, TENSOR_IDS["do"], device, dtype)
    if kind == "randn":
        q = randn_bshd((B, S, Hq, D), seed, TENSOR_IDS["q"], device, dtype)
    elif kind == "zero_q":
        q = torch.zeros((B, S, Hq, D), dtype=dtype, device=device)
    else:
        src = k
        if kind == "sharp_future":
            src = torch.cat([k[:, 1:], k[:, -1:]], dim=1)
        q = (2 * src).repeat_interleave(G, dim=2).contiguous()
    return {"q": q, "k": k, "v": v, "do": do}


LAYER_IDS = {"x": 0, "dy": 1, "w_qkv": 2, "w_o": 3, "w_1": 4, "w_2": 5, "g1": 6, "b1": 7, "g2": 8, "b2": 9}


def make_layer_inputs(S: int, Hq: int, Hkv: int, D: int, seed: int = 0, device="cuda"):
    """Inputs and parameters of one pre-LayerNorm transformer layer of width
    H = Hq*D: x, dy [S, H] ~ N(0, 1) in bf16; weights [in, out] ~ N(0, 1/in)
    in bf16 (w_qkv [H, (Hq+2Hkv)D], w_o [Hq D, H], w_1 [H, 4H], w_2 [4H, H]);
    LayerNorm gamma ~ 1 + 0.1 N(0, 1), beta ~ 0.1 N(0, 1) in fp32.  Each
    tensor has its own seed derived from (seed, tensor)."""
    H, wt = Hq * D, (Hq + 2 * Hkv) * D
    shapes = {"x": (S, H), "dy": (S, H), "w_qkv": (H, wt), "w_o": (Hq * D, H), "w_1": (H, 4 * H),
              "w_2": (4 * H, H), "g1": (H,), "b1": (H,), "g2": (H,), "b2": (H,)}
    gen = torch.Generator(device=device)
    out = {}
    for name, shape in shapes.items():
        gen.manual_seed(_block_seed(seed, 8 + LAYER_IDS[name], 0, 0))
        t = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
        if name.startswith("w_"):
            out[name] = (t * shape[0] ** -0.5).to(torch.bfloat16)
        elif name in ("g1", "g2"):
            out[name] = 1.0 + 0.1 * t
        elif name in ("b1", "b2"):
            out[name] = 0.1 * t
        else:
            out[name] = t.to(torch.bfloat16)
        del t
    inp = {k: out.pop(k) for k in ("x", "dy")}
    return inp, out
