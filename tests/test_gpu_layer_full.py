"""The full-layer walk at the benchmarked size and launch configuration
(128K tokens in 16 chunks of 8192, width 4096 = 32 heads x 128, MLP 16384,
Q/O/LSE and the layer's other saved activations offloaded), checked against
the fp64 layer oracle where the oracle can follow at this size:

  forward   y at sampled rows below 16384 (chunks 0 and 1, including both
            chunk boundaries there): row r depends on rows 0..r only, so the
            oracle needs the K/V projections of that prefix and each sampled
            row's own query and MLP;
  backward  dy is zero past row 1024; causality then makes every gradient
            (dx, the weight and LayerNorm-parameter gradients) equal to that of
            the first 1024 rows as a standalone sequence, which the oracle runs
            in full, and dx past row 1024 exactly zero (a zero upstream
            gradient yields exact zeros at every step).

Same gates as the small layer tests: relative Frobenius error <= 1.2e-2 and
max error <= 1.5e-2 of the largest reference value, per tensor.
"""
import sys
import time

import numpy as np
import pytest
import torch

from oracle import transformer_layer as T
from paper_2503_10377_amd.chunked_layer import ChunkedLayer
from paper_2503_10377_amd.inputs import make_layer_inputs
from parity import to_np

pytestmark = pytest.mark.gpu

S, N, HQ, HKV, D = 131072, 16, 32, 32, 128
R_FWD, R_BWD = 16384, 1024
REL, MAXREL = 1.2e-2, 1.5e-2
PARAMS = ("w_qkv", "w_o", "w_1", "w_2", "g1", "b1", "g2", "b2")


def gate(name, got, ref):
    rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    mx = np.abs(got - ref).max() / np.abs(ref).max()
    print(f"  {name:7s} rel_fro {rel:.2e} max_rel {mx:.2e}", file=sys.stderr, flush=True)
    assert np.isfinite(got).all(), name
    assert rel <= REL and mx <= MAXREL, (name, rel, mx)


def test_layer_at_128k_against_the_oracle():
    print(f"\n[case] layer S={S} N={N} Hq={HQ} Hkv={HKV} D={D} offload=qol, dy zero past row {R_BWD}",
          file=sys.stderr, flush=True)
    inp, p = make_layer_inputs(S, HQ, HKV, D, seed=3, device="cuda")
    inp["dy"][R_BWD:] = 0
    # host copies of the inputs before the HIP path runs
    x_fwd = to_np(inp["x"][:R_FWD])
    x_bwd, dy_bwd = x_fwd[:R_BWD], to_np(inp["dy"][:R_BWD])
    hp = {k: to_np(p[k]) for k in PARAMS}
    lay = ChunkedLayer(S, N, HQ, HKV, D, offload="qol")
    out = lay.alloc_outputs()
    t0 = time.time()
    lay.step(inp, p, out)
    torch.cuda.synchronize()
    print(f"  walk {time.time() - t0:.1f} s", file=sys.stderr, flush=True)
    rng = np.random.default_rng(11)
    rows = sorted(set([0, 1, 2, 255, 256, 8191, 8192, 8193, 16383]) | set(rng.integers(0, R_FWD, 23).tolist()))
    y_rows = to_np(out["y"][rows])
    dx = to_np(out["dx"])
    grads = {k: to_np(out[k]) for k in ("dw_qkv", "dw_o", "dw_1", "dw_2", "dg1", "db1", "dg2", "db2")}
    lay.close()
    del inp, p, out
    t0 = time.time()
    ref_y = T.layer_forward_rows(x_fwd, hp, rows, HQ, HKV, D)
    ref = T.layer(x_bwd, dy_bwd, hp, HQ, HKV, D)
    print(f"  oracle {time.time() - t0:.1f} s", file=sys.stderr, flush=True)
    gate("y[rows]", y_rows, ref_y)
    gate("dx", dx[:R_BWD], ref["dx"])
    assert np.all(dx[R_BWD:] == 0), "dx past the rows with a nonzero dy"
    for k, v in grads.items():
        gate(k, v, ref[k])
