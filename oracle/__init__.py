"""fp64 CPU oracle for sequence-chunked causal attention (forward and backward).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and its
Python binding) may import, call or link anything under this directory.  Only
the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` use it.

The oracle is independent of the GPU path: it shares no code, headers, tables
or helpers with ``paper_2503_10377_amd``.  It takes plain float64 NumPy arrays
(the exact values the GPU received, upcast) and returns float64 arrays.

Layout conventions (BSHD, token-major):
    q, o, do, dq : [B, S, Hq, D]
    k, v, dk, dv : [B, S, Hkv, D]
    lse          : [B, Hq, S]       natural-log logsumexp of each query row
Query head h reads KV head h // (Hq // Hkv) (contiguous grouping).

Pins: every function here is checked in ``tests/test_oracle_*.py`` against
brute-force loops, central finite differences, closed forms and invariants
(see the module docstrings for which pin covers which function).
"""
from .causal_attention import (  # noqa: F401
    attention_fwd,
    attention_bwd,
    attention,
    chunked_attention_fwd,
    chunked_attention_bwd,
    equal_offsets,
    rows_fwd_bwd,
    tail_keys_bwd,
    keys_bwd_rows,
)
from .transformer_layer import (  # noqa: F401
    chunked_layer,
    gelu,
    gelu_grad,
    layer,
    layer_backward,
    layer_forward,
    layer_norm,
    layer_norm_bwd,
)
