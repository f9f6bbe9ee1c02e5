"""The seeded input generator (CPU): every tensor, seed, batch entry and
block gets its own stream of draws, on the CPU generator (which keeps only
the low 32 bits of a seed) as on the device one, and the block seeding keeps
a tensor independent of the sequence length it is cut from."""
import itertools

import numpy as np
import pytest
import torch

from paper_2503_10377_amd.inputs import BLOCK_ROWS, _block_seed, make_inputs, make_layer_inputs


def test_block_seeds_differ_in_their_low_32_bits():
    keys = list(itertools.product((0, 1, 2, 99, 255), range(18), range(8), (0, 1, 2, 255, 256, 65535)))
    low = {_block_seed(*k) & 0xFFFFFFFF for k in keys}
    full = {_block_seed(*k) for k in keys}
    assert len(low) == len(keys) and len(full) == len(keys)
    for bad in ((256, 0, 0, 0), (0, 32, 0, 0), (0, 0, 8, 0), (0, 0, 0, 65536), (-1, 0, 0, 0)):
        with pytest.raises(ValueError):
            _block_seed(*bad)


def test_tensors_seeds_and_blocks_draw_different_values():
    S = 2 * BLOCK_ROWS
    a = make_inputs(2, S, 2, 2, 64, torch.float32, seed=1, device="cpu")
    b = make_inputs(2, S, 2, 2, 64, torch.float32, seed=2, device="cpu")
    names = ("q", "k", "v", "do")
    for x, y in itertools.combinations(names, 2):
        assert not torch.equal(a[x], a[y]), (x, y)
    for n in names:
        assert not torch.equal(a[n], b[n]), n
        assert not torch.equal(a[n][0], a[n][1]), n  # batch entries
        assert not torch.equal(a[n][:, :BLOCK_ROWS], a[n][:, BLOCK_ROWS:]), n  # blocks
    # pairwise correlation of different tensors is that of independent draws
    k, v = a["k"].flatten().double(), a["v"].flatten().double()
    assert abs(float(torch.corrcoef(torch.stack([k, v]))[0, 1])) < 5 / np.sqrt(k.numel())


def test_draws_are_standard_normal():
    x = make_inputs(1, BLOCK_ROWS, 4, 4, 128, torch.float32, seed=3, device="cpu")["v"].double()
    n = x.numel()
    assert abs(float(x.mean())) < 5 / np.sqrt(n)
    assert abs(float(x.var()) - 1.0) < 5 * np.sqrt(2 / n)


def test_a_prefix_of_a_longer_sequence_is_the_shorter_sequence():
    short = make_inputs(1, BLOCK_ROWS + 100, 2, 1, 64, torch.bfloat16, seed=4, device="cpu")
    long = make_inputs(1, 3 * BLOCK_ROWS, 2, 1, 64, torch.bfloat16, seed=4, device="cpu")
    for n in short:
        assert torch.equal(short[n], long[n][:, :BLOCK_ROWS + 100]), n


def test_layer_tensors_draw_different_values():
    inp, p = make_layer_inputs(64, 2, 1, 64, seed=0, device="cpu")
    assert not torch.equal(inp["x"], inp["dy"])
    assert not torch.equal(p["g1"], p["g2"]) and not torch.equal(p["b1"], p["b2"])
    w = p["w_qkv"].float()[:64, :64].flatten()
    x = inp["x"].float()[:, :64].flatten()
    assert abs(float(torch.corrcoef(torch.stack([w, x]))[0, 1])) < 5 / np.sqrt(w.numel())
