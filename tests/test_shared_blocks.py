"""Host check of the shared experts' cut into blocks of the routed width f.

LayerShare runs a shared expert of width m f as m experts of width f inside the
routed experts' call (gate rows, the matching up rows and the matching columns
of W2).  The cut is exact algebra (SiLU(a) * b acts per element of h and the
down product sums over h), so the oracle's FFN of the blocks, summed, must equal
its FFN of the whole expert to fp64 rounding; a wrong slice (gate and up rows
misaligned, W2 columns of another block, a transposed W2) fails it.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_08782_amd.layer import shared_blocks


def _expert(rng, d, f):
    return (rng.standard_normal((2 * f, d)) / np.sqrt(d), rng.standard_normal((d, f)) / np.sqrt(f))


@pytest.mark.parametrize("widths,f", [((256,), 64), ((128, 64), 64), ((192, 64, 128), 64),
                                      ((64,), 64)])
def test_blocks_sum_to_the_shared_experts(widths, f):
    rng = np.random.default_rng(sum(widths) + f)
    d, T = 48, 37
    experts = [_expert(rng, d, w) for w in widths]
    shared = [(torch.from_numpy(a), torch.from_numpy(b)) for a, b in experts]
    b13, b2 = shared_blocks(shared, f)
    assert len(b13) == sum(w // f for w in widths)
    for a, b in zip(b13, b2):
        assert tuple(a.shape) == (2 * f, d) and tuple(b.shape) == (d, f)
    x = rng.standard_normal((T, d))
    whole = sum(oracle.expert_ffn(x, a, b) for a, b in experts)
    cut = sum(oracle.expert_ffn(x, a.numpy(), b.numpy()) for a, b in zip(b13, b2))
    np.testing.assert_allclose(cut, whole, rtol=0, atol=1e-12 * np.abs(whole).max())


def test_block_boundaries_follow_the_gate_and_up_halves():
    """Block j of an expert of width 2f: gate rows [j f, (j+1) f), up rows
    [2f + j f, 2f + (j+1) f), W2 columns [j f, (j+1) f)."""
    d, f = 8, 4
    w13 = torch.arange(4 * f * d, dtype=torch.float64).reshape(4 * f, d)
    w2 = torch.arange(d * 2 * f, dtype=torch.float64).reshape(d, 2 * f)
    b13, b2 = shared_blocks([(w13, w2)], f)
    assert torch.equal(b13[1][:f], w13[f:2 * f]) and torch.equal(b13[1][f:], w13[3 * f:])
    assert torch.equal(b2[1], w2[:, f:])


def test_widths_that_are_not_multiples_of_f_are_refused():
    rng = np.random.default_rng(0)
    a, b = _expert(rng, 16, 96)
    assert shared_blocks([(torch.from_numpy(a), torch.from_numpy(b))], 64) is None
    assert shared_blocks([], 64) is None
    assert shared_blocks([(torch.from_numpy(a), torch.from_numpy(b))], 0) is None
