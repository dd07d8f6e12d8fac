"""Pin the oracle's model forward against an independent PyTorch float64 forward.

The forward follows the SwiGLU decoder of the paper's eq. (1) (Sec. "Drafting"),
with RMSNorm, rotate-half RoPE and grouped-query attention.  The reference in
``torch_ref`` is built from library routines (scaled_dot_product_attention,
complex RoPE, silu), so a dropped term, a wrong sign, a transposed operand or a
wrong KV-head grouping in the oracle fails here.
"""
import numpy as np
import pytest

import oracle
import sd2_inputs as si
import torch_ref
from oracle_fixtures import GQA, weights


def _check(wl, which, toks, add=None, tol=1e-9):
    wv, wd, ws = weights(wl)
    o = oracle.Oracle(wl, wv, wd, ws)
    dm = wl.verifier if which == 0 else wl.drafter
    w = wv if which == 0 else wd
    hF, lg = o.forward(which, toks, add)
    rh, rl = torch_ref.forward(dm, w, wl.dtype, toks, add)
    scale = max(1.0, np.abs(rl).max())
    assert np.abs(hF - rh).max() < tol * max(1.0, np.abs(rh).max())
    assert np.abs(lg - rl).max() < tol * scale
    return lg


@pytest.mark.parametrize("which", [0, 1])
def test_forward_tiny_f32(which):
    toks = si.prompts(si.TINY)[0][0, :20]
    _check(si.TINY, which, toks)


@pytest.mark.parametrize("which", [0, 1])
def test_forward_gqa_bf16(which):
    toks = np.array([5, 17, 300, 2, 2, 511, 0, 44, 9], dtype=np.int32)
    _check(GQA, which, toks)


def test_forward_with_per_position_additive_input():
    """The steering injection adds a vector to each position's input embedding."""
    wl = GQA
    toks = np.array([1, 2, 3, 4, 5, 6], dtype=np.int32)
    rng = np.random.default_rng(0)
    add = rng.normal(0, 0.05, size=(len(toks), wl.drafter.d_model))
    _check(wl, 1, toks, add)


@pytest.mark.slow
def test_forward_small_bf16_verifier():
    """Full 12-layer d=768 verifier shape with a 32000 vocabulary."""
    toks = si.prompts(si.SMALL)[0][0, :12]
    _check(si.SMALL, 0, toks, tol=1e-8)
