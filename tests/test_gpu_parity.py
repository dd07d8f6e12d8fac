"""GPU round vs the CPU oracle, through the C ABI, on seeded synthetic workloads."""
import pytest

import sd2_inputs as si
from oracle_fixtures import GQA

pytestmark = pytest.mark.gpu


def _run(wl, **kw):
    from gpu_harness import parity_run
    st = parity_run(wl, **kw)
    assert st.pinned > 0
    return st


def test_parity_tiny_f32():
    """Tiny fp32 preset end to end (tolerance 1e-4)."""
    _run(si.TINY)


def test_parity_gqa_bf16_batched_ragged():
    """Grouped-query bf16 models, two sequences with different prompt lengths."""
    _run(GQA)


def test_parity_gqa_greedy():
    _run(GQA.with_(temperature=0.0, new_tokens=30))


def test_parity_small_bf16_greedy():
    """12-layer d=768 verifier / 4-layer d=512 drafter, vocab 32000, greedy, 128 new tokens."""
    _run(si.SMALL)
