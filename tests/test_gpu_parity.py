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


@pytest.fixture(scope="module")
def host_8b():
    """Host weights of the 8B-shaped verifier / 1B-shaped drafter (generated once, ~19 GB)."""
    wl = si.LLAMA8B
    return si.model_weights(wl, 0), si.model_weights(wl, 1), si.steer_weights(wl)


def test_parity_8b_shapes_short_prompt(host_8b):
    """Full 8B/1B model dimensions (32 x d4096 GQA verifier, 16 x d2048 drafter, 128256 vocab),
    sampling at T=1, k=5, batch 1; a 16-token prompt keeps the float64 oracle within seconds.
    Rounds run as persistent launches (one per drafter step, one per verify pass)."""
    wl = si.LLAMA8B.with_(prompt=(16, 16), new_tokens=10)
    wv, wd, ws = host_8b
    _run(wl, wv=wv, wd=wd, ws=ws, expect_path=1)


def test_parity_8b_shapes_separate_kernels(host_8b):
    """The same workload with one kernel per operation (the path used where the persistent
    launches do not apply)."""
    wl = si.LLAMA8B.with_(prompt=(16, 16), new_tokens=10)
    wv, wd, ws = host_8b
    _run(wl, wv=wv, wd=wd, ws=ws, expect_path=0, separate_kernels=True)


def test_parity_8b_shapes_two_ragged_sequences(host_8b):
    """Two sequences with different prompt lengths (k=2: 6 verifier rows per pass) on the
    persistent launches: per-sequence positions, catch-up rows and finished sequences inside one
    launch."""
    wl = si.LLAMA8B.with_(batch=2, k=2, prompt=(9, 21), new_tokens=9)
    wv, wd, ws = host_8b
    _run(wl, wv=wv, wd=wd, ws=ws, expect_path=1)


def test_parity_8b_batched_ragged_sampled_sequences(host_8b):
    """Batched configuration (16 sequences, ragged prompts, k=7, T=0.7): the GPU runs all 16
    sequences; the oracle follows two of them, which must match exactly as if run alone."""
    wl = si.LLAMA8B_BATCHED.with_(prompt=(6, 30), new_tokens=5)
    wv, wd, ws = host_8b
    _run(wl, wv=wv, wd=wd, ws=ws, seqs=[0, 11])


def test_parity_70b_width_two_layers():
    """The 70B shape's verifier layer width (d 8192, 64 query / 8 KV heads, F 28672: down
    projection K beyond 16384, split into K ranges) on two layers, with the 1B-shaped drafter,
    k = 8, batch 2 (18 verifier rows: the many-row GEMM and the per-operation path)."""
    from sd2_inputs.configs import Dims
    wl = si.LLAMA70B.with_(verifier=Dims(2, 8192, 64, 8, 28672, 128256, 5e5), batch=2, prompt=(7, 12),
                           new_tokens=9)
    _run(wl)
