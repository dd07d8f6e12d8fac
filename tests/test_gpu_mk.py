"""Persistent-launch round path (one launch per drafter step and per verify pass) against the
CPU oracle on small shapes that path takes, and the one-kernel-per-operation path on the same."""
import pytest

from oracle_fixtures import G8LONG, MK1, MK2, MK3, MK4, MK5, MK6, RAG16, RAG16_LONGEST, RAG16_SHORTEST

pytestmark = pytest.mark.gpu


def _run(wl, **kw):
    from gpu_harness import parity_run
    st = parity_run(wl, **kw)
    assert st.pinned > 0
    return st


def test_mk_one_layer_separate_kernels():
    _run(MK1, expect_path=0, separate_kernels=True)


def test_mk_one_layer_persistent():
    _run(MK1, expect_path=1)


def test_mk_two_layers_two_sequences_persistent():
    _run(MK2, expect_path=1)


def test_mk_split_k_persistent():
    _run(MK3, expect_path=1)


def test_mk_long_ragged_contexts_persistent():
    _run(MK4, expect_path=1)


def test_mk_long_ragged_contexts_separate_kernels():
    _run(MK4, expect_path=0, separate_kernels=True)


def test_mk_more_attention_units_than_workgroups():
    # 288 verifier attention units on 256 workgroups: the second unit of a workgroup waits for its
    # KV head's counter and loads all of its span after the phase has started
    _run(MK5, expect_path=1)


def test_mk_hd128_long_contexts_persistent():
    # verify pass at head dim 128 over 629 and 1114 cached positions: span partials of every live
    # span, the last-arriver fold with a second batch of 16 spans (18 live spans)
    _run(MK6, expect_path=1)


def test_mk_hd128_long_contexts_separate_kernels():
    # the per-operation attention at head dim 128: 5 and 9 spans of 128 merged by the last arriver
    _run(MK6, expect_path=0, separate_kernels=True)


def test_ragged_sixteen_long_prompts_per_operation():
    # the batched workload's structure: 16 prompts from 257 to 1992 tokens, k = 7, T = 0.7, 128
    # verify rows per round (many-row MFMA GEMM, ragged attention); the oracle follows the
    # shortest and the longest sequence, the library runs all sixteen
    _run(RAG16, expect_path=0, seqs=[RAG16_SHORTEST, RAG16_LONGEST])


def test_unsteered_drafter_persistent():
    # SD2_STEER_NONE (no steering projection, nothing added) equals the oracle with W_s = 0
    _run(MK2, expect_path=1, unsteered=True)


def test_unsteered_drafter_separate_kernels():
    _run(MK2, expect_path=0, separate_kernels=True, unsteered=True)


def test_gqa8_nine_rows_long_contexts_per_operation():
    # the 70B shape's verify attention (8 query heads per KV head, 9 rows) over several key spans
    _run(G8LONG, expect_path=0)
