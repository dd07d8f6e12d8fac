"""Persistent-launch round path (one launch per drafter step and per verify pass) against the
CPU oracle on small shapes that path takes, and the one-kernel-per-operation path on the same."""
import pytest

from oracle_fixtures import MK1, MK2, MK3, MK4, MK5

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
