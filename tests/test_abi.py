"""Host-side checks of the C ABI: the library loads, exports every declared entry point,
and rejects bad arguments before touching the GPU."""
import ctypes
import os
import re

import pytest

import sd2_inputs as si
from paper_2511_09844_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "sd2.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(sd2_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    lib = B.load()
    names = declared_functions()
    assert set(names) == set(B.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def test_workspace_bytes_and_invalid_configs():
    lib = B.load()
    for wl in si.PRESETS[:4]:
        c = B.config_of(wl)
        assert lib.sd2_workspace_bytes(ctypes.byref(c)) > 0
    bad = [
        dict(k=0), dict(k=33), dict(max_batch=0), dict(max_seq_len=3), dict(max_new_tokens=0),
        dict(temperature=-1.0),
    ]
    for kw in bad:
        c = B.config_of(si.TINY, **kw)
        assert lib.sd2_workspace_bytes(ctypes.byref(c)) == 0, kw
    c = B.config_of(si.TINY)
    c.drafter.vocab = 999
    assert lib.sd2_workspace_bytes(ctypes.byref(c)) == 0
    c = B.config_of(si.TINY)
    c.verifier.n_kv_heads = 3
    assert lib.sd2_workspace_bytes(ctypes.byref(c)) == 0


def test_create_rejects_bad_arguments_without_gpu():
    lib = B.load()
    c = B.config_of(si.TINY)
    h = B.P()
    assert lib.sd2_create(ctypes.byref(c), None, None, None, None, 0, None, ctypes.byref(h)) == -1
    assert lib.sd2_create(None, None, None, None, None, 0, None, None) == -1
    # null handle calls
    assert lib.sd2_prefill(None, 1, None, None, 1) == -1
    assert lib.sd2_round(None, None, None) == -1
    assert lib.sd2_round_forced(None, None, None, None) == -1
    assert lib.sd2_debug_read(None, 1, None, 0) == -1
    assert lib.sd2_destroy(None) == 0


def test_status_strings():
    lib = B.load()
    for code in (0, -1, -2, -3, -4, -5, 7):
        assert lib.sd2_status_string(code)
