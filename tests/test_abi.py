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


def test_struct_layouts_match_the_header(tmp_path):
    """The binding's ctypes structures have the header's sizes and field offsets (gcc on the host)."""
    prog = tmp_path / "layout.c"
    prog.write_text(
        '#include <stddef.h>\n#include <stdio.h>\n#include "sd2.h"\n'
        "int main(void) {\n"
        '  printf("%zu %zu %zu %zu\\n", sizeof(sd2_config), offsetof(sd2_config, seed),\n'
        "         offsetof(sd2_config, steering), offsetof(sd2_config, temperature));\n"
        '  printf("%zu %zu %zu\\n", sizeof(sd2_mlp_steering), offsetof(sd2_mlp_steering, ln_bias),\n'
        "         offsetof(sd2_mlp_steering, ln_eps));\n"
        '  printf("%zu %zu\\n", sizeof(sd2_weights), sizeof(sd2_dims));\n'
        "  return 0;\n}\n")
    exe = tmp_path / "layout"
    import subprocess
    subprocess.check_call(["gcc", "-I", os.path.join(ROOT, "include"), str(prog), "-o", str(exe)])
    got = [list(map(int, line.split())) for line in subprocess.check_output([str(exe)]).decode().splitlines()]
    C, M = B.Config, B.MlpSteering
    assert got[0] == [ctypes.sizeof(C), C.seed.offset, C.steering.offset, C.temperature.offset]
    assert got[1] == [ctypes.sizeof(M), M.ln_bias.offset, M.ln_eps.offset]
    assert got[2] == [ctypes.sizeof(B.Weights), ctypes.sizeof(B.Dims)]


def test_mlp_steering_configs():
    """The MLP form needs a verifier of at least 3 layers (block 3 is the low tap) and sizes its
    extra buffers; the unsteered form sizes none; an unknown steering form is rejected."""
    lib = B.load()
    for wl in si.PRESETS[:4]:
        base = lib.sd2_workspace_bytes(ctypes.byref(B.config_of(wl)))
        mlp = lib.sd2_workspace_bytes(ctypes.byref(B.config_of(wl, steering=B.STEER_MLP)))
        dm = wl.drafter
        assert mlp >= base + wl.batch * dm.n_layers * dm.d_ff * 4
    for wl in si.PRESETS[:4]:
        base = lib.sd2_workspace_bytes(ctypes.byref(B.config_of(wl)))
        after = lib.sd2_workspace_bytes(ctypes.byref(B.config_of(wl, steering=B.STEER_MLP_OUT)))
        assert after >= base + wl.batch * wl.drafter.d_model * 4
    for wl in si.PRESETS[:4]:
        # the unsteered drafter needs exactly the input form's workspace
        base = lib.sd2_workspace_bytes(ctypes.byref(B.config_of(wl)))
        assert lib.sd2_workspace_bytes(ctypes.byref(B.config_of(wl, steering=B.STEER_NONE))) == base
    c = B.config_of(si.TINY, steering=4)
    assert lib.sd2_workspace_bytes(ctypes.byref(c)) == 0
    c = B.config_of(si.TINY, steering=B.STEER_MLP)
    c.verifier.n_layers = 2
    assert lib.sd2_workspace_bytes(ctypes.byref(c)) == 0


def test_create_mlp_rejects_bad_arguments_without_gpu():
    lib = B.load()
    h = B.P()
    c = B.config_of(si.TINY, steering=B.STEER_MLP)
    assert lib.sd2_create_mlp(ctypes.byref(c), None, None, None, None, 0, None, ctypes.byref(h)) == -1
    # the input form's entry point refuses an MLP configuration, and the reverse
    assert lib.sd2_create(ctypes.byref(c), None, None, None, None, 0, None, ctypes.byref(h)) == -1
    ms = B.MlpSteering(None, None, None, None, 1e-5)
    c0 = B.config_of(si.TINY)
    assert lib.sd2_create_mlp(ctypes.byref(c0), None, None, ctypes.byref(ms), None, 0, None, ctypes.byref(h)) == -1


def test_create_noalloc_argument_errors_without_gpu():
    """Checked before any device call: a workspace larger than the static array, MLP forms."""
    lib = B.load()
    h = B.P()
    assert lib.sd2_workspace_bytes(ctypes.byref(B.config_of(si.LLAMA8B))) > (64 << 20)
    assert lib.sd2_create_noalloc(ctypes.byref(B.config_of(si.LLAMA8B)), None, None, None, None,
                                  ctypes.byref(h)) == -2
    c = B.config_of(si.TINY, steering=B.STEER_MLP)
    assert lib.sd2_create_noalloc(ctypes.byref(c), None, None, None, None, ctypes.byref(h)) == -1
    assert lib.sd2_create_noalloc(ctypes.byref(B.config_of(si.TINY)), None, None, None, None, None) == -1


def test_train_loss_scratch_sizes_without_gpu():
    """Scratch of the training-objective forward: the input form only, 2 <= n <= max_seq_len,
    1..512 rows per chunk; it grows with the chunk (two logit blocks of chunk x vocab floats)."""
    lib = B.load()
    c = B.config_of(si.GQA if hasattr(si, "GQA") else si.TINY)
    a = lib.sd2_train_loss_scratch_bytes(ctypes.byref(c), 20, 8)
    b = lib.sd2_train_loss_scratch_bytes(ctypes.byref(c), 20, 16)
    assert a > 0 and b - a >= 2 * 8 * c.verifier.vocab * 4
    assert lib.sd2_train_loss_scratch_bytes(ctypes.byref(c), 1, 8) == 0
    assert lib.sd2_train_loss_scratch_bytes(ctypes.byref(c), c.max_seq_len + 1, 8) == 0
    assert lib.sd2_train_loss_scratch_bytes(ctypes.byref(c), 20, 0) == 0
    assert lib.sd2_train_loss_scratch_bytes(ctypes.byref(c), 20, 513) == 0
    for form in (B.STEER_MLP, B.STEER_NONE):
        assert lib.sd2_train_loss_scratch_bytes(ctypes.byref(B.config_of(si.TINY, steering=form)), 20, 8) == 0
    assert lib.sd2_train_loss(None, None, None, 20, 8, None, None, None, 0) == -1
