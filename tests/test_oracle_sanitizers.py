"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

tests/sanitize_oracle.c drives oracle.c through every entry point a parity run uses (create,
prefill of two ragged prompts, rounds to completion, whole-sequence forward, training-objective
forward) for float32 and bf16 weights and all four steering forms.  Both are compiled with gcc's
address and undefined-behaviour sanitizers (no recovery, leak checking on) and the driver must
exit cleanly.  A planted one-past-the-end read and a planted signed overflow show that each
sanitizer is live here, so that a clean run means something.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
FLAGS = ["-std=c11", "-g", "-O1", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
         "-fno-omit-frame-pointer"]

# one planted mistake per sanitizer, each built with that sanitizer alone
PLANTED = {
    "address": (r"""
#include <stdlib.h>
int main(void) {
    volatile int* p = calloc(4, sizeof(int));
    int s = 0;
    for (int i = 0; i <= 4; ++i) s += p[i];
    free((void*)p);
    return s == 12345;
}
""", "heap-buffer-overflow"),
    "undefined": (r"""
#include <limits.h>
int main(int argc, char** argv) {
    (void)argv;
    volatile int x = INT_MAX - 1 + argc;
    volatile int y = x + 1;
    return y == 0;
}
""", "signed integer overflow"),
}


def _build(out, sources, flags=FLAGS):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not found")
    res = subprocess.run([gcc, *flags, "-o", out, *sources, "-lm"], capture_output=True, text=True, timeout=300)
    if res.returncode != 0:
        pytest.skip("gcc cannot build with the sanitizers here: " + res.stderr[-400:])


@pytest.fixture(scope="module")
def workdir(tmp_path_factory):
    d = tmp_path_factory.mktemp("sanitize")
    for name, (code, _) in PLANTED.items():
        (d / f"planted_{name}.c").write_text(code)
        flags = ["-std=c11", "-g", "-O0", f"-fsanitize={name}", "-fno-sanitize-recover=all"]
        _build(str(d / f"planted_{name}"), [str(d / f"planted_{name}.c")], flags)
    return d


@pytest.mark.parametrize("name", sorted(PLANTED))
def test_planted_mistake_is_reported(workdir, name):
    res = subprocess.run([str(workdir / f"planted_{name}")], capture_output=True, text=True, timeout=60)
    assert res.returncode != 0 and PLANTED[name][1] in res.stderr, res.stderr[-1000:]


def test_oracle_is_clean_under_asan_and_ubsan(workdir):
    exe = str(workdir / "oracle_driver")
    _build(exe, [os.path.join(HERE, "sanitize_oracle.c"), os.path.join(ROOT, "oracle", "oracle.c")])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    res = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert res.returncode == 0, res.stderr[-3000:]
    assert "runtime error" not in res.stderr and "ERROR:" not in res.stderr, res.stderr[-3000:]
    assert "8 configurations clean" in res.stdout
