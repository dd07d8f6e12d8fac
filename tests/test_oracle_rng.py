"""Pins of the oracle's random-number contract: Philox4x32-10, uniforms, Gumbel-max.

The sampler draws with a counter-based Philox4x32-10 (Salmon et al., SC'11).
Pins: the published known-answer vectors, an independent implementation (the
input generator's own copy, and the rocRAND header's, compiled on the host),
and the law of Gumbel-max draws (softmax).
"""
import math
import os
import shutil
import subprocess

import numpy as np
import pytest
from scipy import stats

import oracle
import sd2_inputs as si

HERE = os.path.dirname(os.path.abspath(__file__))


def _kat_rows():
    rows = []
    with open(os.path.join(HERE, "golden", "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            w = [int(x, 16) for x in line.split()]
            rows.append((w[0:4], w[4:6], w[6:10]))
    return rows


@pytest.mark.parametrize("row", _kat_rows())
def test_philox_known_answers(row):
    ctr, key, want = row
    assert list(oracle.philox(ctr, key)) == want


@pytest.mark.parametrize("row", _kat_rows())
def test_generator_philox_known_answers(row):
    ctr, key, want = row
    lib = si._load()
    c = np.array(ctr, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib.gen_philox_block(c.ctypes.data, key[0] | (key[1] << 32), out.ctypes.data)
    assert list(out) == want


def test_philox_matches_generator_copy_on_random_counters():
    rng = np.random.default_rng(1)
    lib = si._load()
    for _ in range(200):
        ctr = rng.integers(0, 2**32, size=4, dtype=np.uint64).astype(np.uint32)
        key = rng.integers(0, 2**32, size=2, dtype=np.uint64).astype(np.uint32)
        out = np.zeros(4, dtype=np.uint32)
        lib.gen_philox_block(ctr.ctypes.data, int(key[0]) | (int(key[1]) << 32), out.ctypes.data)
        assert list(oracle.philox(ctr, key)) == list(out)


_ROCRAND_SRC = r"""
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
#include <cstdlib>
// argv: seed subsequence offset_blocks  -> prints the 4 words of block (offset, subsequence) under key seed
int main(int argc, char** argv) {
  unsigned long long seed = strtoull(argv[1], 0, 0), sub = strtoull(argv[2], 0, 0), off = strtoull(argv[3], 0, 0);
  rocrand_state_philox4x32_10 st(seed, sub, off * 4ull);
  uint4 r = st.next4();
  printf("%u %u %u %u\n", r.x, r.y, r.z, r.w);
  return 0;
}
"""


def test_philox_matches_rocrand_header(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc) or not os.path.exists("/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"):
        pytest.skip("rocRAND headers / hipcc not available")
    src = tmp_path / "rr.hip"
    src.write_text(_ROCRAND_SRC)
    exe = tmp_path / "rr"
    subprocess.check_call([hipcc, "-O1", "--offload-arch=gfx950", str(src), "-o", str(exe)],
                          stderr=subprocess.DEVNULL)
    rng = np.random.default_rng(2)
    for _ in range(8):
        seed = int(rng.integers(0, 2**63))
        sub = int(rng.integers(0, 2**63))
        off = int(rng.integers(0, 2**61))
        out = subprocess.check_output([str(exe), str(seed), str(sub), str(off)]).split()
        want = [int(x) for x in out]
        ctr = [off & 0xFFFFFFFF, off >> 32, sub & 0xFFFFFFFF, sub >> 32]
        key = [seed & 0xFFFFFFFF, seed >> 32]
        assert list(oracle.philox(ctr, key)) == want


def test_uniform_range_and_exactness():
    for w in [0, 1, 255, 256, 0x7FFFFFFF, 0xFFFFFF00, 0xFFFFFFFF]:
        u = oracle.uniform(w)
        assert 0.0 < u < 1.0
        assert u == ((w >> 9) + 0.5) / 2**23
    assert oracle.uniform(0) == 2.0**-24
    assert oracle.uniform(0xFFFFFFFF) == 1.0 - 2.0**-24


def test_gumbel_values():
    for w in [0, 12345678, 0x80000000, 0xFFFFFFFF]:
        u = ((w >> 9) + 0.5) / 2**23
        want = -math.log(-math.log(u))
        assert abs(oracle.gumbel(w) - want) <= 1e-5 * max(1.0, abs(want))


def test_gumbel_max_law_is_softmax():
    """argmax(l/T + G) over vocabulary is distributed as softmax(l/T)."""
    V, T = 6, 0.7
    logits = np.array([0.3, -1.0, 1.2, 0.0, 0.9, -0.4], dtype=np.float32)
    N = 20000
    counts = np.zeros(V)
    for t in range(N):
        x, _ = oracle.pick(logits, T, seed=11, j=1, t=t, b=3)
        counts[x] += 1
    p = np.exp(logits / T) / np.exp(logits / T).sum()
    chi = stats.chisquare(counts, p * N)
    assert chi.pvalue > 1e-3, (counts / N, p)


def test_greedy_pick_ties_to_lowest_id():
    q = np.array([0.5, 2.0, -1.0, 2.0, 2.0], dtype=np.float32)
    x, margin = oracle.pick(q, 0.0, seed=0, j=1, t=5, b=0)
    assert x == 1 and margin == 0.0
