"""Host logic of bench.py (no GPU): the round byte model against an explicit enumeration of
what one round streams, the kernel-trace summaries on a synthetic trace whose durations are
known, and the refusal of more than one GPU."""
import csv
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import sd2_inputs as si  # noqa: E402


def _matrices(dm):
    """Every weight matrix one forward streams, as (rows, cols): per layer Q, K, V, O, gate,
    up, down, then the LM head (the embedding table is gathered by row, the norm gains are
    vectors)."""
    hd = dm.d_model // dm.n_heads
    out = []
    for _ in range(dm.n_layers):
        out += [(dm.n_heads * hd, dm.d_model), (dm.n_kv_heads * hd, dm.d_model), (dm.n_kv_heads * hd, dm.d_model),
                (dm.d_model, dm.n_heads * hd), (dm.d_ff, dm.d_model), (dm.d_ff, dm.d_model), (dm.d_model, dm.d_ff)]
    out.append((dm.vocab, dm.d_model))
    return out


@pytest.mark.parametrize("wl", [si.TINY, si.LLAMA8B, si.LLAMA70B], ids=lambda w: w.name)
def test_round_bytes_equal_an_enumeration_of_the_round(wl):
    es = 2 if wl.dtype == "bf16" else 4
    k, t = wl.k, 600
    w, kv_v, kv_d = bench.round_bytes(wl, t)
    # weights: the verifier once, the drafter once per step, W_s [d_D][d_V] once
    want_w = sum(r * c for r, c in _matrices(wl.verifier)) * es
    want_w += k * sum(r * c for r, c in _matrices(wl.drafter)) * es
    want_w += wl.drafter.d_model * wl.verifier.d_model * es
    assert w == want_w

    def row(dm):  # K and V of one position over all layers, fp32
        return dm.n_layers * dm.n_kv_heads * (dm.d_model // dm.n_heads) * 2 * 4

    # verify pass: reads every position up to the block's last (t + k) and appends the k + 1 rows
    assert kv_v == (t + k + (k + 1)) * row(wl.verifier)
    # drafter step j reads positions [0, t + j); step 0 appends two rows, the others one
    reads = sum(t + j for j in range(k))
    appends = 2 + (k - 1)
    assert kv_d == (reads + appends) * row(wl.drafter)


def test_llama8b_verifier_weights_match_the_published_parameter_count():
    # Llama-3-8B has 8,030,261,248 parameters; without the 128256 x 4096 embedding table and the
    # 2 x 32 + 1 norm gains of 4096 the projections and the LM head are the rest
    dm = si.LLAMA8B.verifier
    params = 8_030_261_248 - 128256 * 4096 - (2 * 32 + 1) * 4096
    assert bench.weight_bytes(dm, 2) == 2 * params


def _write_trace(path, rounds):
    """A kernel trace of `rounds` per-operation rounds (k = 2 drafter steps) between two
    prefill kernels; durations in ns chosen so every stage total is distinct."""
    rows, t = [], 1000

    def add(name, dur):
        nonlocal t
        rows.append({"Kernel_Name": f"void sd2::{name}(sd2::Args)", "Start_Timestamp": t, "End_Timestamp": t + dur})
        t += dur + 100

    add("k_pgemm<1>", 50_000)  # prefill
    for _ in range(rounds):
        add("k_set_flag", 1_000)
        for step in range(2):
            add("k_wsgemv<4, 4, 1>", 10_000 if step == 0 else 20_000)
            add("k_attn<64, 8>", 3_000)
            add("k_pick_partial", 500)
            add("k_pick_final", 400)
        add("k_pgemm<1>", 70_000)
        add("k_pattn_pk<128>", 30_000)
        add("k_row_partial", 2_000)
        add("k_accept", 4_000)
        add("k_commit", 600)
    add("k_pgemm<2>", 80_000)  # another prefill
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        w.writerows(rows)


def test_summarize_stages_splits_the_round(tmp_path, capsys):
    p = str(tmp_path / "k_kernel_trace.csv")
    _write_trace(p, rounds=3)
    bench.summarize_stages(p, 2)
    out = capsys.readouterr().out
    assert out.splitlines()[0] == "3 rounds"
    lines = {l.split(":")[0]: l for l in out.splitlines() if "ms/round" in l and not l.startswith(" ")}
    # step 1: set flag 1.0 + projection 10 + attention 3 + picks 0.9 us; step 2: 20 + 3 + 0.9;
    # verify: 70 + 30; accept and commit: 2 + 4 + 0.6
    assert lines["drafter step 1"].endswith("0.015 ms/round")
    assert lines["drafter steps 2-2"].endswith("0.024 ms/round")
    assert lines["verify pass"].endswith("0.100 ms/round")
    assert lines["accept, commit"].endswith("0.007 ms/round")


def test_summarize_trace_keeps_prefill_apart(tmp_path, capsys):
    p = str(tmp_path / "k_kernel_trace.csv")
    _write_trace(p, rounds=4)
    bench.summarize_trace(p)
    out = capsys.readouterr().out
    first = out.splitlines()[0]
    # per round: 1 + 2 * (3 + 0.9) + 10 + 20 + 70 + 30 + 2 + 4 + 0.6 = 145.4 us
    assert first.startswith("4 rounds in the trace") and first.endswith("0.145 ms/round")
    outside = [l for l in out.splitlines() if l.startswith("kernels outside rounds")][0]
    assert outside.endswith("0.13 ms")  # the two prefill kernels, 50 + 80 us


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
