"""Pins of the oracle's speculative round (drafting, verification, commit, steering).

What the paper fixes and these tests check:
  - block structure: a block returns the accepted drafts plus one final token,
    1 <= tau <= k+1 (Sec. "Metrics"), and generation stops at the token budget;
  - verification scores the block with the cached prefix, so every verifier
    row equals a from-scratch forward of the committed sequence (KV rollback and
    reuse are exact);
  - steering (Sec. "Drafting"): each drafter position keeps the steering vector
    that was active when it was processed; a zero W_s leaves the drafter
    unchanged (the paper's initialisation W_s = 0);
  - the steering tap is the verifier's final-norm hidden state at the position
    of the last token returned (Sec. "Verification");
  - greedy speculative decoding reproduces the verifier's own greedy decode.
"""
import numpy as np
import pytest

import oracle
import sd2_inputs as si
import torch_ref
from oracle_fixtures import GQA, weights, to_f64


def _run(wl, wv, wd, ws, max_rounds=1000, seqs=None, on_round=None):
    o = oracle.Oracle(wl, wv, wd, ws)
    toks, lens = si.prompts(wl)
    seqs = list(range(wl.batch)) if seqs is None else seqs
    o.prefill(toks, lens, seqs)
    outs = {b: [] for b in seqs}
    for r in range(max_rounds):
        live = [b for b in seqs if not o.state(b)["done"]]
        if not live:
            break
        for b in live:
            before = o.state(b)
            s_before = o.steer_vec(b)
            out, lg, dumps = o.round_one(b, dump=on_round is not None)
            outs[b].extend(out.tolist())
            if on_round:
                on_round(o, b, before, s_before, out, lg, dumps)
    return o, toks, lens, outs


def test_block_structure_and_budget():
    wl = GQA
    wv, wd, ws = weights(wl)
    seen = []

    def chk(o, b, before, s_before, out, lg, dumps):
        assert lg.active == 1
        assert 0 <= lg.n <= wl.k
        assert 1 <= len(out) <= lg.n + 1
        full = list(lg.drafts[: lg.n]) + [lg.y]
        assert list(out) == full[: len(out)]
        after = o.state(b)
        if not after["done"]:
            assert len(out) == lg.n + 1
            assert after["t"] == before["t"] + lg.n + 1
            assert after["len_v"] == before["t"] + lg.n
            assert after["len_d"] == min(before["t"] + wl.k - 1, before["t"] + lg.n)
            assert after["t"] - after["len_d"] in (1, 2)
        seen.append(lg.n)

    o, toks, lens, outs = _run(wl, wv, wd, ws, on_round=chk)
    for b in range(wl.batch):
        assert len(outs[b]) == wl.new_tokens
        assert o.state(b)["done"] == 1
        assert list(o.hist(b, lens[b] + wl.new_tokens)[lens[b]:]) == outs[b]
    assert len(set(seen)) > 1


def test_verifier_rows_equal_full_forward_and_torch():
    """KV reuse across rounds with rollback is exact: verifier rows == from-scratch forward."""
    wl = GQA
    wv, wd, ws = weights(wl)
    checks = []

    def chk(o, b, before, s_before, out, lg, dumps):
        t = before["t"]
        seq = list(o.hist(b, t)) + list(lg.drafts[: wl.k])
        _, ref = o.forward(0, np.array(seq, dtype=np.int32))
        want = ref[t - 1 : t + wl.k].astype(np.float32)
        assert np.array_equal(dumps["logits_v"], want)
        _, tref = torch_ref.forward(wl.verifier, wv, wl.dtype, seq)
        assert np.abs(dumps["logits_v"] - tref[t - 1 : t + wl.k]).max() < 1e-5
        checks.append(1)

    _run(wl, wv, wd, ws, on_round=chk, seqs=[0, 1])
    assert len(checks) > 4


def test_drafter_steering_bookkeeping_against_torch():
    """Drafter rows == a drafter forward whose inputs carry, per position, the steering of the round
    that (last) processed it; prompt positions carry none."""
    wl = GQA
    wv, wd, ws = weights(wl)
    b = 1
    toks, lens = si.prompts(wl)
    p = int(lens[b])
    add_of_pos = {i: np.zeros(wl.drafter.d_model) for i in range(p - 1)}
    checks = []

    def chk(o, bb, before, s_before, out, lg, dumps):
        t, ld = before["t"], before["len_d"]
        assert t - ld in (1, 2)
        # positions processed this round: ld .. t+k-2, all with this round's steering
        for pos in range(ld, t + wl.k - 1):
            add_of_pos[pos] = s_before.copy()
        seq = list(o.hist(bb, t)) + list(lg.drafts[: wl.k - 1])
        add = np.stack([add_of_pos[i] for i in range(len(seq))])
        _, ref = torch_ref.forward(wl.drafter, wd, wl.dtype, seq, add)
        assert np.abs(dumps["logits_d"] - ref[t - 1 : t + wl.k - 1]).max() < 1e-5
        # the next round starts from the committed cache length; drop stale entries
        after = o.state(bb)
        for pos in list(add_of_pos):
            if pos >= after["len_d"]:
                del add_of_pos[pos]
        checks.append(1)

    _run(wl, wv, wd, ws, on_round=chk, seqs=[b])
    assert len(checks) > 4


def test_steering_vector_is_projection_of_last_returned_position():
    wl = GQA
    wv, wd, ws = weights(wl)
    W = to_f64(ws, wl.dtype)
    toks, lens = si.prompts(wl)
    o = oracle.Oracle(wl, wv, wd, ws)
    o.prefill(toks, lens, [0])
    p = int(lens[0])
    # after prefill: tap at position p-2
    hF, _ = torch_ref.forward(wl.verifier, wv, wl.dtype, toks[0, : p - 1])
    assert np.abs(o.steer_vec(0) - W @ hF[p - 2]).max() < 1e-9
    for _ in range(4):
        out, lg, _ = o.round_one(0)
        t = o.state(0)["t"]
        hF, _ = torch_ref.forward(wl.verifier, wv, wl.dtype, o.hist(0, t - 1))
        assert np.abs(o.steer_vec(0) - W @ hF[t - 2]).max() < 1e-9


def test_zero_steering_leaves_drafter_unchanged():
    wl = GQA
    wv, wd, ws = weights(wl)
    zero = np.zeros_like(ws)
    checks = []

    def chk(o, b, before, s_before, out, lg, dumps):
        assert not s_before.any()
        t = before["t"]
        seq = np.array(list(o.hist(b, t)) + list(lg.drafts[: wl.k - 1]), dtype=np.int32)
        _, ref = o.forward(1, seq)  # no additive input at all
        assert np.array_equal(dumps["logits_d"], ref[t - 1 : t + wl.k - 1].astype(np.float32))
        checks.append(1)

    _run(wl, wv, wd, zero, on_round=chk, seqs=[0])
    assert len(checks) > 3


def test_self_drafting_accepts_every_draft():
    """Drafter == verifier and W_s = 0: p == q, so every draft is accepted (tau = k+1)."""
    wl = GQA.with_(drafter=GQA.verifier)
    wv = si.model_weights(wl, 0)
    zero = np.zeros((wl.drafter.d_model, wl.verifier.d_model), dtype=np.uint16)
    for T in (1.0, 0.0):
        o = oracle.Oracle(wl, wv, wv, zero, temperature=T)
        toks, lens = si.prompts(wl)
        o.prefill(toks, lens, [0])
        first = True
        while not o.state(0)["done"]:
            before = o.state(0)
            if not first:
                assert before["t"] - before["len_d"] == 2  # catch-up of two tokens after full acceptance
            out, lg, _ = o.round_one(0)
            if not o.state(0)["done"]:
                assert lg.n == wl.k and len(out) == wl.k + 1
            first = False


def test_greedy_matches_plain_verifier_greedy_decode():
    """At T = 0 the output is exactly the verifier's greedy continuation (argmax, ties to lowest id)."""
    wl = GQA.with_(temperature=0.0, new_tokens=40)
    wv, wd, ws = weights(wl)
    o, toks, lens, outs = _run(wl, wv, wd, ws)
    for b in range(wl.batch):
        p = int(lens[b])
        seq = np.array(list(toks[b, :p]) + outs[b], dtype=np.int32)
        _, lg = o.forward(0, seq[:-1])
        greedy = lg[p - 1 :].astype(np.float32).argmax(axis=1)
        assert list(greedy) == outs[b]


@pytest.mark.slow
def test_greedy_small_preset_matches_plain_decode():
    """Same invariant on the 12-layer bf16 preset shapes (shortened generation)."""
    wl = si.SMALL.with_(new_tokens=24)
    wv, wd, ws = weights(wl)
    o, toks, lens, outs = _run(wl, wv, wd, ws)
    p = int(lens[0])
    seq = np.array(list(toks[0, :p]) + outs[0], dtype=np.int32)
    _, lg = o.forward(0, seq[:-1])
    assert list(lg[p - 1 :].astype(np.float32).argmax(axis=1)) == outs[0]


def test_tiny_preset_runs_to_budget():
    wl = si.TINY
    wv, wd, ws = weights(wl)
    o, toks, lens, outs = _run(wl, wv, wd, ws)
    assert len(outs[0]) == wl.new_tokens
