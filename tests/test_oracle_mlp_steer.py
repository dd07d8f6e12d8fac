"""Pins of the oracle's MLP steering (the paper's own form, eq. (2)).

What the paper fixes and these tests check:
  - the steering vector comes from three verifier activations, high, middle and
    low, taken after decoder blocks L-2, L/2 and 3 (training details), at the
    position of the last token returned (Sec. "Verification"), concatenated and
    mapped by W_hml, then passed through a LayerNorm (training details);
  - W_s g is one bias per drafter MLP layer, added to the up projection before
    the gating product (eq. (2)); it is computed once per drafting stage and
    every drafter token processed in that stage carries it, while positions
    keep the bias of the stage that processed them (Sec. "Drafting");
  - W_s = 0 (the paper's initialisation) leaves the drafter unchanged, and
    W_hml = [I I I] maps the three activations to their sum (initialisation);
  - greedy speculative decoding still reproduces the verifier's greedy decode;
  - the ablation "Inv. bias after MLP" (Sec. "Ablation"): the same g, and one bias
    W_s g added to the output of every drafter MLP.
Each check compares with the independent PyTorch float64 reference
(``torch_ref``: library LayerNorm, attention and SiLU) or with an invariant.
"""
import numpy as np
import pytest

import oracle
import sd2_inputs as si
import torch_ref
from sd2_inputs.configs import Dims, Workload

# Verifier of 8 layers: taps after blocks 6, 4 and 3 (all distinct); small drafter.
MLP8 = Workload(
    name="mlp-steer-8", verifier=Dims(8, 128, 4, 2, 256, 256, 5e5), drafter=Dims(2, 128, 4, 2, 192, 256, 5e5),
    dtype="bf16", k=3, batch=2, prompt=(5, 9), new_tokens=16, temperature=1.0, seed=21)


def _oracle(wl, hml="normal", ln="normal", zero_ws=False, form=1, **kw):
    wv, wd = si.model_weights(wl, 0), si.model_weights(wl, 1)
    mlp = si.mlp_steer_weights(wl, hml=hml, ln=ln, form=form)
    if zero_ws:
        mlp["w_s"] = np.zeros_like(mlp["w_s"])
    return oracle.Oracle(wl, wv, wd, None, mlp=mlp, **kw), wv, wd, mlp


@pytest.mark.parametrize("L", [8, 4, 3])
def test_taps_match_torch(L):
    """Residual stream after blocks L-2, L/2, 3 (from 1), in that order; blocks may coincide."""
    wl = MLP8.with_(verifier=Dims(L, 128, 4, 2, 256, 256, 5e5))
    o, wv, _, _ = _oracle(wl)
    toks = np.array([3, 200, 17, 5, 99, 250, 1], dtype=np.int32)
    hF, lg, tp = o.forward_mlp(0, toks, taps=True)
    rh, rl, rt = torch_ref.forward(wl.verifier, wv, wl.dtype, toks, taps=True)
    assert np.abs(tp - rt).max() < 1e-9 * max(1.0, np.abs(rt).max())
    assert np.abs(lg - rl).max() < 1e-9 * max(1.0, np.abs(rl).max())


def test_up_bias_forward_matches_torch():
    """eq. (2): W_d((W_u a + b) * SiLU(W_g a)), one bias per layer."""
    wl = MLP8
    o, _, wd, _ = _oracle(wl)
    rng = np.random.default_rng(4)
    ub = rng.normal(0, 0.5, size=(wl.drafter.n_layers, wl.drafter.d_ff))
    toks = np.array([7, 8, 9, 10, 11], dtype=np.int32)
    _, lg, _ = o.forward_mlp(1, toks, ubias=ub)
    _, rl = torch_ref.forward(wl.drafter, wd, wl.dtype, toks, ubias=ub)
    assert np.abs(lg - rl).max() < 1e-9 * max(1.0, np.abs(rl).max())
    # the bias changes the output (it is not dropped)
    _, plain = o.forward(1, toks)
    assert np.abs(lg - plain).max() > 1e-3


@pytest.mark.parametrize("hml,ln", [("normal", "normal"), ("identity", "unit"), ("identity", "normal")])
def test_mlp_steer_matches_torch(hml, ln):
    wl = MLP8
    o, _, _, mlp = _oracle(wl, hml=hml, ln=ln)
    rng = np.random.default_rng(5)
    z = rng.normal(0, 1.0, size=(3, wl.verifier.d_model))
    ub = o.mlp_steer(z)
    ref = torch_ref.mlp_steer(z, mlp, wl.dtype, wl.drafter.n_layers, wl.drafter.d_ff)
    assert np.abs(ub - ref).max() < 1e-10 * max(1.0, np.abs(ref).max())


def test_identity_hml_depends_on_the_sum_only():
    """W_hml = [I I I] gives g = h + m + l: any split of the same sum steers alike; the
    LayerNorm makes the result invariant to a positive scale of the activations."""
    wl = MLP8
    o, _, _, _ = _oracle(wl, hml="identity", ln="normal")
    rng = np.random.default_rng(6)
    z = rng.normal(0, 1.0, size=(3, wl.verifier.d_model))
    base = o.mlp_steer(z)
    moved = z.copy()
    moved[0] += 0.7 * z[2]
    moved[2] -= 0.7 * z[2]
    assert np.abs(o.mlp_steer(moved) - base).max() < 1e-9 * np.abs(base).max()
    assert np.abs(o.mlp_steer(z[::-1].copy()) - base).max() < 1e-9 * np.abs(base).max()
    # scale invariance holds up to the LayerNorm's eps: 1/sqrt(var + eps) moves by ~eps/(2 var)
    # relative (var ~ 3 here), well under 1e-5
    assert np.abs(o.mlp_steer(3.0 * z) - base).max() < 1e-5 * np.abs(base).max()


def test_bias_comes_from_last_returned_position():
    """After prefill: taps at position p-2; after each round: taps at the last committed input."""
    wl = MLP8
    o, wv, _, mlp = _oracle(wl)
    toks, lens = si.prompts(wl)
    o.prefill(toks, lens, [1])
    L, Fd = wl.drafter.n_layers, wl.drafter.d_ff

    def expect(seq):
        _, _, tp = torch_ref.forward(wl.verifier, wv, wl.dtype, seq, taps=True)
        return torch_ref.mlp_steer(tp[-1], mlp, wl.dtype, L, Fd)

    p = int(lens[1])
    ref = expect(toks[1, : p - 1])
    assert np.abs(o.ubias(1) - ref).max() < 1e-9 * np.abs(ref).max()
    for _ in range(4):
        o.round_one(1)
        t = o.state(1)["t"]
        ref = expect(o.hist(1, t - 1))
        assert np.abs(o.ubias(1) - ref).max() < 1e-9 * np.abs(ref).max()


def test_drafter_bias_bookkeeping_against_torch():
    """Drafter rows == a forward whose rows carry, per position, the bias of the round that
    (last) processed it; prompt positions carry none."""
    wl = MLP8
    o, _, wd, _ = _oracle(wl)
    b = 0
    toks, lens = si.prompts(wl)
    o.prefill(toks, lens, [b])
    p = int(lens[b])
    L, Fd = wl.drafter.n_layers, wl.drafter.d_ff
    bias_of_pos = {i: np.zeros((L, Fd)) for i in range(p - 1)}
    rounds = 0
    while not o.state(b)["done"]:
        before = o.state(b)
        ub = o.ubias(b)
        t, ld = before["t"], before["len_d"]
        out, lg, dumps = o.round_one(b, dump=True)
        for pos in range(ld, t + wl.k - 1):
            bias_of_pos[pos] = ub
        seq = list(o.hist(b, t)) + list(lg.drafts[: wl.k - 1])
        rows = np.stack([bias_of_pos[i] for i in range(len(seq))])
        _, ref = torch_ref.forward(wl.drafter, wd, wl.dtype, seq, ubias=rows)
        assert np.abs(dumps["logits_d"] - ref[t - 1 : t + wl.k - 1]).max() < 1e-5
        after = o.state(b)
        for pos in list(bias_of_pos):
            if pos >= after["len_d"]:
                del bias_of_pos[pos]
        rounds += 1
    assert rounds > 3


def test_zero_ws_leaves_drafter_unchanged():
    """The paper's initialisation W_s = 0: every bias is exactly zero, so the drafter's logits
    equal those of a forward without any steering, bit for bit."""
    wl = MLP8
    o, _, _, _ = _oracle(wl, zero_ws=True)
    toks, lens = si.prompts(wl)
    o.prefill(toks, lens, [0])
    for _ in range(4):
        assert not o.ubias(0).any()
        t = o.state(0)["t"]
        out, lg, dumps = o.round_one(0, dump=True)
        seq = np.array(list(o.hist(0, t)) + list(lg.drafts[: wl.k - 1]), dtype=np.int32)
        _, ref = o.forward(1, seq)
        assert np.array_equal(dumps["logits_d"], ref[t - 1 : t + wl.k - 1].astype(np.float32))


def test_greedy_with_mlp_steering_matches_verifier_greedy_decode():
    wl = MLP8.with_(temperature=0.0, new_tokens=24)
    o, _, _, _ = _oracle(wl)
    toks, lens = si.prompts(wl)
    o.prefill(toks, lens)
    outs = {b: [] for b in range(wl.batch)}
    while any(not o.state(b)["done"] for b in range(wl.batch)):
        for b in range(wl.batch):
            if not o.state(b)["done"]:
                outs[b].extend(o.round_one(b)[0].tolist())
    for b in range(wl.batch):
        p = int(lens[b])
        seq = np.array(list(toks[b, :p]) + outs[b], dtype=np.int32)
        _, lg = o.forward(0, seq[:-1])
        assert list(lg[p - 1 :].astype(np.float32).argmax(axis=1)) == outs[b]


def test_single_token_prompt_has_no_bias():
    wl = MLP8.with_(prompt=(1, 1), batch=1)
    o, _, _, _ = _oracle(wl)
    toks, lens = si.prompts(wl)
    o.prefill(toks, lens)
    assert not o.ubias(0).any()


def test_two_layer_verifier_is_rejected():
    """Block 3 must exist for the low tap."""
    wl = MLP8.with_(verifier=Dims(2, 128, 4, 2, 256, 256, 5e5))
    with pytest.raises(ValueError):
        _oracle(wl)


def test_bias_after_mlp_forward_matches_torch():
    wl = MLP8
    o, _, wd, _ = _oracle(wl, form=2)
    rng = np.random.default_rng(7)
    ob = rng.normal(0, 0.3, size=(wl.drafter.d_model,))
    toks = np.array([7, 8, 9, 10, 11], dtype=np.int32)
    _, lg, _ = o.forward_mlp(1, toks, obias=ob)
    _, rl = torch_ref.forward(wl.drafter, wd, wl.dtype, toks, obias=ob)
    assert np.abs(lg - rl).max() < 1e-9 * max(1.0, np.abs(rl).max())
    _, plain = o.forward(1, toks)
    assert np.abs(lg - plain).max() > 1e-3


def test_bias_after_mlp_round_against_torch():
    """Form 2 over whole generations: the bias after each round is W_s LayerNorm(W_hml [h; m; l])
    of the last committed input, and every drafter row carries the bias of the round that
    processed it (a forward with per-position biases after every MLP)."""
    wl = MLP8
    o, wv, wd, mlp = _oracle(wl, form=2)
    b = 1
    toks, lens = si.prompts(wl)
    o.prefill(toks, lens, [b])
    p = int(lens[b])
    dD = wl.drafter.d_model
    bias_of_pos = {i: np.zeros(dD) for i in range(p - 1)}
    rounds = 0
    while not o.state(b)["done"]:
        before = o.state(b)
        ob = o.ubias(b)
        t, ld = before["t"], before["len_d"]
        _, _, tp = torch_ref.forward(wl.verifier, wv, wl.dtype, o.hist(b, t - 1), taps=True)
        ref_b = torch_ref.mlp_steer(tp[-1], mlp, wl.dtype, wl.drafter.n_layers, wl.drafter.d_ff)
        assert ob.shape == (dD,) and np.abs(ob - ref_b).max() < 1e-9 * np.abs(ref_b).max()
        out, lg, dumps = o.round_one(b, dump=True)
        for pos in range(ld, t + wl.k - 1):
            bias_of_pos[pos] = ob
        seq = list(o.hist(b, t)) + list(lg.drafts[: wl.k - 1])
        rows = np.stack([bias_of_pos[i] for i in range(len(seq))])
        _, ref = torch_ref.forward(wl.drafter, wd, wl.dtype, seq, obias=rows)
        assert np.abs(dumps["logits_d"] - ref[t - 1 : t + wl.k - 1]).max() < 1e-5
        for pos in list(bias_of_pos):
            if pos >= o.state(b)["len_d"]:
                del bias_of_pos[pos]
        rounds += 1
    assert rounds > 3


def test_bias_after_mlp_greedy_matches_verifier_greedy_decode():
    wl = MLP8.with_(temperature=0.0, new_tokens=20)
    o, _, _, _ = _oracle(wl, form=2)
    toks, lens = si.prompts(wl)
    o.prefill(toks, lens)
    outs = {b: [] for b in range(wl.batch)}
    while any(not o.state(b)["done"] for b in range(wl.batch)):
        for b in range(wl.batch):
            if not o.state(b)["done"]:
                outs[b].extend(o.round_one(b)[0].tolist())
    for b in range(wl.batch):
        p = int(lens[b])
        seq = np.array(list(toks[b, :p]) + outs[b], dtype=np.int32)
        _, lg = o.forward(0, seq[:-1])
        assert list(lg[p - 1 :].astype(np.float32).argmax(axis=1)) == outs[b]
