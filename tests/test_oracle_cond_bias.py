"""Pins of the oracle's "Cond. bias in MLP" ablation.

The paper compares three steering mechanisms (Sec. "Ablation"): its own bias in
the MLP (eq. (2)), a bias after the MLP, and a bias in the MLP computed not from
g alone but also from the previous layer's output.  It gives no formula for the
last; the oracle reads it as a two-layer MLP per drafter layer l,
b = U_l SiLU(V_l [f; g]), f the residual stream entering layer l at the token's
own position and g the same LayerNorm(W_hml [h; m; l]) as eq. (2), added to the
up projection as in eq. (2).  The oracle evaluates V_l [f; g] as V_l^f f plus a
per-round V_l^g g.  Checked here against the PyTorch float64 reference, which
concatenates [f; g] and multiplies by the concatenated V_l:
  - one forward with a fixed g;
  - whole generations: the g part of every round comes from the verifier's taps
    at the last committed input, and the drafter logits equal a forward whose
    rows carry the g of the round that processed them (prompt rows: no bias);
  - U = 0 leaves the drafter unchanged bit for bit; greedy decoding still
    reproduces the verifier's greedy decode.
"""
import numpy as np
import pytest

import oracle
import sd2_inputs as si
import torch_ref
from sd2_inputs.configs import Dims, Workload

COND = Workload(
    name="cond-bias", verifier=Dims(4, 128, 4, 2, 256, 256, 5e5), drafter=Dims(2, 128, 4, 2, 192, 256, 5e5),
    dtype="bf16", k=3, batch=2, prompt=(5, 9), new_tokens=14, temperature=1.0, seed=23)
RANK = 32


def _oracle(wl, zero_u=False, scale=0.2, **kw):
    wv, wd = si.model_weights(wl, 0), si.model_weights(wl, 1)
    mlp = si.mlp_steer_weights(wl, form=3, rank=RANK, cond_scale=scale)
    if zero_u:
        mlp["w_cu"] = np.zeros_like(mlp["w_cu"])
    return oracle.Oracle(wl, wv, wd, None, mlp=mlp, **kw), wv, wd, mlp


def _c_of(mlp, g, wl):
    """V_l^g g of every layer, [L][R] (torch)."""
    import torch
    vg = torch_ref._t(mlp["w_s"], wl.dtype)
    return (vg @ torch.as_tensor(g, dtype=torch.float64)).numpy().reshape(wl.drafter.n_layers, RANK)


def _cond(mlp, g_rows, on):
    return {"vf": mlp["w_cf"], "vg": mlp["w_s"], "u": mlp["w_cu"], "rank": RANK, "g": g_rows, "on": on}


def test_cond_bias_forward_matches_torch():
    wl = COND
    o, _, wd, mlp = _oracle(wl)
    rng = np.random.default_rng(8)
    g = rng.normal(0, 1.0, wl.verifier.d_model)
    toks = np.array([7, 8, 9, 10, 11, 200], dtype=np.int32)
    _, lg = o.forward_cond(1, toks, _c_of(mlp, g, wl))
    _, ref = torch_ref.forward(wl.drafter, wd, wl.dtype, toks,
                               cond=_cond(mlp, np.tile(g, (len(toks), 1)), np.ones(len(toks))))
    _, plain = torch_ref.forward(wl.drafter, wd, wl.dtype, toks)
    assert np.abs(lg - ref).max() < 1e-9 * max(1.0, np.abs(ref).max())
    assert np.abs(ref - plain).max() > 1e-3  # the bias changes the logits


def test_cond_bias_g_part_comes_from_last_returned_position():
    wl = COND
    o, wv, _, mlp = _oracle(wl)
    toks, lens = si.prompts(wl)
    o.prefill(toks, lens, [1])

    def expect(seq):
        _, _, tp = torch_ref.forward(wl.verifier, wv, wl.dtype, seq, taps=True)
        return _c_of(mlp, torch_ref.steer_g(tp[-1], mlp, wl.dtype), wl)

    p = int(lens[1])
    ref = expect(toks[1, : p - 1])
    assert np.abs(o.ubias(1) - ref).max() < 1e-9 * np.abs(ref).max()
    for _ in range(4):
        o.round_one(1)
        t = o.state(1)["t"]
        ref = expect(o.hist(1, t - 1))
        assert np.abs(o.ubias(1) - ref).max() < 1e-9 * np.abs(ref).max()


def test_cond_bias_drafter_rows_against_torch():
    """Drafter logits of every round == a forward whose rows carry the g of the round that (last)
    processed them; prompt rows carry no bias."""
    wl = COND
    o, wv, wd, mlp = _oracle(wl)
    b = 0
    toks, lens = si.prompts(wl)
    o.prefill(toks, lens, [b])
    p = int(lens[b])
    dV = wl.verifier.d_model
    g_of_pos = {i: None for i in range(p - 1)}
    rounds = 0
    while not o.state(b)["done"]:
        before = o.state(b)
        t, ld = before["t"], before["len_d"]
        _, _, tp = torch_ref.forward(wl.verifier, wv, wl.dtype, o.hist(b, t - 1), taps=True)
        g = torch_ref.steer_g(tp[-1], mlp, wl.dtype)
        out, lg, dumps = o.round_one(b, dump=True)
        for pos in range(ld, t + wl.k - 1):
            g_of_pos[pos] = g
        seq = list(o.hist(b, t)) + list(lg.drafts[: wl.k - 1])
        rows = np.stack([g_of_pos[i] if g_of_pos[i] is not None else np.zeros(dV) for i in range(len(seq))])
        on = np.array([g_of_pos[i] is not None for i in range(len(seq))], dtype=np.float64)
        _, ref = torch_ref.forward(wl.drafter, wd, wl.dtype, seq, cond=_cond(mlp, rows, on))
        assert np.abs(dumps["logits_d"] - ref[t - 1 : t + wl.k - 1]).max() < 1e-5
        after = o.state(b)
        for pos in list(g_of_pos):
            if pos >= after["len_d"]:
                del g_of_pos[pos]
        rounds += 1
    assert rounds > 3


def test_zero_u_leaves_drafter_unchanged():
    wl = COND
    o, _, _, _ = _oracle(wl, zero_u=True)
    toks, lens = si.prompts(wl)
    o.prefill(toks, lens, [0])
    for _ in range(4):
        t = o.state(0)["t"]
        out, lg, dumps = o.round_one(0, dump=True)
        seq = np.array(list(o.hist(0, t)) + list(lg.drafts[: wl.k - 1]), dtype=np.int32)
        _, ref = o.forward(1, seq)
        assert np.array_equal(dumps["logits_d"], ref[t - 1 : t + wl.k - 1].astype(np.float32))


def test_greedy_with_cond_bias_matches_verifier_greedy_decode():
    wl = COND.with_(temperature=0.0, new_tokens=20)
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


def test_cond_form_needs_its_matrices():
    wl = COND
    wv, wd = si.model_weights(wl, 0), si.model_weights(wl, 1)
    mlp = si.mlp_steer_weights(wl, form=3, rank=RANK)
    mlp["rank"] = 0
    with pytest.raises(ValueError):
        oracle.Oracle(wl, wv, wd, None, mlp=mlp)
