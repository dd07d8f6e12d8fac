"""Pins of the oracle's training-objective forward (Sec. "Training").

The paper trains the steering with a uniformly random offset delta in [1, k]: the drafter's
prediction of a token, steered by the g extracted delta positions earlier, is pulled towards
the verifier's distribution by the KL divergence.  The oracle's reading (input-form steering):
target x_tau with offset delta uses s = W_s hF_V(tau - delta - 1), the steering a round that
starts at tau - delta + 1 would use (zero before the sequence start), and in the one-pass
forward every drafter input position carries the steering of the target it predicts.

Checked against:
  - a PyTorch float64 forward of both models (library attention, SiLU) with the KL divergence
    from ``torch.nn.functional.kl_div`` on log-softmax rows;
  - drafter == verifier with W_s = 0: the loss is exactly zero;
  - W_s = 0: the loss does not depend on the offsets, bit for bit;
  - the KL divergence is never negative.

The spread E_pV|d - KL| (d = log p_V - log p_D), which scales the GPU parity tolerance, is checked
against the same PyTorch rows and is zero for self-drafting.
"""
import numpy as np
import torch
import torch.nn.functional as F

import oracle
import sd2_inputs as si
import torch_ref
from sd2_inputs.configs import Dims, Workload

LOSS = Workload(
    name="train-loss", verifier=Dims(2, 128, 4, 2, 256, 256, 5e5), drafter=Dims(2, 64, 4, 2, 128, 256, 5e5),
    dtype="bf16", k=4, batch=1, prompt=(8, 8), new_tokens=8, temperature=1.0, seed=31)


def _setup(wl, ws_scale=0.3, same_models=False):
    wv = si.model_weights(wl, 0)
    wd = wv if same_models else si.model_weights(wl, 1)
    ws = si.normal((wl.drafter.d_model, wl.verifier.d_model), wl.dtype, wl.seed, si.tensor_id(2, 0, "w_s"), ws_scale)
    if ws_scale == 0:
        ws = np.zeros_like(ws)
    return oracle.Oracle(wl, wv, wd, ws, cap=64), wv, wd, ws


def _torch_loss(wl, wv, wd, ws, toks, deltas):
    n = len(toks)
    hF, lv = torch_ref.forward(wl.verifier, wv, wl.dtype, toks[:-1])
    W = torch_ref._t(ws, wl.dtype)
    add = np.zeros((n - 1, wl.drafter.d_model))
    for p in range(n - 1):
        q = p - int(deltas[p + 1])
        if q >= 0:
            add[p] = (W @ torch.as_tensor(hF[q])).numpy()
    _, ld = torch_ref.forward(wl.drafter, wd, wl.dtype, toks[:-1], add=add)
    lp, lq = F.log_softmax(torch.as_tensor(lv), -1), F.log_softmax(torch.as_tensor(ld), -1)
    kl = F.kl_div(lq, lp, reduction="none", log_target=True).sum(-1)
    spread = (lp.exp() * (lp - lq - kl[:, None]).abs()).sum(-1)
    return kl.numpy(), spread.numpy()


def test_loss_matches_torch_kl_div():
    wl = LOSS
    o, wv, wd, ws = _setup(wl)
    toks, deltas = si.loss_inputs(wl, 24)
    assert deltas[1:].min() >= 1 and deltas[1:].max() <= wl.k and len(set(deltas[1:])) == wl.k
    mean, kl, spread = o.train_loss(toks, deltas, spread=True)
    ref, ref_spread = _torch_loss(wl, wv, wd, ws, toks, deltas)
    assert kl[0] == 0.0
    assert np.abs(kl[1:] - ref).max() < 1e-9 * max(1.0, ref.max())
    assert abs(mean - ref.mean()) < 1e-9 * max(1.0, ref.mean())
    assert ref_spread.min() > 0
    assert np.abs(spread[1:] - ref_spread).max() < 1e-9 * max(1.0, ref_spread.max())


def test_self_drafting_without_steering_has_zero_loss():
    wl = LOSS.with_(drafter=LOSS.verifier)
    o, _, _, _ = _setup(wl, ws_scale=0, same_models=True)
    toks, deltas = si.loss_inputs(wl, 20)
    mean, kl, spread = o.train_loss(toks, deltas, spread=True)
    assert mean == 0.0 and not kl.any() and not spread.any()


def test_zero_steering_makes_the_loss_independent_of_offsets():
    wl = LOSS
    o, _, _, _ = _setup(wl, ws_scale=0)
    toks, deltas = si.loss_inputs(wl, 20)
    m1, k1 = o.train_loss(toks, deltas)
    m2, k2 = o.train_loss(toks, np.ones_like(deltas))
    assert m1 == m2 and np.array_equal(k1, k2)
    o2, _, _, _ = _setup(wl)
    m3, _ = o2.train_loss(toks, deltas)
    m4, _ = o2.train_loss(toks, np.ones_like(deltas))
    assert m3 != m4  # with steering, the offsets matter


def test_kl_is_never_negative():
    wl = LOSS
    o, _, _, _ = _setup(wl, ws_scale=1.0)
    for stream in range(3):
        toks, deltas = si.loss_inputs(wl, 16, stream=stream)
        _, kl = o.train_loss(toks, deltas)
        assert kl.min() >= -1e-12
