"""The training-objective forward (sd2_train_loss) against the oracle's, through the C ABI.

Tolerance, derived from the logit tolerance eps of the dtype (2e-2 bf16, 1e-4 f32): with
KL(p || q) = sum p (a - b) - lse(a) + lse(b) for verifier logits a and drafter logits b,
dKL/db = q - p (so an error of eps in b moves KL by at most 2 eps) and dKL/da_v = p_v (d_v - KL)
with d = log p - log q (at most eps * E_p|d - KL|, the spread the oracle reports).  Each target's
KL must lie within 1.5 eps (2 + spread) of the oracle's, plus fp32 summation over the vocabulary
(1e-5 relative); the mean within the mean of those bounds."""
import numpy as np
import pytest
import torch

import oracle
import sd2_inputs as si
from oracle_fixtures import GQA

pytestmark = pytest.mark.gpu

EPS = {"f32": 1e-4, "bf16": 2e-2}


def _check(wl, n, chunk, wv=None, wd=None, ws=None):
    from gpu_harness import device_model
    from paper_2511_09844_amd import binding as B
    if wv is None:
        wv, wd, ws = si.model_weights(wl, 0), si.model_weights(wl, 1), si.steer_weights(wl)
    toks, deltas = si.loss_inputs(wl, n)
    o = oracle.Oracle(wl, wv, wd, ws, cap=max(n, wl.max_seq_len))
    mean_o, kl_o, spread = o.train_loss(toks, deltas, spread=True)
    cfg = B.config_of(wl, max_seq_len=max(n, wl.max_seq_len))
    eng = B.Engine(cfg, device_model(wl, 0, wv), device_model(wl, 1, wd), B.to_device(ws))
    mean_g, kl_g = eng.train_loss(torch.from_numpy(toks).cuda(), torch.from_numpy(deltas).cuda(), chunk)
    eps = EPS[wl.dtype]
    tol = 1.5 * eps * (2.0 + spread[1:]) + 1e-5 * np.abs(kl_o[1:])
    err = np.abs(kl_g[1:] - kl_o[1:])
    print(f"[loss] {wl.name} n={n} chunk={chunk}: mean {mean_g:.6f} vs {mean_o:.6f}, max err {err.max():.3g}, "
          f"max err/tol {(err / tol).max():.3g}")
    assert kl_g[0] == 0.0
    assert (err <= tol).all(), np.argwhere(err > tol)
    assert abs(mean_g - mean_o) <= tol.mean()
    # the generation state is gone: a round needs a new prefill
    with pytest.raises(B.Sd2Error):
        eng.round()
    eng.close()
    return mean_o


def test_train_loss_several_chunks_ragged_tail():
    # 99 targets in chunks of 32 (the last holds 3): steering sources in earlier chunks
    _check(GQA, 100, 32)


def test_train_loss_one_chunk_f32():
    _check(si.TINY, 40, 512)


def test_train_loss_without_steering_matches_offsets_free_loss():
    # W_s = 0: both sides' loss, and the oracle's, cannot depend on the offsets
    wv, wd = si.model_weights(GQA, 0), si.model_weights(GQA, 1)
    ws = np.zeros_like(si.steer_weights(GQA))
    _check(GQA, 48, 16, wv, wd, ws)


@pytest.fixture(scope="module")
def host_8b():
    wl = si.LLAMA8B
    return si.model_weights(wl, 0), si.model_weights(wl, 1), si.steer_weights(wl)


def test_train_loss_8b_shapes(host_8b):
    # full 8B/1B model shapes and the 128256-token vocabulary; 23 targets in chunks of 8
    wv, wd, ws = host_8b
    _check(si.LLAMA8B, 24, 8, wv, wd, ws)
