"""The non-finite flag (SD2_DBG_NONFINITE): every verifier and drafter logit a round's decisions
use is checked as the sampler reads it.

A clean model never raises it; one NaN planted in the verifier's LM head (one weight of one
vocabulary row, so every verifier logit row holds a NaN) raises it in the first round.  Reading
the flag clears it, and the next round raises it again.  Per-operation path (f32, sampled and
greedy) and persistent path (bf16).  A NaN changes no control flow on the GPU: every round is the
same fixed sequence of kernels, so the poisoned rounds end like the clean ones."""
import numpy as np
import pytest
import torch

import sd2_inputs as si
from oracle_fixtures import MK2

pytestmark = pytest.mark.gpu


def _engine(wl, poison):
    from gpu_harness import device_model
    from paper_2511_09844_amd import binding as B
    wv, wd, ws = si.model_weights(wl, 0), si.model_weights(wl, 1), si.steer_weights(wl)
    if poison:
        lm = wv["lm_head"].copy()
        lm[5, 3] = 0x7FC0 if lm.dtype == np.uint16 else np.nan  # bf16 or f32 quiet NaN
        wv = dict(wv, lm_head=lm)
    eng = B.Engine(B.config_of(wl), device_model(wl, 0, wv), device_model(wl, 1, wd), B.to_device(ws))
    toks, lens = si.prompts(wl)
    eng.prefill(torch.from_numpy(toks).cuda(), torch.from_numpy(lens).cuda(), wl.max_prompt)
    return eng


@pytest.mark.parametrize("wl, path", [(si.TINY.with_(new_tokens=16), 0),
                                      (si.TINY.with_(new_tokens=16, temperature=0.0), 0),
                                      (MK2, 1)], ids=["f32-sampled", "f32-greedy", "bf16-persistent"])
def test_nonfinite_flag(wl, path):
    from paper_2511_09844_amd import binding as B
    clean = _engine(wl, poison=False)
    assert int(clean.debug(B.DBG_PATH)[0]) == path
    for _ in range(3):
        clean.round()
    assert int(clean.debug(B.DBG_NONFINITE)[0]) == 0
    clean.close()

    bad = _engine(wl, poison=True)
    assert int(bad.debug(B.DBG_NONFINITE)[0]) == 0  # nothing sampled yet
    bad.round()
    assert int(bad.debug(B.DBG_NONFINITE)[0]) == 1
    assert int(bad.debug(B.DBG_NONFINITE)[0]) == 0  # the read cleared it
    if not all(s["done"] for s in bad.state()):
        bad.round()
        assert int(bad.debug(B.DBG_NONFINITE)[0]) == 1
    assert int(bad.debug(B.DBG_PATH)[1]) == 0  # no persistent launch timed out
    bad.close()
