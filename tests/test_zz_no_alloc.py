"""sd2_create_noalloc (the library's static device workspace) against sd2_create (the caller's
workspace) on the same inputs: two handles in a row on one GPU, the second with a smaller
workload, each run through prefill and whole generations side by side with a regular handle.

Both handles run the same kernels on the same inputs, so the comparison is exact: emitted tokens,
counts and per-sequence state bit for bit, logits and steering vectors equal.  The second handle
reuses the static array the first one filled, so it also checks that creation clears it."""
import ctypes

import numpy as np
import pytest
import torch

import sd2_inputs as si
from oracle_fixtures import MK2

pytestmark = pytest.mark.gpu


def _models(wl):
    from gpu_harness import device_model
    from paper_2511_09844_amd import binding as B
    wv, wd, ws = si.model_weights(wl, 0), si.model_weights(wl, 1), si.steer_weights(wl)
    return device_model(wl, 0, wv), device_model(wl, 1, wd), B.to_device(ws)


def _side_by_side(wl, max_rounds=200):
    from paper_2511_09844_amd import binding as B
    dv, dd, ws = _models(wl)
    cfg = B.config_of(wl)
    ref = B.Engine(cfg, dv, dd, ws)
    nal = B.Engine(cfg, dv, dd, ws, noalloc=True)
    assert nal.workspace is None
    toks, lens = si.prompts(wl)
    t_tok, t_len = torch.from_numpy(toks).cuda(), torch.from_numpy(lens).cuda()
    ref.prefill(t_tok, t_len, wl.max_prompt)
    nal.prefill(t_tok, t_len, wl.max_prompt)
    assert np.array_equal(ref.debug(B.DBG_STEER), nal.debug(B.DBG_STEER))
    rounds = 0
    while not all(s["done"] for s in ref.state()):
        a_tok, a_cnt = (x.cpu().numpy().copy() for x in ref.round())
        b_tok, b_cnt = (x.cpu().numpy().copy() for x in nal.round())
        assert np.array_equal(a_cnt, b_cnt), f"round {rounds}: counts {a_cnt} vs {b_cnt}"
        for b in range(wl.batch):
            assert np.array_equal(a_tok[b, : a_cnt[b]], b_tok[b, : b_cnt[b]]), f"round {rounds} seq {b}"
        assert ref.state() == nal.state()
        for what in (B.DBG_LOGITS_V, B.DBG_LOGITS_D, B.DBG_STEER):
            assert np.array_equal(ref.debug(what), nal.debug(what)), f"round {rounds}: debug {what}"
        rounds += 1
        assert rounds < max_rounds
    assert all(s["done"] for s in nal.state())
    path = int(nal.debug(B.DBG_PATH)[0])
    ref.close()
    nal.close()
    return rounds, path


def test_noalloc_matches_caller_workspace_twice_second_smaller():
    r1, p1 = _side_by_side(MK2)                               # 19.9 MiB, persistent path, 2 sequences
    r2, p2 = _side_by_side(si.TINY.with_(new_tokens=16))      # 6.1 MiB, f32, per-operation path
    assert r1 > 0 and r2 > 0 and p1 == 1 and p2 == 0


def test_noalloc_one_live_handle_per_device_and_size_limit():
    from paper_2511_09844_amd import binding as B
    wl = si.TINY.with_(new_tokens=4)
    dv, dd, ws = _models(wl)
    cfg = B.config_of(wl)
    first = B.Engine(cfg, dv, dd, ws, noalloc=True)
    lib = B.load()
    h = B.P()
    rc = lib.sd2_create_noalloc(ctypes.byref(cfg), ctypes.byref(dv.w), ctypes.byref(dd.w), ws.data_ptr(),
                                torch.cuda.current_stream().cuda_stream, ctypes.byref(h))
    assert rc == -3 and not h.value  # SD2_ERR_STATE while the first one is alive
    first.close()
    big = B.config_of(si.LLAMA8B)
    rc = lib.sd2_create_noalloc(ctypes.byref(big), ctypes.byref(dv.w), ctypes.byref(dd.w), ws.data_ptr(),
                                torch.cuda.current_stream().cuda_stream, ctypes.byref(h))
    assert rc == -2  # SD2_ERR_CAPACITY: the 8B workspace exceeds the static array
    again = B.Engine(cfg, dv, dd, ws, noalloc=True)  # the slot is free again after destroy
    again.close()
