"""Shared GPU-vs-oracle parity driver for the `gpu` tests and the smoke check.

The oracle runs free on the CPU (its own Philox draws); the GPU library runs the
same rounds with the oracle's decisions forced (sd2_round_forced), records its
own decisions, and every comparison uses identical inputs:
  - integer decisions (drafts, accepted count, final token) must match exactly
    wherever the oracle's decision margin exceeds MARGIN;
  - logits and steering vectors must match within the dtype's tolerance;
  - emitted tokens, counts and cache lengths must match exactly.
"""
import os

import numpy as np
import torch

import oracle
import sd2_inputs as si
from paper_2511_09844_amd import binding as B

MARGIN = 1e-2
TOL = {"f32": 1e-4, "bf16": 2e-2}


def device_model(wl, which, host=None):
    if host is not None:
        items = [(("embed",), host["embed"])]
        for l, layer in enumerate(host["layers"]):
            for n, t in zip(si.LAYER_TENSORS, layer):
                items.append((("layers", l, n), t))
        items += [(("final_norm",), host["final_norm"]), (("lm_head",), host["lm_head"])]
        return B.DeviceModel(items)
    return B.DeviceModel(si.iter_model_tensors(wl, which))


class Stats:
    def __init__(self):
        self.decisions = 0
        self.pinned = 0
        self.unpinned = 0
        self.max_err_v = 0.0
        self.max_err_d = 0.0
        self.max_err_s = 0.0
        self.rounds = 0
        self.tokens = 0

    def __repr__(self):
        return (f"rounds={self.rounds} tokens={self.tokens} decisions={self.decisions} pinned={self.pinned} "
                f"unpinned={self.unpinned} err_logits_v={self.max_err_v:.3g} err_logits_d={self.max_err_d:.3g} "
                f"err_steer={self.max_err_s:.3g}")


def parity_run(wl, wv=None, wd=None, ws=None, seqs=None, max_rounds=10**6, check_logits=True, log=print,
               expect_path=None, separate_kernels=False, mlp=None, unsteered=False):
    """Run prefill + rounds on both sides; assert parity; return Stats.

    expect_path: 0 (one kernel per operation) or 1 (one persistent launch per drafter step and
    verify pass) -- the execution path the library must have chosen; separate_kernels forces 0.
    mlp: host weights of the MLP steering form (sd2_inputs.mlp_steer_weights); the per-layer
    up-projection biases are then compared where the steering vector is otherwise.
    unsteered: the library runs the unsteered drafter (SD2_STEER_NONE), the oracle W_s = 0."""
    if wv is None:
        wv, wd, ws = si.model_weights(wl, 0), si.model_weights(wl, 1), si.steer_weights(wl)
    if unsteered:
        ws = np.zeros_like(ws)
    tol = TOL[wl.dtype]
    toks, lens = si.prompts(wl)
    seqs = list(range(wl.batch)) if seqs is None else list(seqs)
    o = oracle.Oracle(wl, wv, wd, ws, mlp=mlp)
    o.prefill(toks, lens, seqs)
    dv, dd = device_model(wl, 0, wv), device_model(wl, 1, wd)
    if unsteered:
        ws_dev = None
        eng = B.Engine(B.config_of(wl, steering=B.STEER_NONE), dv, dd, None)
    elif mlp is None:
        ws_dev = B.to_device(ws)
        eng = B.Engine(B.config_of(wl), dv, dd, ws_dev)
    else:
        keys = ("w_s", "w_hml", "ln_gain", "ln_bias") + (("w_cf", "w_cu") if int(mlp.get("form", 1)) == 3 else ())
        ws_dev = {key: B.to_device(mlp[key]) for key in keys}
        ws_dev["ln_eps"] = mlp["ln_eps"]
        form = {1: B.STEER_MLP, 2: B.STEER_MLP_OUT, 3: B.STEER_MLP_COND}[int(mlp.get("form", 1))]
        eng = B.Engine(B.config_of(wl, steering=form, cond_rank=int(mlp.get("rank", 0))), dv, dd, None, mlp=ws_dev)

    def steer_err(b, dev):
        # the steering state of sequence b: s (input form) or the per-layer biases (MLP form)
        ref = o.steer_vec(b) if mlp is None else o.ubias(b)
        return float(np.abs(dev[b] - ref).max())

    dbg_steer = B.DBG_STEER if mlp is None else B.DBG_UBIAS
    old = os.environ.pop("SD2_NO_MK", None)
    if separate_kernels:
        os.environ["SD2_NO_MK"] = "1"
    try:
        eng.prefill(torch.from_numpy(toks).cuda(), torch.from_numpy(lens).cuda(), wl.max_prompt)
    finally:
        os.environ.pop("SD2_NO_MK", None)
        if old is not None:
            os.environ["SD2_NO_MK"] = old
    path = int(eng.debug(B.DBG_PATH)[0])
    log(f"[parity] {wl.name}: execution path {path}")
    if expect_path is not None:
        assert path == expect_path, f"execution path {path}, expected {expect_path}"
    st = Stats()
    s_gpu = eng.debug(dbg_steer)
    for b in seqs:
        err = steer_err(b, s_gpu)
        st.max_err_s = max(st.max_err_s, err)
        assert err <= tol, f"prefill steering b={b} err={err}"
    k = wl.k
    for r in range(max_rounds):
        live = [b for b in seqs if not o.state(b)["done"]]
        if not live:
            break
        forced = np.zeros((wl.batch, k + 2), dtype=np.int32)
        logs, outs, dumps = {}, {}, {}
        for b in live:
            out, lg, dm = o.round_one(b, dump=check_logits)
            logs[b], outs[b], dumps[b] = lg, out, dm
            forced[b, :k] = lg.drafts[:k]
            forced[b, k] = lg.n
            forced[b, k + 1] = lg.y
        ot, oc = eng.round(torch.from_numpy(forced).cuda())
        ot, oc = ot.cpu().numpy(), oc.cpu().numpy()
        own_d = eng.debug(B.DBG_OWN_DRAFTS)
        own_n = eng.debug(B.DBG_OWN_N)
        own_y = eng.debug(B.DBG_OWN_Y)
        if check_logits:
            lv = eng.debug(B.DBG_LOGITS_V)
            ld = eng.debug(B.DBG_LOGITS_D)
        sg = eng.debug(dbg_steer)
        state = eng.state()
        for b in live:
            lg = logs[b]
            where = f"round {r} seq {b}"
            # emitted tokens and counts follow the forced (oracle) trajectory exactly
            assert oc[b] == lg.count, f"{where}: count {oc[b]} vs {lg.count}"
            assert list(ot[b, : lg.count]) == list(outs[b]), f"{where}: tokens"
            ost = o.state(b)
            for key in ("t", "len_v", "len_d", "produced", "done"):
                assert state[b][key] == ost[key], f"{where}: state {key} {state[b][key]} vs {ost[key]}"
            # continuous outputs
            if check_logits:
                ev = float(np.abs(lv[b] - dumps[b]["logits_v"]).max())
                ed = float(np.abs(ld[b] - dumps[b]["logits_d"]).max())
                st.max_err_v = max(st.max_err_v, ev)
                st.max_err_d = max(st.max_err_d, ed)
                assert ev <= tol and ed <= tol, f"{where}: logits err v={ev} d={ed}"
            es = steer_err(b, sg)
            st.max_err_s = max(st.max_err_s, es)
            assert es <= tol, f"{where}: steering err {es}"
            # the library's own decisions, where the oracle's margin pins them
            for j in range(k):
                st.decisions += 1
                if lg.draft_margin[j] > MARGIN:
                    st.pinned += 1
                    assert own_d[b, j] == lg.drafts[j], f"{where}: draft {j} {own_d[b, j]} vs {lg.drafts[j]}"
                else:
                    st.unpinned += 1
            tested = range(min(lg.n + 1, k))
            st.decisions += 1
            if all(lg.accept_margin[i] > MARGIN for i in tested):
                st.pinned += 1
                assert own_n[b] == lg.n, f"{where}: n {own_n[b]} vs {lg.n}"
            else:
                st.unpinned += 1
            st.decisions += 1
            if lg.final_margin > MARGIN:
                st.pinned += 1
                assert own_y[b] == lg.y, f"{where}: y {own_y[b]} vs {lg.y}"
            else:
                st.unpinned += 1
            st.tokens += int(lg.count)
        st.rounds += 1
    for b in seqs:
        assert o.state(b)["done"] == 1
    assert int(eng.debug(B.DBG_PATH)[1]) == 0, "a persistent launch timed out at a grid barrier"
    eng.close()
    del eng, dv, dd, ws_dev
    torch.cuda.empty_cache()
    log(f"[parity] {wl.name}: {st}")
    return st


def free_run(wl, wv=None, wd=None, ws=None, seqs=None, expect_path=None, separate_kernels=False, min_rounds=3,
             log=print):
    """Both sides run free: the library's own sd2_round (no forced decisions, the path the
    benchmark times) against the oracle's own rounds on the same seeded inputs.

    A sequence is compared round by round -- emitted tokens, counts, cache lengths exactly;
    logits and steering vector within the dtype's tolerance -- until its first round in which
    some decision the oracle took has a margin of at most MARGIN.  From there the two
    trajectories may legitimately differ, so that sequence is followed no further.  Returns
    (rounds compared per sequence, Stats)."""
    if wv is None:
        wv, wd, ws = si.model_weights(wl, 0), si.model_weights(wl, 1), si.steer_weights(wl)
    tol = TOL[wl.dtype]
    toks, lens = si.prompts(wl)
    seqs = list(range(wl.batch)) if seqs is None else list(seqs)
    o = oracle.Oracle(wl, wv, wd, ws)
    o.prefill(toks, lens, seqs)
    dv, dd = device_model(wl, 0, wv), device_model(wl, 1, wd)
    ws_dev = B.to_device(ws)
    eng = B.Engine(B.config_of(wl), dv, dd, ws_dev)
    old = os.environ.pop("SD2_NO_MK", None)
    if separate_kernels:
        os.environ["SD2_NO_MK"] = "1"
    try:
        eng.prefill(torch.from_numpy(toks).cuda(), torch.from_numpy(lens).cuda(), wl.max_prompt)
    finally:
        os.environ.pop("SD2_NO_MK", None)
        if old is not None:
            os.environ["SD2_NO_MK"] = old
    path = int(eng.debug(B.DBG_PATH)[0])
    log(f"[free] {wl.name}: execution path {path}")
    if expect_path is not None:
        assert path == expect_path, f"execution path {path}, expected {expect_path}"
    st = Stats()
    compared = {b: 0 for b in seqs}
    following = set(seqs)
    k = wl.k
    while following:
        live = [b for b in following if not o.state(b)["done"]]
        if not live:
            break
        outs, logs, dumps = {}, {}, {}
        for b in live:
            outs[b], logs[b], dumps[b] = o.round_one(b, dump=True)
        ot, oc = eng.round()
        ot, oc = ot.cpu().numpy(), oc.cpu().numpy()
        lv, ld = eng.debug(B.DBG_LOGITS_V), eng.debug(B.DBG_LOGITS_D)
        sg = eng.debug(B.DBG_STEER)
        state = eng.state()
        for b in live:
            lg = logs[b]
            margins = list(lg.draft_margin[:k]) + [lg.final_margin]
            margins += [lg.accept_margin[i] for i in range(min(lg.n + 1, k))]
            st.decisions += len(margins)
            if min(margins) <= MARGIN:
                # a near-tie: the library may take the other branch from here on
                st.unpinned += 1
                following.discard(b)
                continue
            st.pinned += len(margins)
            where = f"free round {compared[b]} seq {b}"
            assert oc[b] == lg.count, f"{where}: count {oc[b]} vs {lg.count}"
            assert list(ot[b, : lg.count]) == list(outs[b]), f"{where}: tokens {ot[b, :lg.count]} vs {outs[b]}"
            ost = o.state(b)
            for key in ("t", "len_v", "len_d", "produced", "done"):
                assert state[b][key] == ost[key], f"{where}: state {key} {state[b][key]} vs {ost[key]}"
            ev = float(np.abs(lv[b] - dumps[b]["logits_v"]).max())
            ed = float(np.abs(ld[b] - dumps[b]["logits_d"]).max())
            es = float(np.abs(sg[b] - o.steer_vec(b)).max())
            st.max_err_v, st.max_err_d, st.max_err_s = max(st.max_err_v, ev), max(st.max_err_d, ed), max(st.max_err_s, es)
            assert ev <= tol and ed <= tol and es <= tol, f"{where}: errors v={ev} d={ed} s={es}"
            compared[b] += 1
            st.tokens += int(lg.count)
        st.rounds += 1
    assert int(eng.debug(B.DBG_PATH)[1]) == 0, "a persistent launch timed out at a grid barrier"
    eng.close()
    del eng, dv, dd, ws_dev
    torch.cuda.empty_cache()
    log(f"[free] {wl.name}: compared rounds {compared} {st}")
    # how far the comparison reaches is a property of the oracle's own trajectory (where its first
    # near-tie falls), fixed by the seed; the tests choose inputs that reach several rounds
    assert sum(compared.values()) >= min_rounds, f"only {compared} rounds compared before near-ties"
    return compared, st
