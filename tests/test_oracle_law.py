"""Pins of the oracle's sampler against the law speculative sampling must have.

The paper verifies drafts by speculative rejection sampling (Sec.
"Verification", citing Leviathan et al. 2023 and Chen et al. 2023) and relies
on it preserving the verifier's distribution (Sec. "Metrics").  With a
vocabulary of 8 the law of one round's emitted block is enumerable:
  P(n accepted drafts a_1..a_n, final y) =
      prod_{i<=n} min(p_i(a_i), q_i(a_i)) * (p_{n+1}(y) - q_{n+1}(y))+   (n < k)
      prod_{i<=k} min(p_i(a_i), q_i(a_i)) * p_{k+1}(y)                    (n = k)
and "round, then continue with the verifier" must give the verifier's own law.
Monte-Carlo runs of the oracle's round are compared with that law (chi-square),
and the closed forms P(accept) = sum_v min(p, q) and, for identically
distributed positions, E[tau] = (1 - a^{k+1}) / (1 - a) are checked on
synthetic logit tables.
"""
import itertools

import numpy as np
import pytest
from scipy import stats

import oracle
import sd2_inputs as si
from oracle_fixtures import LAW, scaled_weights


def _softmax(x):
    e = np.exp(x - x.max())
    return e / e.sum()


@pytest.fixture(scope="module")
def law_setup():
    wl = LAW
    wv = scaled_weights(wl, 0, 0.6)
    wd = scaled_weights(wl, 1, 0.6)
    ws = si.normal((wl.drafter.d_model, wl.verifier.d_model), wl.dtype, wl.seed, si.tensor_id(2, 0, "w_s"), 0.6)
    o = oracle.Oracle(wl, wv, wd, ws)
    toks, lens = si.prompts(wl)
    prompt = toks[0, : lens[0]]
    o.prefill_one(0, prompt)
    s = o.steer_vec(0)
    p = len(prompt)
    V, k = wl.verifier.vocab, wl.k

    def pv(prefix_extra):
        seq = np.array(list(prompt) + list(prefix_extra), dtype=np.int32)
        return _softmax(o.forward(0, seq)[1][-1])

    def qd(prefix_extra):
        # the drafter sees prompt positions 0..p-2 unsteered and everything from p-1 on with s
        seq = np.array(list(prompt) + list(prefix_extra), dtype=np.int32)
        add = np.zeros((len(seq), wl.drafter.d_model))
        add[p - 1 :] = s
        return _softmax(o.forward(1, seq, add)[1][-1])

    P = {(): pv(())}
    Q = {(): qd(())}
    for depth in range(1, k + 1):
        for pre in itertools.product(range(V), repeat=depth):
            P[pre] = pv(pre)
            if depth < k:
                Q[pre] = qd(pre)
    return dict(wl=wl, o=o, prompt=prompt, P=P, Q=Q, V=V, k=k)


def _block_law(P, Q, V, k):
    """Exact law of the emitted block (tuple of 1..k+1 tokens)."""
    law = {}
    for n in range(k + 1):
        for acc in itertools.product(range(V), repeat=n):
            w = 1.0
            for i in range(n):
                w *= min(P[acc[:i]][acc[i]], Q[acc[:i]][acc[i]])
            if w == 0.0:
                continue
            if n < k:
                r = np.maximum(P[acc] - Q[acc], 0.0)
            else:
                r = P[acc]
            for y in range(V):
                if r[y] > 0:
                    law[acc + (y,)] = w * r[y]
    return law


def test_round_law_preserves_verifier_law(law_setup):
    P, Q, V, k = law_setup["P"], law_setup["Q"], law_setup["V"], law_setup["k"]
    law = _block_law(P, Q, V, k)
    assert abs(sum(law.values()) - 1.0) < 1e-12
    cont = {}
    for blk, w in law.items():
        rest = k + 1 - len(blk)
        for tail in itertools.product(range(V), repeat=rest):
            seq = blk + tail
            pr = w
            for i in range(len(blk), k + 1):
                pr *= P[seq[:i]][seq[i]]
            cont[seq] = cont.get(seq, 0.0) + pr
    for seq in itertools.product(range(V), repeat=k + 1):
        want = 1.0
        for i in range(k + 1):
            want *= P[seq[:i]][seq[i]]
        assert abs(cont.get(seq, 0.0) - want) < 1e-12


def test_oracle_round_samples_the_block_law(law_setup):
    o, prompt, P, Q, V, k = (law_setup[x] for x in ("o", "prompt", "P", "Q", "V", "k"))
    law = _block_law(P, Q, V, k)
    N = 30000
    counts = {}
    for seed in range(N):
        o.set_seed(seed * 7919 + 1)
        o.prefill_one(0, prompt)
        out, lg, _ = o.round_one(0)
        key = tuple(int(x) for x in out)
        assert len(key) == lg.n + 1
        counts[key] = counts.get(key, 0) + 1
    assert set(counts) <= set(law)
    keys = sorted(law, key=lambda x: -law[x])
    exp = np.array([law[x] * N for x in keys])
    obs = np.array([counts.get(x, 0) for x in keys], dtype=float)
    big = exp >= 5
    exp_p = np.append(exp[big], exp[~big].sum())
    obs_p = np.append(obs[big], obs[~big].sum())
    chi = stats.chisquare(obs_p, exp_p)
    assert chi.pvalue > 1e-3, chi
    # and the acceptance rate of the first draft matches sum_v min(p_1, q_1)
    acc1 = sum(c for kk, c in counts.items() if len(kk) >= 2) / N
    a = np.minimum(P[()], Q[()]).sum()
    assert abs(acc1 - a) < 4 * np.sqrt(a * (1 - a) / N)


def _table_round(pl, ql, T, seed, t):
    k = ql.shape[0]
    drafts = [oracle.pick(ql[j - 1], T, seed, j, t, 0)[0] for j in range(1, k + 1)]
    return drafts, oracle.accept_final(drafts, pl, ql, T, seed, t, 0)


def test_acceptance_closed_form_and_expected_block_length():
    """Identical rows: each draft is accepted independently w.p. a = sum min(p, q)."""
    rng = np.random.default_rng(5)
    V, k, T = 12, 4, 1.0
    lp = rng.normal(0, 1.0, V).astype(np.float32)
    lq = rng.normal(0, 1.0, V).astype(np.float32)
    pl = np.tile(lp, (k + 1, 1))
    ql = np.tile(lq, (k, 1))
    a = np.minimum(_softmax(lp.astype(np.float64)), _softmax(lq.astype(np.float64))).sum()
    N = 20000
    taus = np.array([_table_round(pl, ql, T, 99, t)[1].n + 1 for t in range(N)], dtype=float)
    want = (1 - a ** (k + 1)) / (1 - a)
    assert abs(taus.mean() - want) < 4 * taus.std() / np.sqrt(N)
    assert abs((taus >= 2).mean() - a) < 4 * np.sqrt(a * (1 - a) / N)


def test_final_token_law_after_rejection_and_after_full_acceptance():
    rng = np.random.default_rng(6)
    V, k, T = 6, 2, 0.8
    pl = rng.normal(0, 1.5, (k + 1, V)).astype(np.float32)
    ql = rng.normal(0, 1.5, (k, V)).astype(np.float32)
    p = np.array([_softmax(r.astype(np.float64) / T) for r in pl])
    q = np.array([_softmax(r.astype(np.float64) / T) for r in ql])
    N = 40000
    by_n = {n: np.zeros(V) for n in range(k + 1)}
    for t in range(N):
        _, lg = _table_round(pl, ql, T, 123, t)
        by_n[lg.n][lg.y] += 1
    for n in range(k + 1):
        want = p[n] if n == k else np.maximum(p[n] - q[n], 0)
        want = want / want.sum()
        c = by_n[n]
        if c.sum() < 200:
            continue
        m = want > 0
        assert c[~m].sum() == 0
        chi = stats.chisquare(c[m], want[m] * c.sum())
        assert chi.pvalue > 1e-3, (n, c / c.sum(), want)


def test_greedy_decisions():
    V, k = 5, 3
    pl = np.zeros((k + 1, V), dtype=np.float32)
    ql = np.zeros((k, V), dtype=np.float32)
    pl[0, 2] = pl[1, 4] = pl[2, 0] = pl[3, 1] = 1.0
    lg = oracle.accept_final([2, 4, 3], pl, ql, 0.0, 0, 10, 0)
    assert lg.n == 2 and lg.y == 0
    lg = oracle.accept_final([2, 4, 0], pl, ql, 0.0, 0, 10, 0)
    assert lg.n == 3 and lg.y == 1
    lg = oracle.accept_final([1, 4, 0], pl, ql, 0.0, 0, 10, 0)
    assert lg.n == 0 and lg.y == 2
