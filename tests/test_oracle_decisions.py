"""Pins of the oracle's decision margins and of its empty-residual fallback.

The parity harness enforces a GPU decision only where the oracle's margin for it
exceeds 1e-2, so the margins decide what is checked.  They are pinned here on
known tables, each against a definition computed independently of oracle.c:

  - greedy picks (T = 0): the margin is the gap between the largest and the
    second-largest logit (exact closed forms on hand-written rows; ties give 0
    and the lowest id);
  - Gumbel-max picks (T > 0): raising the winner's logit by d*T raises the
    margin by d, and lowering it by more than margin*T hands the pick to the
    runner-up; so the margin is the gap of the perturbed scores l/T + G;
  - accept tests: the margin is |log u_i - (log p_i(x) - log q_i(x))|, with
    log p and log q from scipy's log-softmax and u_i the Philox uniform of the
    accept purpose (both pinned elsewhere); the decision must be log u < ratio.

The fallback (a rejected draft whose residual (p - q)+ has no positive entry in
float32) is mathematically impossible and numerically reachable only when p and
q agree on every other token to the last bit.  The oracle then draws the final
token from p_{n+1} with the same Gumbel noise as the bonus draw (speculative
sampling as the paper cites it, Sec. "Verification"; the reading for the
numerically empty residual is the library's own).
"""
import numpy as np
import pytest
from scipy.special import log_softmax

import oracle

PURPOSE_ACCEPT = 2


def _logu(seed, i, t, b):
    w = oracle.philox([i, 0, t, (PURPOSE_ACCEPT << 24) | b], [seed & 0xFFFFFFFF, seed >> 32])[0]
    return float(np.log(np.float32(oracle.uniform(int(w)))))


@pytest.mark.parametrize("row, best, gap", [
    ([0.1, 0.5, 0.3], 1, 0.2),
    ([-1.0, -2.0, 3.25, 3.0], 2, 0.25),
    ([7.0, -7.0], 0, 14.0),
    ([-3.0, -1.5, -1.5, -4.0], 1, 0.0),      # tie: lowest id, zero margin
    ([2.0, 2.0, 2.0], 0, 0.0),
])
def test_greedy_margin_is_top1_minus_top2(row, best, gap):
    x, m = oracle.pick(np.array(row, dtype=np.float32), 0.0, seed=0, j=1, t=3, b=0)
    assert x == best
    assert m == pytest.approx(np.float32(gap), abs=1e-6)


def test_greedy_margin_single_entry_vocabulary():
    x, m = oracle.pick(np.array([0.5], dtype=np.float32), 0.0, seed=0, j=1, t=3, b=0)
    assert x == 0 and m == np.inf


def test_greedy_accept_margins_are_verifier_top2_gaps():
    V, k = 6, 2
    pl = np.zeros((k + 1, V), dtype=np.float32)
    ql = np.zeros((k, V), dtype=np.float32)
    pl[0] = [0.0, 1.0, 0.75, 0.0, 0.0, 0.0]     # argmax 1, gap 0.25
    pl[1] = [0.0, 0.0, 0.0, -1.0, 2.5, 0.5]     # argmax 4, gap 2.0
    pl[2] = [3.0, 0.0, 0.0, 0.0, 0.0, 2.0]      # argmax 0, gap 1.0
    lg = oracle.accept_final([1, 4], pl, ql, 0.0, 0, 5, 0)
    assert lg.n == 2 and lg.y == 0
    assert lg.accept_margin[0] == pytest.approx(0.25, abs=1e-6)
    assert lg.accept_margin[1] == pytest.approx(2.0, abs=1e-6)
    assert lg.final_margin == pytest.approx(1.0, abs=1e-6)


@pytest.mark.parametrize("T", [1.0, 0.7])
def test_gumbel_margin_is_the_perturbed_score_gap(T):
    rng = np.random.default_rng(21)
    V = 40
    for trial in range(30):
        q = rng.normal(0, 1.0, V).astype(np.float32)
        x, m = oracle.pick(q, T, seed=5, j=2, t=100 + trial, b=1)
        assert m >= 0
        # raising the winner's logit by d*T raises its perturbed score, and so the margin, by d
        q2 = q.copy()
        q2[x] += np.float32(0.5 * T)
        x2, m2 = oracle.pick(q2, T, seed=5, j=2, t=100 + trial, b=1)
        assert x2 == x and m2 == pytest.approx(m + 0.5, abs=2e-5)
        # lowering it by more than margin*T hands the pick to another token
        q3 = q.copy()
        q3[x] -= np.float32((m + 0.05) * T)
        x3, m3 = oracle.pick(q3, T, seed=5, j=2, t=100 + trial, b=1)
        assert x3 != x
        # the old winner now trails the old runner-up by 0.05 (a third token may be closer)
        assert m3 <= 0.05 + 2e-5
        # lowering it by less keeps it, with the margin reduced by the same amount
        if m > 0.1:
            q4 = q.copy()
            q4[x] -= np.float32((m - 0.05) * T)
            x4, m4 = oracle.pick(q4, T, seed=5, j=2, t=100 + trial, b=1)
            assert x4 == x and m4 == pytest.approx(0.05, abs=2e-5)


@pytest.mark.parametrize("T", [1.0, 0.7])
def test_accept_margin_is_distance_of_log_u_from_log_ratio(T):
    rng = np.random.default_rng(22)
    V, k, seed = 16, 4, 77
    seen = {True: 0, False: 0}
    for t in range(200):
        pl = rng.normal(0, 1.5, (k + 1, V)).astype(np.float32)
        ql = rng.normal(0, 1.5, (k, V)).astype(np.float32)
        drafts = rng.integers(0, V, k).astype(np.int32)
        lg = oracle.accept_final(drafts, pl, ql, T, seed, t, 3)
        logp = log_softmax(pl.astype(np.float64) / T, axis=1)
        logq = log_softmax(ql.astype(np.float64) / T, axis=1)
        for i in range(min(lg.n + 1, k)):
            ratio = logp[i, drafts[i]] - logq[i, drafts[i]]
            logu = _logu(seed, i, t, 3)
            assert lg.accept_margin[i] == pytest.approx(abs(logu - ratio), abs=2e-5)
            accepted = i < lg.n
            seen[accepted] += 1
            # where the margin is clear, the decision is log u < ratio
            if abs(logu - ratio) > 1e-4:
                assert accepted == (logu < ratio), (t, i, logu, ratio)
    assert seen[True] > 50 and seen[False] > 50


def test_empty_residual_falls_back_to_verifier_row():
    """Rejected draft, residual numerically empty: the final token is p_{n+1}'s Gumbel-max draw.

    The tables agree on every token but x, where the verifier's logit is 20 below the drafter's:
    the acceptance ratio is about e^-20, below the smallest uniform (2^-24), so x is always
    rejected; p and q then round to the same float32 value on every other token, and (p - q)+
    has no positive entry.  The same row drawn as the bonus token (all drafts accepted, same
    round start t and sequence) must give the same token: both use the final-token noise."""
    V, T, seed = 64, 1.0, 9
    x = 17
    base = np.zeros(V, dtype=np.float32)
    base[:8] = np.linspace(2.0, 4.0, 8, dtype=np.float32)
    lp, lq = base.copy(), base.copy()
    lq[x] = -60.0
    lp[x] = -80.0
    hits = 0
    for t in range(40):
        a = oracle.accept_final([x], np.stack([lp, base]), lq[None, :], T, seed, t, 2)
        assert a.n == 0 and a.used_fallback == 1
        # bonus draw from the same row: draft accepted with certainty (p == q), n = k = 1
        bonus = oracle.accept_final([0], np.stack([base, lp]), base[None, :], T, seed, t, 2)
        assert bonus.n == 1 and bonus.used_fallback == 0
        assert a.y == bonus.y and a.y != x
        assert a.final_margin == pytest.approx(bonus.final_margin, abs=1e-6)
        hits += a.y < 8
    # the draw follows p: the eight raised logits hold about 78 % of its mass
    assert hits >= 22


def test_nonempty_residual_never_uses_fallback_and_never_draws_where_p_le_q():
    rng = np.random.default_rng(23)
    V, k, T = 10, 2, 1.0
    for t in range(300):
        pl = rng.normal(0, 1.0, (k + 1, V)).astype(np.float32)
        ql = rng.normal(0, 1.0, (k, V)).astype(np.float32)
        drafts = rng.integers(0, V, k).astype(np.int32)
        lg = oracle.accept_final(drafts, pl, ql, T, 4, t, 0)
        assert lg.used_fallback == 0
        if lg.n < k:
            p = np.exp(log_softmax(pl[lg.n].astype(np.float64) / T))
            q = np.exp(log_softmax(ql[lg.n].astype(np.float64) / T))
            assert p[lg.y] > q[lg.y]
