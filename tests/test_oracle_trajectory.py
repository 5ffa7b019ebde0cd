"""Pins of the oracle's trajectory sums (Section "Trajectory-Aware
Differentiable Optimization": p_t of Eq. 4, A_t of Eq. 5, s_i of Eq. 6 and
K_bar of Eq. 7).

Each pin checks the oracle against something other than its own formulas: a
library softmax, an identity that holds only when p_t sums to one over the
same candidates that the alive probability discounts, and closed forms in the
cold (tau -> 0) and hot (tau -> inf) limits.
"""
import math

import numpy as np
import torch

import oracle
from oracle.selection import STOP


def _episode(rng, n, h):
    K = rng.standard_normal((n, h))
    Q = rng.standard_normal((n, h))
    V = rng.standard_normal((n, h))
    start = tuple(rng.standard_normal(h) for _ in range(3))
    k_stop = rng.standard_normal(h)
    c = rng.standard_normal(h) * 0.3
    return K, Q, V, start, k_stop, c


def test_step_distribution_is_the_library_softmax_over_candidates():
    """p_t over the unselected tokens and STOP is torch.softmax(l / tau) of
    those candidates; selected tokens get exactly 0."""
    rng = np.random.default_rng(31)
    for trial in range(30):
        n, h = int(rng.integers(1, 12)), int(rng.integers(1, 6))
        tau = float(rng.uniform(0.2, 3.0))
        args = _episode(rng, n, h)
        tr = oracle.run_trajectory(*args, int(rng.integers(1, n + 2)), float(rng.normal()), h,
                                   tau=tau, beta=0.9, ignore_stop=bool(trial % 2))
        for st in tr.episode.steps:
            p = oracle.step_distribution(st.logits, st.stop_logit, tau)
            cand = torch.from_numpy(np.append(st.logits, st.stop_logit))
            fin = torch.isfinite(cand)
            want = torch.softmax(cand[fin] / tau, dim=0).numpy()
            assert np.allclose(p[fin.numpy()], want, rtol=0, atol=1e-14)
            assert (p[~fin.numpy()] == 0).all()


def test_scores_sum_to_the_soft_count_without_discount():
    """beta = 1: sum_i s_i = K_bar, since the token probabilities of a step
    sum to 1 - p_t(STOP) (Eq. 6 summed over i against Eq. 7)."""
    rng = np.random.default_rng(32)
    for trial in range(40):
        n, h = int(rng.integers(1, 15)), int(rng.integers(1, 6))
        args = _episode(rng, n, h)
        tr = oracle.run_trajectory(*args, int(rng.integers(1, n + 3)), float(rng.normal()), h,
                                   tau=float(rng.uniform(0.3, 2.0)), beta=1.0,
                                   ignore_stop=bool(trial % 2))
        assert abs(tr.s.sum() - tr.kbar) < 1e-12 * max(1.0, tr.kbar)
        assert all(0.0 <= a <= 1.0 for a in tr.alive)
        assert all(x >= y for x, y in zip(tr.alive, tr.alive[1:]))


def test_cold_limit_is_the_hard_trajectory():
    """tau -> 0: p_t is one-hot on a_t, so A_t = 1 until the STOP step,
    s_i = beta^t_i for the token taken at step t_i (0 for the others) and
    K_bar = K, the number of tokens taken before STOP."""
    rng = np.random.default_rng(33)
    checked = 0
    for trial in range(40):
        n, h = int(rng.integers(2, 12)), int(rng.integers(2, 6))
        args = _episode(rng, n, h)
        beta = float(rng.uniform(0.5, 1.0))
        tr = oracle.run_trajectory(*args, n + 1, float(rng.normal()), h, tau=1e-9, beta=beta)
        ep = tr.episode
        if min(st.margin for st in ep.steps) < 1e-6:
            continue
        want = np.zeros(n)
        for t, a in enumerate(ep.actions, start=1):
            want[a] = beta ** t
        assert np.allclose(tr.s, want, rtol=0, atol=1e-12)
        assert ep.stopped and abs(tr.kbar - len(ep.actions)) < 1e-12
        assert tr.pstop[-1] == 1.0 and all(p < 1e-12 for p in tr.pstop[:-1])
        checked += 1
    assert checked >= 20


def test_hot_limit_is_uniform_over_the_candidates():
    """tau -> inf over the full rollout (cap = n, STOP never taken): every
    candidate has probability 1 / (n - t + 2) at step t, so
    A_t = (n - t + 2) / (n + 1), K_bar = n / 2 and
    s_i = sum_{t <= t_i} beta^t / (n + 1) for the token taken at step t_i."""
    rng = np.random.default_rng(34)
    for trial in range(20):
        n, h = int(rng.integers(1, 14)), int(rng.integers(1, 6))
        args = _episode(rng, n, h)
        beta = float(rng.uniform(0.5, 1.0))
        tr = oracle.run_trajectory(*args, n, float(rng.normal()), h, tau=1e13, beta=beta,
                                   ignore_stop=True)
        ep = tr.episode
        assert len(ep.actions) == n and not ep.stopped
        assert np.allclose(tr.alive, [(n - t + 2) / (n + 1) for t in range(1, n + 1)], atol=1e-9)
        assert abs(tr.kbar - n / 2) < 1e-9
        want = np.zeros(n)
        for ti, a in enumerate(ep.actions, start=1):
            want[a] = sum(beta ** t for t in range(1, ti + 1)) / (n + 1)
        assert np.allclose(tr.s, want, rtol=0, atol=1e-9)


def test_full_rollout_takes_the_best_token_at_every_step():
    """ignore_stop decides as a run whose STOP logit is -inf (the token logits
    do not depend on b_stop) and runs to min(cap, n) steps, plus a final STOP
    step when the tokens run out first; p_t still scores STOP with its bias."""
    rng = np.random.default_rng(35)
    for trial in range(30):
        n, h = int(rng.integers(1, 12)), int(rng.integers(1, 6))
        args = _episode(rng, n, h)
        cap = int(rng.integers(1, n + 3))
        b = float(rng.normal()) + 2.0
        roll = oracle.run_trajectory(*args, cap, b, h, tau=1.0, beta=0.9, ignore_stop=True)
        never = oracle.run_episode(*args, cap, -math.inf, h)
        assert roll.episode.actions == never.actions
        assert len(roll.episode.steps) == (cap if cap <= n else n + 1)
        for st in roll.episode.steps:
            assert st.stop_logit == st.stop_raw + b
