"""Pins of the oracle's grouped selection (Eq. 11; Algorithm 1 step 3c): g
tokens per round, the round stopping only when STOP is the largest logit,
the group entering the history together and the next query being the mean
of the group's query rows (the reading taken where the paper leaves the
group query open).

As for g = 1, none of these compares the oracle with a retyping of its own
code: every round is recomputed with torch's attention and matmul, the
group is checked by brute force over subsets, and the round count, order
invariance and no-history cases are closed forms.
"""
import itertools
import math

import numpy as np
import pytest
import torch

import oracle
from oracle.selection import STOP
from paper_2609_13804_amd import workloads as W


def _random_episode(rng, n, h):
    K = rng.standard_normal((n, h))
    Q = rng.standard_normal((n, h))
    V = rng.standard_normal((n, h))
    start = tuple(rng.standard_normal(h) for _ in range(3))
    k_stop = rng.standard_normal(h)
    c = rng.standard_normal(h) * 0.3
    return K, Q, V, start, k_stop, c


def _torch_round(K, Q, V, start, k_stop, c, groups, b, h):
    """Logits of the round after `groups` (list of token lists), with torch:
    history [START] + all grouped tokens, query the mean of the last group's
    Q rows (START's query before the first group)."""
    k_s, q_s, v_s = start
    hist_k = [torch.from_numpy(k_s)] + [torch.from_numpy(K[j]) for grp in groups for j in grp]
    hist_v = [torch.from_numpy(v_s)] + [torch.from_numpy(V[j]) for grp in groups for j in grp]
    q = torch.from_numpy(q_s) if not groups else torch.from_numpy(Q[groups[-1]]).mean(dim=0)
    kk = torch.stack(hist_k).view(1, 1, -1, h)
    vv = torch.stack(hist_v).view(1, 1, -1, h)
    att = torch.nn.functional.scaled_dot_product_attention(q.view(1, 1, 1, h), kk, vv,
                                                           scale=1.0 / math.sqrt(h))
    u = torch.from_numpy(c) + q + att.view(h)
    logits = ((torch.from_numpy(K) @ u) / math.sqrt(h)).numpy().copy()
    for grp in groups:
        logits[grp] = -np.inf
    stop = float(torch.dot(torch.from_numpy(k_stop), u) / math.sqrt(h)) + b
    return logits, stop


def test_every_round_matches_library_attention_and_best_subset():
    """Free-running grouped episodes on tiny inputs: every round's logits are
    torch's, the round stops exactly when STOP beats every unselected token,
    and otherwise the group is the subset of min(g, unselected) tokens with
    the largest logit sum (brute force over all subsets)."""
    rng = np.random.default_rng(21)
    for trial in range(40):
        n, h = int(rng.integers(2, 9)), int(rng.integers(1, 6))
        g = int(rng.integers(2, 5))
        K, Q, V, start, k_stop, c = _random_episode(rng, n, h)
        cap = int(rng.integers(1, n + 2))
        b = float(rng.normal()) * 0.5
        res = oracle.run_episode(K, Q, V, start, k_stop, c, cap, b, h, g=g)
        for r, step in enumerate(res.steps):
            want, want_stop = _torch_round(K, Q, V, start, k_stop, c, res.groups[:r], b, h)
            fin = np.isfinite(want)
            assert np.allclose(step.logits[fin], want[fin], rtol=0, atol=1e-12)
            assert (step.logits[~fin] == -np.inf).all()
            assert abs(step.stop_logit - want_stop) < 1e-12
            free = np.flatnonzero(fin)
            if free.size == 0 or want_stop > want[free].max():
                assert step.action == STOP and r == len(res.steps) - 1 and res.stopped
                continue
            k = min(g, free.size)
            best = max(itertools.combinations(free.tolist(), k), key=lambda s: want[list(s)].sum())
            assert sorted(res.groups[r]) == sorted(best)
            # descending-logit order inside the group
            assert list(want[res.groups[r]]) == sorted(want[res.groups[r]], reverse=True)


def test_round_count_is_ceil_k_over_g_plus_stop():
    """P12: a run that stops takes ceil(K / g) + 1 rounds, every group but the
    last has g tokens, and a run that does not stop ends at the cap or when no
    token is left (Section "Grouped Execution for High-Resolution Inputs")."""
    rng = np.random.default_rng(22)
    for trial in range(60):
        n, h = int(rng.integers(1, 30)), int(rng.integers(1, 6))
        g = int(rng.integers(1, 7))
        K, Q, V, start, k_stop, c = _random_episode(rng, n, h)
        cap = int(rng.integers(1, 12))
        b = float(rng.normal()) * 0.8
        res = oracle.run_episode(K, Q, V, start, k_stop, c, cap, b, h, g=g, keep_vectors=False)
        k = len(res.actions)
        assert all(len(grp) == g for grp in res.groups[:-1])
        assert sum(len(grp) for grp in res.groups) == k
        assert len(set(res.actions)) == k <= min(n, cap * g)
        if res.stopped:
            assert res.n_steps == -(-k // g) + 1
        else:
            assert res.n_steps == len(res.groups) == min(cap, -(-n // g))


def test_group_order_inside_history_does_not_change_the_next_rounds():
    """The mean query and the softmax over the history are functions of the
    set of entries: replaying the same groups in another order inside each
    group gives the same logits at every round (to rounding)."""
    rng = np.random.default_rng(23)
    for trial in range(15):
        n, h, g = 12, 5, 4
        K, Q, V, start, k_stop, c = _random_episode(rng, n, h)
        res = oracle.run_episode(K, Q, V, start, k_stop, c, 3, -math.inf, h, g=g)
        shuffled = [list(rng.permutation(grp)) for grp in res.groups]
        rep = oracle.run_episode(K, Q, V, start, k_stop, c, 3, -math.inf, h, g=g, forced=shuffled)
        for a, b_ in zip(res.steps, rep.steps):
            assert np.allclose(a.logits, b_.logits, rtol=0, atol=1e-12, equal_nan=True)


def test_no_history_keeps_whole_groups_of_the_first_scores():
    """Without the history the query never changes, so every round takes the
    next g tokens of the first round's order, and the run stops at the first
    round whose best remaining token is not above STOP: K = min(cap g, n,
    g * ceil(#{l_1(j) > l_1(STOP)} / g)) (torch.sort for the order)."""
    rng = np.random.default_rng(24)
    for trial in range(30):
        n, h = int(rng.integers(1, 40)), int(rng.integers(1, 9))
        g = int(rng.integers(2, 6))
        K, Q, V, start, k_stop, c = _random_episode(rng, n, h)
        cap = int(rng.integers(1, 8))
        b = float(rng.normal())
        res = oracle.run_episode(K, Q, V, start, k_stop, c, cap, b, h, no_history=True, g=g)
        u1 = torch.from_numpy(c + start[1] + start[2])
        l1 = (torch.from_numpy(K) @ u1) / math.sqrt(h)
        stop1 = float(torch.dot(torch.from_numpy(k_stop), u1) / math.sqrt(h)) + b
        order = torch.sort(l1, descending=True, stable=True).indices.tolist()
        above = int((l1 > stop1).sum())
        k = min(cap * g, n, g * (-(-above // g)))
        assert res.actions == order[:k]


def test_group_larger_than_the_episode_takes_everything_at_once():
    """g >= n: the first round keeps every token (unless STOP leads), in
    descending-logit order, and the next round has only STOP left."""
    rng = np.random.default_rng(25)
    for trial in range(10):
        n, h = int(rng.integers(1, 7)), 3
        K, Q, V, start, k_stop, c = _random_episode(rng, n, h)
        res = oracle.run_episode(K, Q, V, start, k_stop, c, 3, -math.inf, h, g=n + int(rng.integers(0, 3)))
        assert len(res.groups) == 1 and sorted(res.groups[0]) == list(range(n))
        assert res.stopped and res.n_steps == 2 and res.steps[1].action == STOP


@pytest.mark.parametrize("g", [2, 5])
def test_grouped_calibration_reproduces_predicted_counts(g):
    """The STOP bias chosen from a never-stopping grouped run retains exactly
    the predicted total when the selection is run again with it."""
    w = W.WORKLOADS["tiny_bf16"]
    inp, lay = W.make_inputs(w), W.make_layout(w)
    KQV = oracle.project(inp["X"], inp["s_start"], inp["s_stop"], inp["W_kqv"], w.dtype)
    ctx = oracle.text_context(inp["E_text"], lay.text_off, inp["W_text"])
    pm = oracle.stop_thresholds(KQV, ctx, lay.grp_off, lay.grp_img, lay.grp_cap, w.h, g=g)
    for target in (0, 7, 20, 10 ** 6):
        b, total = oracle.choose_stop_bias(pm, target)
        res = oracle.select(KQV, ctx, lay.img_off, lay.grp_off, lay.grp_img, lay.grp_cap, b, w.h, g=g)
        assert int(res.kept_cnt.sum()) == total
