"""Property-based pins of the oracle's pointer recurrence (oracle/selection.py),
over random small groups drawn by hypothesis.

Every property is fixed by the method's definition and checked from outside
the oracle's loop:
  * validity (Eq. 2, Eq. 11): tokens are taken at most once, at most g per
    round and at most cap rounds; an episode ends by STOP, by the cap, or when
    no token is left;
  * an infinite STOP bias stops at the first step (K = T* - 1 = 0), and a
    bias of minus infinity keeps every token when the cap allows (a STOP
    round follows the last token), in ceil(n / g) rounds (the round count of
    grouped selection);
  * the STOP bias enters only the STOP logit, so a larger bias gives a prefix
    of the rounds of a smaller one; a larger cap extends the rounds of a
    smaller one;
  * without the history (u_t = u_1), the selection is the top K of one fixed
    score vector, computed here directly: the history holds START alone, so
    u_1 = c + q_start + v_start and the scores are K u_1 / sqrt(h);
  * permuting the tokens permutes the selection (continuous draws, no ties);
  * each round takes the top g tokens of the query formed from the history
    so far (the mean query of the newest round attending over START and every
    token taken), recomputed here from Eq. 4 and Eq. 11;
  * at the first step STOP wins exactly when its logit exceeds the best
    token's, which is checked at biases just below and above the tie.
A plausible slip in the oracle (a token taken twice, the cap counted in
tokens instead of rounds, the bias added to every logit, the history ignored,
a wrong query after a group) breaks one of them.
"""
import math

import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from oracle.selection import run_episode

SETTINGS = dict(max_examples=60, deadline=None, suppress_health_check=[HealthCheck.too_slow])


def _group(seed, n, h):
    rng = np.random.default_rng(seed)
    K, Q, V = (rng.standard_normal((n, h)) for _ in range(3))
    start = tuple(rng.standard_normal(h) for _ in range(3))
    k_stop = rng.standard_normal(h)
    c = rng.standard_normal(h)
    return K, Q, V, start, k_stop, c


def _episode(inst, cap, b, h, g=1, **kw):
    K, Q, V, start, k_stop, c = inst
    return run_episode(K, Q, V, start, k_stop, c, cap, b, h, keep_steps=False, g=g, **kw)


shapes = st.tuples(st.integers(0, 2**31 - 1), st.integers(1, 24), st.sampled_from([2, 4, 8]))


@settings(**SETTINGS)
@given(shapes, st.integers(0, 30), st.integers(1, 5),
       st.one_of(st.floats(-3, 3), st.sampled_from([math.inf, -math.inf])))
def test_episode_is_valid(shape, cap, g, b):
    seed, n, h = shape
    ep = _episode(_group(seed, n, h), cap, b, h, g)
    a = ep.actions
    assert len(set(a)) == len(a) and all(0 <= x < n for x in a)
    assert len(ep.groups) <= cap
    assert sum(len(x) for x in ep.groups) == len(a)
    left = n
    for grp in ep.groups:
        assert len(grp) == min(g, left)          # a round keeps g tokens, or all that remain
        left -= len(grp)
    assert ep.n_steps <= cap
    assert ep.stopped or len(ep.groups) == cap or left == 0


@settings(**SETTINGS)
@given(shapes, st.integers(1, 30), st.integers(1, 5))
def test_infinite_bias_stops_at_once(shape, cap, g):
    seed, n, h = shape
    ep = _episode(_group(seed, n, h), cap, math.inf, h, g)
    assert ep.actions == [] and ep.stopped and ep.n_steps == 1


@settings(**SETTINGS)
@given(shapes, st.integers(1, 5))
def test_never_stopping_keeps_every_token_in_ceil_n_over_g_rounds(shape, g):
    seed, n, h = shape
    rounds = -(-n // g)
    ep = _episode(_group(seed, n, h), rounds + 1, -math.inf, h, g)
    assert sorted(ep.actions) == list(range(n))
    assert len(ep.groups) == rounds
    assert ep.stopped and ep.n_steps == rounds + 1   # the round after the last token is STOP
    # with the cap exactly at the round count, no STOP round is run
    ep2 = _episode(_group(seed, n, h), rounds, -math.inf, h, g)
    assert ep2.groups == ep.groups and not ep2.stopped


@settings(**SETTINGS)
@given(shapes, st.integers(0, 30), st.integers(1, 5), st.floats(-3, 3), st.floats(0, 3))
def test_larger_bias_gives_a_prefix(shape, cap, g, b1, db):
    seed, n, h = shape
    inst = _group(seed, n, h)
    lo, hi = _episode(inst, cap, b1, h, g), _episode(inst, cap, b1 + db, h, g)
    assert hi.groups == lo.groups[:len(hi.groups)]


@settings(**SETTINGS)
@given(shapes, st.integers(0, 20), st.integers(0, 10), st.integers(1, 5),
       st.one_of(st.floats(-3, 3), st.just(-math.inf)))
def test_larger_cap_extends(shape, cap, extra, g, b):
    seed, n, h = shape
    inst = _group(seed, n, h)
    short, long = _episode(inst, cap, b, h, g), _episode(inst, cap + extra, b, h, g)
    assert long.groups[:len(short.groups)] == short.groups


@settings(**SETTINGS)
@given(shapes, st.integers(0, 30))
def test_no_history_is_top_k_of_the_first_scores(shape, cap):
    seed, n, h = shape
    inst = _group(seed, n, h)
    K, Q, V, (k_s, q_s, v_s), k_stop, c = inst
    u1 = c + q_s + v_s                      # attention over START alone has weight 1
    scores = K @ u1 / math.sqrt(h)
    order = sorted(range(n), key=lambda j: (-scores[j], j))
    ep = _episode(inst, cap, -math.inf, h, no_history=True)
    assert ep.actions == order[:min(cap, n)]


@settings(**SETTINGS)
@given(shapes, st.integers(0, 30), st.integers(1, 5), st.floats(-2, 2), st.integers(0, 2**31 - 1))
def test_permuting_tokens_permutes_the_selection(shape, cap, g, b, pseed):
    seed, n, h = shape
    K, Q, V, start, k_stop, c = _group(seed, n, h)
    p = np.random.default_rng(pseed).permutation(n)        # new row i is old row p[i]
    ref = _episode((K, Q, V, start, k_stop, c), cap, b, h, g)
    per = _episode((K[p], Q[p], V[p], start, k_stop, c), cap, b, h, g)
    assert [sorted(int(p[x]) for x in grp) for grp in per.groups] == [sorted(grp) for grp in ref.groups]
    assert per.stopped == ref.stopped


def _round_query(inst, h, chosen, last_group):
    """The query after the rounds so far (Eq. 4; Eq. 11 for a group): the newest
    round's mean query attends over START and every chosen token (keys and
    values), plus the text context.  Written out independently of the
    oracle's loop."""
    K, Q, V, (k_s, q_s, v_s), k_stop, c = inst
    q = q_s if not last_group else np.mean([Q[j] for j in last_group], axis=0)
    keys = [k_s] + [K[j] for j in chosen]
    vals = [v_s] + [V[j] for j in chosen]
    s = np.array([float(k @ q) for k in keys]) / math.sqrt(h)
    w = np.exp(s - s.max())
    w = w / w.sum()
    return c + q + sum(wi * vi for wi, vi in zip(w, vals))


@settings(**SETTINGS)
@given(shapes, st.integers(1, 5))
def test_each_round_follows_the_history_query(shape, g):
    """Replays the oracle's rounds with the query recomputed from the history
    at each round: its group must be the top g of that query's scores over the
    tokens not yet taken (ties to the lower index)."""
    seed, n, h = shape
    inst = _group(seed, n, h)
    K = inst[0]
    ep = _episode(inst, n + 1, -math.inf, h, g)
    chosen, last = [], []
    for grp in ep.groups:
        u = _round_query(inst, h, chosen, last)
        scores = K @ u / math.sqrt(h)
        free = [j for j in range(n) if j not in chosen]
        want = sorted(free, key=lambda j: (-scores[j], j))[:g]
        assert sorted(grp) == sorted(want)
        chosen += list(grp)
        last = list(grp)


@settings(**SETTINGS)
@given(shapes, st.integers(1, 5), st.floats(1e-6, 1e-2))
def test_stop_decision_at_the_first_step(shape, g, eps):
    """At step 1 the STOP logit is <u_1, k_stop> / sqrt(h) + b and the best
    token's is max_j <u_1, k_j> / sqrt(h), with u_1 = c + q_start + v_start:
    a bias eps below the tie takes a token, eps above it stops."""
    seed, n, h = shape
    inst = _group(seed, n, h)
    K, Q, V, (k_s, q_s, v_s), k_stop, c = inst
    u1 = c + q_s + v_s
    tie = float(np.max(K @ u1) / math.sqrt(h) - k_stop @ u1 / math.sqrt(h))
    below = _episode(inst, 3, tie - eps, h, g)
    above = _episode(inst, 3, tie + eps, h, g)
    assert len(below.groups) >= 1 and below.groups[0]
    assert above.actions == [] and above.stopped
