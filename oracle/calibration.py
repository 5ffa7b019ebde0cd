"""The STOP bias that makes a workload retain a target number of tokens.

The paper trains separate selectors per operating point and reports the mean
retained count of each (Section "Baselines and Implementation Details");
with random-initialised selector weights that count is instead set by an
additive bias b on the STOP logit (a reading: the paper has no such bias).

b enters only the STOP logit, so the token trajectory of an episode does not
depend on it: run every episode once with b = -inf for its whole cap and
record, per step t, m_t = (largest token logit) - sigma <u_t, k_stop>.  STOP
is taken at the first step with b > m_t (STOP loses exact ties), hence
K(b) = #{t : min(m_1..m_t) >= b}, and the batch total sum_g K_g(b) is the
number of prefix minima >= b.  The bias is placed halfway between two
adjacent prefix minima so that no STOP decision sits near a tie.

With g tokens per round (Eq. 11) STOP still decides only against the largest
token logit of a round, so the same m_t applies per round; a round that does
not stop keeps its whole group, so each prefix minimum is counted once per
token of that round's group.
"""
import math
from typing import List, Sequence, Tuple

import numpy as np

from .selection import run_episode


def stop_thresholds(KQV, ctx, grp_off, grp_img, grp_cap, h: int, g: int = 1) -> List[np.ndarray]:
    """Per group, the prefix minima of m_t over the rounds of a never-stopping
    run, each repeated once per token its round keeps."""
    KQV = np.asarray(KQV, np.float64)
    T_vis = KQV.shape[0] - 2
    Kall, Qall, Vall = KQV[:, :h], KQV[:, h:2 * h], KQV[:, 2 * h:3 * h]
    start = (Kall[T_vis], Qall[T_vis], Vall[T_vis])
    k_stop = Kall[T_vis + 1]
    out = []
    for gi in range(len(grp_img)):
        r0, r1 = int(grp_off[gi]), int(grp_off[gi + 1])
        rounds = min(int(grp_cap[gi]), -(-(r1 - r0) // g))
        ep = run_episode(Kall[r0:r1], Qall[r0:r1], Vall[r0:r1], start, k_stop,
                         ctx[int(grp_img[gi])], rounds, -math.inf, h, keep_vectors=False, g=g)
        m = np.array([s.token_max - s.stop_raw for s in ep.steps], np.float64)
        pm = np.minimum.accumulate(m) if m.size else m
        out.append(np.repeat(pm, [len(x) for x in ep.groups]))
    return out


def retained_total(prefix_minima: Sequence[np.ndarray], b: float) -> int:
    return int(sum(int(np.count_nonzero(pm >= b)) for pm in prefix_minima))


def choose_stop_bias(prefix_minima: Sequence[np.ndarray], target_total: float,
                     stop_inside_cap: bool = False) -> Tuple[float, int]:
    """A float32 bias whose batch total retained count is the achievable total
    closest to ``target_total``; returns (bias, total).  ``stop_inside_cap``
    excludes the total at which no episode takes a STOP step."""
    v = np.sort(np.concatenate([np.asarray(p, np.float64) for p in prefix_minima]))[::-1]
    n = v.size
    # total k is achievable when v[k] < v[k-1] strictly (k = 0 and k = n always are).
    feasible = [0] + [k for k in range(1, n) if v[k] < v[k - 1]] + ([] if stop_inside_cap else [n])
    k = min(feasible, key=lambda k: (abs(k - target_total), k))
    if k == 0:
        b = v[0] + max(1.0, abs(v[0]))
    elif k == n:
        b = v[n - 1] - max(1.0, abs(v[n - 1]))
    else:
        b = 0.5 * (v[k - 1] + v[k])
    b32 = float(np.float32(b))
    got = retained_total(prefix_minima, b32)
    if got != k:
        raise RuntimeError(f"float32 rounding of the stop bias moved the total ({got} != {k})")
    return b32, k
