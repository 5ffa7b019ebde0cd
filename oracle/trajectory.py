"""The trajectory-aggregated pointer distributions (Section "Trajectory-Aware
Differentiable Optimization": Eq. 4's p_t, Eqs. 5-7).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Along a pointer trajectory (one episode, g = 1), the oracle computes in
float64:

    p_t       = softmax(l_t / tau) over the candidates of step t: the
                unselected tokens and STOP (selected tokens have probability 0)
    A_1 = 1,  A_{t+1} = A_t (1 - p_t(STOP))                  (Eq. 5)
    s_i       = sum_t A_t p_t(i) beta^t                      (Eq. 6)
    K_bar     = sum_t A_t (1 - p_t(STOP))                    (Eq. 7)

Readings taken here:
* The sums run over the steps the trajectory executes.  With ``ignore_stop``
  the trajectory is the full rollout: the best token is taken at every step
  (STOP is scored but never taken while a token is left) up to the cap, which
  plays the role of T_max.  Without it the trajectory ends at the first STOP
  step, which is included.
* The logits are those of the inference path (the same l_t that decide a_t;
  Eq. 4 with the STOP bias), scaled by 1 / tau only inside p_t.
* A step with no finite candidate (no token left and a STOP logit of -inf)
  has p_t(STOP) = 1.
"""
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

from .selection import EpisodeResult, run_episode


@dataclass
class TrajectoryResult:
    s: np.ndarray             # [n] Eq. 6 per token of the episode
    kbar: float               # Eq. 7
    pstop: List[float]        # p_t(STOP) per executed step
    alive: List[float]        # A_t per executed step
    episode: EpisodeResult


def step_distribution(logits: np.ndarray, stop_logit: float, tau: float) -> np.ndarray:
    """Eq. 4's p_t = softmax(l_t / tau) over [tokens..., STOP]; -inf logits
    (selected tokens) get probability 0."""
    cand = np.append(np.asarray(logits, np.float64), stop_logit)
    p = np.zeros_like(cand)
    fin = np.isfinite(cand)
    if not fin.any():
        p[-1] = 1.0
        return p
    x = cand[fin] / tau
    w = np.exp(x - x.max())
    p[fin] = w / w.sum()
    return p


def aggregate(ep: EpisodeResult, n: int, tau: float, beta: float) -> TrajectoryResult:
    """Eqs. 5-7 over the executed steps of an episode run with keep_vectors."""
    A = 1.0
    s = np.zeros(n)
    kbar = 0.0
    pstop: List[float] = []
    alive: List[float] = []
    for st in ep.steps:
        p = step_distribution(st.logits, st.stop_logit, tau)
        alive.append(A)
        s += A * beta ** st.t * p[:n]
        kbar += A * (1.0 - p[n])
        pstop.append(float(p[n]))
        A *= 1.0 - p[n]
    return TrajectoryResult(s=s, kbar=kbar, pstop=pstop, alive=alive, episode=ep)


def run_trajectory(K, Q, V, start, k_stop, c, cap: int, b_stop: float, h: int, tau: float,
                   beta: float, ignore_stop: bool = False, no_history: bool = False,
                   forced: Optional[Sequence] = None) -> TrajectoryResult:
    """One episode (as ``selection.run_episode``) and its trajectory sums."""
    ep = run_episode(K, Q, V, start, k_stop, c, cap, b_stop, h, no_history=no_history,
                     forced=forced, keep_steps=True, keep_vectors=True, ignore_stop=ignore_stop)
    return aggregate(ep, np.asarray(K).shape[0], tau, beta)
