"""Algorithm 1, steps 2-4: the adaptive sequential pointer selection.

Paper: Problem Formulation (Eq. 2: ordered trajectory, K = T* - 1 for the
first STOP at step T*), Conditional Sequential Pointer Policy (candidate
memory M = [H; s_stop], START query, pointer step of Eq. 4 with the mask
update and q_{t+1} = M[a_t] in the forward pass), Algorithm 1 step 3 (the
round loop with cap T_max, the TopG group of step 3c) and step 4
(native-order restore), and Section "Grouped Execution for High-Resolution
Inputs" (Eq. 11: g tokens per round).

Per episode (one group of one image) with tokens j = 0..n-1, the oracle runs,
in float64 on the exact stored values:

    history = [START]; e = START; selected = {}
    for t = 1 .. cap:
        s_tau   = sigma * <q_e, k_tau>         for every history entry tau
        alpha   = softmax(s)
        u_t     = c_b + q_e + sum_tau alpha_tau v_tau
        l_t(j)  = sigma * <u_t, k_j>           (-inf for selected j)
        l_t(STOP) = sigma * <u_t, k_stop> + b_stop
        a_t     = first maximal index over (tokens..., STOP)
        if a_t is STOP: stop
        selected += a_t; history += a_t; e = a_t
    kept = sorted(selected)

With g tokens per round (Eq. 11), a round that does not stop keeps the
min(g, unselected) largest unselected token logits U_r, all of them appended
to the history; the next round's query row is the mean of the Q rows of U_r.
With g = 1 this is the loop above.

with sigma = h^(-1/2).  Readings taken here (the paper leaves these open):
* One decoder layer, one head, no normalisation and no feed-forward block: the
  pointer logits are the cross-attention logits, and the value path of the
  cross-attention and the feed-forward block never reach a_t.  The causal
  self-attention over the history uses the history entries' keys and values
  and the newest entry's query, which is also its residual in query space.
* The text context c_b enters the pointer query additively (the encoder of
  Eq. 3 is not on this path).
* b_stop is an additive scalar on the STOP logit, set per workload.
* The cap counts rounds; at the cap the episode ends without a STOP step.
* Ties go to the lowest index and STOP, last in M, loses exact ties.  When no
  token is left unselected only STOP remains and it is taken.
* The temperature and the straight-through estimator of Eq. 4 do not change
  a_t and are not part of the forward path.
* Groups of an image are independent episodes; the image's kept list is the
  concatenation of its groups' kept lists in group order (ascending, since
  groups are contiguous).
* g > 1: STOP ends the episode only when it is the largest logit of the round
  (Eq. 11 and the sentence before it); otherwise U_r is the g largest
  unselected token logits, ties to the lowest index, fewer when fewer tokens
  are left.  U_r enters the history in descending-logit order, and the next
  query (the newest entry's query and residual at g = 1) is the mean of the Q
  rows of U_r, which does not depend on that order.  The cap counts rounds.
"""
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

STOP = -1


@dataclass
class StepRecord:
    """What one pointer step (one round of g tokens) saw (Eq. 4, Eq. 11)."""
    t: int
    action: int              # taken action: first token of the group, or STOP
    argmax: int              # the oracle's own argmax (differs only when forced)
    token_max: float         # largest unselected token logit (-inf if none left)
    stop_raw: float          # sigma * <u, k_stop>, the STOP logit without b_stop
    stop_logit: float
    top1: float              # largest finite candidate logit (tokens and STOP)
    top2: float              # second largest finite candidate logit (-inf if none)
    margin: float            # (top1 - top2) / scale, inf with fewer than 2 candidates
    logits: Optional[np.ndarray] = None   # token logits, -inf where selected
    u: Optional[np.ndarray] = None        # pointer query
    group: List[int] = field(default_factory=list)    # taken tokens, descending logit
    best_group: List[int] = field(default_factory=list)   # the oracle's own group
    group_min: float = -np.inf     # smallest logit in the taken group
    runner_up: float = -np.inf     # largest candidate left out (STOP included if not taken)
    margin_stop: float = np.inf    # relative gap between the top token and STOP
    margin_member: float = np.inf  # relative gap between the g-th and (g+1)-th token


@dataclass
class EpisodeResult:
    actions: List[int]                       # selected tokens in selection order
    stopped: bool                            # True if a STOP step was taken
    steps: List[StepRecord] = field(default_factory=list)
    groups: List[List[int]] = field(default_factory=list)   # tokens taken per round

    @property
    def kept(self) -> List[int]:
        return sorted(self.actions)

    @property
    def n_steps(self) -> int:
        """Rounds run: one per taken group, plus the STOP round."""
        return len(self.groups) + (1 if self.stopped else 0)


@dataclass
class SelectResult:
    episodes: List[EpisodeResult]            # one per group
    kept: List[List[int]]                    # per image, image-local, ascending
    kept_cnt: np.ndarray                     # [B]
    grp_cnt: np.ndarray                      # [G]


def _relative_margin(cand: np.ndarray):
    """Top-2 gap of the finite candidates over their scale.

    The scale is the larger of |top1|, |top2| and the root mean square of all
    finite candidate logits, so that a gap between two logits close to zero is
    not reported as large.
    """
    fin = cand[np.isfinite(cand)]
    if fin.size == 0:
        return -np.inf, -np.inf, np.inf
    if fin.size == 1:
        return float(fin[0]), -np.inf, np.inf
    top = np.sort(fin)[::-1]
    t1, t2 = float(top[0]), float(top[1])
    scale = max(abs(t1), abs(t2), float(np.sqrt(np.mean(fin * fin))))
    if scale == 0.0:
        return t1, t2, np.inf if t1 != t2 else 0.0
    return t1, t2, (t1 - t2) / scale


def _rel_gap(a: float, b: float, fin: np.ndarray) -> float:
    """(a - b) over max(|a|, |b|, rms of the finite candidates); inf if b is -inf."""
    if not np.isfinite(b):
        return np.inf
    scale = max(abs(a), abs(b), float(np.sqrt(np.mean(fin * fin))) if fin.size else 0.0)
    if scale == 0.0:
        return np.inf if a != b else 0.0
    return (a - b) / scale


def run_episode(K, Q, V, start, k_stop, c, cap: int, b_stop: float, h: int,
                no_history: bool = False, forced: Optional[Sequence] = None,
                keep_steps: bool = True, keep_vectors: bool = True, g: int = 1,
                ignore_stop: bool = False) -> EpisodeResult:
    """One episode of the pointer recurrence (Eq. 4 with the STOP rule of Eq. 2;
    g tokens per round as in Eq. 11).

    K, Q, V: [n, h] projected rows of the group's tokens; start: (k, q, v) of
    the START embedding; k_stop: [h] key of the STOP embedding; c: [h] text
    context of the image.  ``no_history`` keeps u_t = u_1 (the query never sees
    the selection history).  ``forced`` replays a given action sequence instead
    of taking the argmax: per round a token index (g = 1) or a sequence of
    token indices, STOP as -1.  ``keep_vectors`` stores the logits and the
    query of every step in its record.  ``ignore_stop`` runs the full rollout
    over which the trajectory sums of Eqs. 5-7 run to T_max: the action is the
    best token even where STOP is the largest logit (STOP is still scored, and
    taken only once no token is left).
    """
    if g < 1:
        raise ValueError("g must be at least 1")
    K = np.asarray(K, np.float64)
    Q = np.asarray(Q, np.float64)
    V = np.asarray(V, np.float64)
    k_s, q_s, v_s = (np.asarray(r, np.float64) for r in start)
    k_stop = np.asarray(k_stop, np.float64)
    c = np.asarray(c, np.float64)
    n = K.shape[0]
    sigma = 1.0 / np.sqrt(h)

    hist_k = [k_s]
    hist_v = [v_s]
    q_e = q_s
    selected = np.zeros(n, dtype=bool)
    actions: List[int] = []
    groups: List[List[int]] = []
    steps: List[StepRecord] = []
    stopped = False
    u1 = None
    for t in range(1, cap + 1):
        if no_history and u1 is not None:
            u = u1
        else:
            Kh = np.stack(hist_k)
            Vh = np.stack(hist_v)
            s = sigma * (Kh @ q_e)
            w = np.exp(s - s.max())
            alpha = w / w.sum()
            u = c + q_e + alpha @ Vh
            if u1 is None:
                u1 = u
        logits = sigma * (K @ u)
        logits[selected] = -np.inf
        stop_raw = float(sigma * (k_stop @ u))
        stop_logit = stop_raw + b_stop
        # unselected tokens by descending logit, ties to the lower index
        free = np.flatnonzero(~selected)
        order = free[np.lexsort((free, -logits[free]))]
        if order.size == 0:
            best = STOP
            token_max = -np.inf
        else:
            token_max = float(logits[order[0]])
            best = STOP if stop_logit > token_max and not ignore_stop else int(order[0])
        best_group = [] if best == STOP else [int(x) for x in order[:g]]
        cand = np.append(logits, stop_logit)
        t1, t2, margin = _relative_margin(cand)
        fin = cand[np.isfinite(cand)]
        m_stop = _rel_gap(token_max, stop_logit, fin) if order.size else np.inf
        m_stop = abs(m_stop)
        m_member = (_rel_gap(float(logits[order[g - 1]]), float(logits[order[g]]), fin)
                    if order.size > g else np.inf)
        if forced is not None:
            if t - 1 >= len(forced):
                break
            f = forced[t - 1]
            grp = [int(x) for x in f] if isinstance(f, (list, tuple, np.ndarray)) else [int(f)]
            act = STOP if grp == [STOP] else grp[0]
            if act == STOP:
                grp = []
        else:
            act = best
            grp = best_group
        if keep_steps:
            chosen = set(grp)
            left = [x for x in order if x not in chosen]
            runner = float(logits[left[0]]) if left else -np.inf
            if act != STOP:
                runner = max(runner, stop_logit)
            steps.append(StepRecord(t=t, action=act, argmax=best, token_max=token_max,
                                    stop_raw=stop_raw, stop_logit=stop_logit, top1=t1,
                                    top2=t2, margin=margin,
                                    logits=logits if keep_vectors else None,
                                    u=u if keep_vectors else None,
                                    group=list(grp), best_group=best_group,
                                    group_min=min((float(logits[x]) for x in grp), default=-np.inf),
                                    runner_up=runner, margin_stop=m_stop,
                                    margin_member=m_member))
        if act == STOP:
            stopped = True
            break
        for a in grp:
            if selected[a]:
                raise ValueError(f"forced action {a} at step {t} selects a token twice")
            selected[a] = True
            actions.append(a)
            hist_k.append(K[a])
            hist_v.append(V[a])
        groups.append(list(grp))
        # the next query: the newest entry's query (g = 1), the mean of the
        # group's query rows in general
        q_e = Q[grp[0]] if len(grp) == 1 else Q[grp].sum(axis=0) / len(grp)
    return EpisodeResult(actions=actions, stopped=stopped, steps=steps, groups=groups)


def select(KQV, ctx, img_off, grp_off, grp_img, grp_cap, b_stop: float, h: int,
           no_history: bool = False, keep_steps: bool = True, keep_vectors: bool = True,
           groups: Optional[Sequence[int]] = None, g: int = 1) -> SelectResult:
    """All episodes of a batch (Algorithm 1 steps 2-4).

    KQV: [T_vis + 2, 3h] projected rows (row T_vis is START, T_vis + 1 STOP);
    ctx: [B, h]; img_off[B+1], grp_off[G+1] row offsets; grp_img[G] owner
    image; grp_cap[G] round caps.  ``groups`` restricts the run to a subset of
    episodes (the others report no selection); g is the tokens per round.
    """
    KQV = np.asarray(KQV, np.float64)
    T_vis = KQV.shape[0] - 2
    Kall, Qall, Vall = KQV[:, :h], KQV[:, h:2 * h], KQV[:, 2 * h:3 * h]
    start = (Kall[T_vis], Qall[T_vis], Vall[T_vis])
    k_stop = Kall[T_vis + 1]
    B = len(img_off) - 1
    G = len(grp_img)
    run = range(G) if groups is None else groups
    episodes = [EpisodeResult(actions=[], stopped=False) for _ in range(G)]
    for gi in run:
        r0, r1 = int(grp_off[gi]), int(grp_off[gi + 1])
        episodes[gi] = run_episode(Kall[r0:r1], Qall[r0:r1], Vall[r0:r1], start, k_stop,
                                   ctx[int(grp_img[gi])], int(grp_cap[gi]), b_stop, h,
                                   no_history=no_history, keep_steps=keep_steps,
                                   keep_vectors=keep_vectors, g=g)
    kept: List[List[int]] = [[] for _ in range(B)]
    for gi in range(G):
        b = int(grp_img[gi])
        base = int(grp_off[gi]) - int(img_off[b])
        kept[b].extend(base + j for j in episodes[gi].kept)
    kept_cnt = np.array([len(k) for k in kept], np.int32)
    grp_cnt = np.array([len(e.actions) for e in episodes], np.int32)
    return SelectResult(episodes=episodes, kept=kept, kept_cnt=kept_cnt, grp_cnt=grp_cnt)
