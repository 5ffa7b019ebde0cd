"""Comparison of the HIP path with the CPU oracle (test helper).

Tolerances (the bar every GPU parity test applies):
  * projected rows: per-row normwise relative error <= 1e-3 for bfloat16
    storage, 1e-5 for float32 (the GPU accumulates in float32 and rounds once;
    the oracle rounds the exact product once, so stored values may differ by one
    unit in the last place);
  * text context: per-row normwise relative error <= 1e-5 (float32 both sides);
  * logits: |l_gpu - l_oracle| <= tol * scale_t with tol = 1e-3 (bfloat16
    workloads) or 1e-5 (float32), scale_t the larger of the two top logits'
    magnitudes and the root mean square of the step's finite logits; with the
    SP_LOGITS dump this holds for every candidate of every step (tokens and
    STOP), and the masked tokens (-inf) must be exactly the selected ones;
  * selections: staged (the oracle runs on the GPU's own projected rows and
    context) and teacher-forced (the oracle replays the GPU's actions): every
    GPU action must equal the oracle's argmax, except at steps whose oracle
    top-2 relative margin is below 1e-4, where the GPU's action must be within
    1e-4 * scale_t of the oracle maximum; such steps are counted, not hidden;
  * kept indices and counts: equal to the GPU's own action sets, and equal to
    the free-running oracle for every episode without an exempt step;
  * compaction: bit-exact.

With g tokens per round (Eq. 11) the same protocol applies per round: the
GPU's group must be the oracle's as a set, except in rounds where the STOP
decision or the membership of the g-th token is a near-tie (relative gap
below 1e-4 between the top token and STOP, or between the g-th and (g+1)-th
token), which are counted like exempt steps.
"""
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

import oracle
from oracle.selection import STOP

MARGIN_EXEMPT = 1e-4


def logit_tol(dtype: str) -> float:
    return 1e-3 if dtype == "bf16" else 1e-5


def rows_relerr(got: np.ndarray, want: np.ndarray) -> float:
    num = np.linalg.norm(got - want, axis=1)
    den = np.maximum(np.linalg.norm(want, axis=1), 1e-30)
    return float((num / den).max()) if len(num) else 0.0


@dataclass
class SelectReport:
    episodes: int = 0
    steps: int = 0
    exempt_steps: int = 0
    max_logit_err: float = 0.0
    logits_checked: int = 0            # logit values compared element by element (SP_LOGITS)
    free_running_equal: int = 0
    free_running_checked: int = 0
    divergences: List[str] = field(default_factory=list)


def _scale(step) -> float:
    fin = step.logits[np.isfinite(step.logits)]
    parts = [abs(step.top1) if np.isfinite(step.top1) else 0.0,
             abs(step.top2) if np.isfinite(step.top2) else 0.0]
    cand = np.append(fin, step.stop_logit) if np.isfinite(step.stop_logit) else fin
    if cand.size:
        parts.append(float(np.sqrt(np.mean(cand * cand))))
    return max(parts + [1e-30])


def _close(a: float, b: float, tol: float) -> bool:
    if np.isinf(a) or np.isinf(b):
        return a == b
    return abs(a - b) <= tol


def check_logit_vector(got: np.ndarray, st, n: int, tol: float, scale: float, where: str) -> float:
    """One step's dumped logit vector (SP_LOGITS: token slots, then STOP)
    against the oracle's step record: the same tokens masked (-inf), slots past
    the group -inf, and every finite logit and the STOP logit within
    tol * scale.  Returns the largest error over the scale."""
    got = np.asarray(got, np.float64)
    tok, stop = got[:n], got[-1]
    want = np.asarray(st.logits, np.float64)
    assert np.array_equal(np.isneginf(tok), np.isneginf(want)), f"{where}: masked tokens differ"
    assert np.isneginf(got[n:-1]).all(), f"{where}: slots past the group are not -inf"
    fin = np.isfinite(want)
    assert np.isfinite(tok[fin]).all(), f"{where}: non-finite logit"
    err = float(np.abs(tok[fin] - want[fin]).max()) if fin.any() else 0.0
    if np.isfinite(st.stop_logit):
        err = max(err, abs(float(stop) - st.stop_logit))
    else:
        assert stop == st.stop_logit, f"{where}: STOP logit {stop!r} vs {st.stop_logit!r}"
    assert err <= tol * scale, f"{where}: logit error {err:.3e} above {tol:g} x {scale:.3g}"
    return err / scale


def check_selection(KQV: np.ndarray, ctx: np.ndarray, grp_off, grp_img, caps, b_stop: float, h: int,
                    actions: Sequence[Sequence[int]], trace: Optional[np.ndarray], dtype: str,
                    no_history: bool = False, groups: Optional[Sequence[int]] = None,
                    ignore_stop: bool = False, logits: Optional[np.ndarray] = None) -> SelectReport:
    """Staged, teacher-forced check of every episode in ``groups``.

    ``actions[g]`` is the GPU's taken-candidate sequence of group g (token index,
    -1 for STOP) and ``trace[g, t]`` its step record {taken, logit, runner-up,
    STOP logit}; ``logits[g, t]`` (SP_LOGITS) the step's whole logit vector,
    token slots then STOP.  Raises AssertionError on the first violation."""
    tol = logit_tol(dtype)
    rep = SelectReport()
    T_vis = KQV.shape[0] - 2
    Kall, Qall, Vall = KQV[:, :h], KQV[:, h:2 * h], KQV[:, 2 * h:3 * h]
    start = (Kall[T_vis], Qall[T_vis], Vall[T_vis])
    k_stop = Kall[T_vis + 1]
    gs = range(len(grp_img)) if groups is None else groups
    for g in gs:
        r0, r1 = int(grp_off[g]), int(grp_off[g + 1])
        n = r1 - r0
        cap = int(caps[g])
        seq = list(actions[g])
        c = ctx[int(grp_img[g])]
        args = (Kall[r0:r1], Qall[r0:r1], Vall[r0:r1], start, k_stop, c, cap, b_stop, h)
        forced = [STOP if a == -1 else a for a in seq]
        ep = oracle.run_episode(*args, no_history=no_history, forced=forced, ignore_stop=ignore_stop)
        rep.episodes += 1
        where = f"group {g} (n={n}, cap={cap})"
        assert len(ep.steps) == len(seq), f"{where}: oracle replay took {len(ep.steps)} steps, GPU {len(seq)}"
        # The episode ended where the method ends it: at a STOP or at the cap.
        assert (seq and seq[-1] == -1) or len(seq) == cap, f"{where}: GPU episode ended early"
        assert len(set(a for a in seq if a != -1)) == sum(1 for a in seq if a != -1), f"{where}: repeat"
        exempt_here = 0
        for t, (a, st) in enumerate(zip(forced, ep.steps)):
            rep.steps += 1
            scale = _scale(st)
            v_or = st.stop_logit if a == STOP else float(st.logits[a])
            if a != st.argmax:
                assert st.margin < MARGIN_EXEMPT, (
                    f"{where} step {t + 1}: GPU took {a}, oracle argmax {st.argmax}, "
                    f"relative margin {st.margin:.3e}")
                assert st.top1 - v_or <= MARGIN_EXEMPT * scale, f"{where} step {t + 1}: not a near-tie"
                exempt_here += 1
                rep.exempt_steps += 1
                rep.divergences.append(f"{where} step {t + 1}: {a} vs {st.argmax} (margin {st.margin:.2e})")
            if trace is not None:
                rec = trace[g, t]
                taken = int(np.asarray(rec[0], np.float32).view(np.int32))
                assert taken == a or (taken == -1 and a == STOP), f"{where} step {t + 1}: trace mismatch"
                err = abs(float(rec[1]) - v_or) if np.isfinite(v_or) else 0.0
                assert _close(float(rec[1]), v_or, tol * scale), (
                    f"{where} step {t + 1}: logit {float(rec[1])!r} vs oracle {v_or!r} (scale {scale:.3g})")
                assert _close(float(rec[3]), st.stop_logit, tol * scale), (
                    f"{where} step {t + 1}: STOP logit {float(rec[3])!r} vs {st.stop_logit!r}")
                pair_gpu = sorted([float(rec[1]), float(rec[2])])
                pair_or = sorted([st.top1, st.top2])
                assert all(_close(x, y, tol * scale) for x, y in zip(pair_gpu, pair_or)), (
                    f"{where} step {t + 1}: top-2 {pair_gpu} vs {pair_or}")
                rep.max_logit_err = max(rep.max_logit_err, err / scale)
            if logits is not None:
                e = check_logit_vector(logits[g, t], st, n, tol, scale, f"{where} step {t + 1}")
                rep.max_logit_err = max(rep.max_logit_err, e)
                rep.logits_checked += int(np.isfinite(st.logits).sum()) + 1
        if exempt_here == 0:
            free = oracle.run_episode(*args, no_history=no_history, keep_steps=False,
                                      ignore_stop=ignore_stop)
            rep.free_running_checked += 1
            gpu_sel = [a for a in seq if a != -1]
            assert free.actions == gpu_sel, f"{where}: free-running oracle differs without near-ties"
            rep.free_running_equal += 1
    return rep


def _flat(seq):
    """Taken tokens of an action sequence (ints, or per-round lists)."""
    out = []
    for a in seq:
        out.extend(a if isinstance(a, (list, tuple)) else [a])
    return [a for a in out if a != -1]


def kept_from_actions(actions, grp_off, grp_img, img_off, B):
    kept = [[] for _ in range(B)]
    for g, seq in enumerate(actions):
        b = int(grp_img[g])
        base = int(grp_off[g]) - int(img_off[b])
        kept[b].extend(base + a for a in sorted(_flat(seq)))
    return kept


def check_grouped_selection(KQV: np.ndarray, ctx: np.ndarray, grp_off, grp_img, caps, b_stop: float,
                            h: int, gsize: int, rounds: Sequence[Sequence[Sequence[int]]],
                            trace: Optional[np.ndarray], dtype: str, no_history: bool = False,
                            groups: Optional[Sequence[int]] = None,
                            logits: Optional[np.ndarray] = None) -> SelectReport:
    """The staged, teacher-forced check with g = gsize tokens per round.

    ``rounds[g]`` is the GPU's round sequence of group g: per round the taken
    tokens, or [-1] for STOP; ``trace[g, r]`` its round record {taken tokens
    (-1 STOP, -3 unused slot), smallest taken logit (the STOP logit when STOP
    is taken), largest logit left out, STOP logit}."""
    tol = logit_tol(dtype)
    rep = SelectReport()
    T_vis = KQV.shape[0] - 2
    Kall, Qall, Vall = KQV[:, :h], KQV[:, h:2 * h], KQV[:, 2 * h:3 * h]
    start = (Kall[T_vis], Qall[T_vis], Vall[T_vis])
    k_stop = Kall[T_vis + 1]
    gs = range(len(grp_img)) if groups is None else groups
    for g in gs:
        r0, r1 = int(grp_off[g]), int(grp_off[g + 1])
        n = r1 - r0
        cap = int(caps[g])
        seq = [list(r) for r in rounds[g]]
        c = ctx[int(grp_img[g])]
        args = (Kall[r0:r1], Qall[r0:r1], Vall[r0:r1], start, k_stop, c, cap, b_stop, h)
        forced = [STOP if r == [-1] else r for r in seq]
        ep = oracle.run_episode(*args, no_history=no_history, forced=forced, g=gsize)
        rep.episodes += 1
        where = f"group {g} (n={n}, cap={cap}, g={gsize})"
        assert len(ep.steps) == len(seq), f"{where}: oracle replay took {len(ep.steps)} rounds, GPU {len(seq)}"
        assert (seq and seq[-1] == [-1]) or len(seq) == cap, f"{where}: GPU episode ended early"
        taken = _flat(seq)
        assert len(set(taken)) == len(taken), f"{where}: repeat"
        exempt_here = 0
        for t, (r, st) in enumerate(zip(seq, ep.steps)):
            rep.steps += 1
            scale = _scale(st)
            gpu_stop = r == [-1]
            or_stop = st.argmax == STOP
            if gpu_stop != or_stop or (not gpu_stop and sorted(r) != sorted(st.best_group)):
                near = st.margin_stop < MARGIN_EXEMPT if gpu_stop != or_stop else st.margin_member < MARGIN_EXEMPT
                assert near, (f"{where} round {t + 1}: GPU took {r}, oracle {st.best_group or 'STOP'} "
                              f"(stop margin {st.margin_stop:.3e}, member margin {st.margin_member:.3e})")
                exempt_here += 1
                rep.exempt_steps += 1
                rep.divergences.append(f"{where} round {t + 1}: {r} vs {st.best_group or 'STOP'}")
            if not gpu_stop:
                assert len(r) == min(gsize, n - sum(len(x) for x in seq[:t])), f"{where} round {t + 1}: size"
                # appended in descending-logit order
                lv = [float(st.logits[x]) for x in r]
                assert all(lv[i] >= lv[i + 1] - tol * scale for i in range(len(lv) - 1)), (
                    f"{where} round {t + 1}: group order {r} has logits {lv}")
            if trace is not None:
                rec = trace[g, t]
                ids = [int(x) for x in np.asarray(rec[:gsize], np.float32).view(np.int32)]
                if gpu_stop:
                    assert ids[0] == -1 and all(x == -3 for x in ids[1:]), f"{where} round {t + 1}: trace"
                else:
                    assert ids[:len(r)] == r and all(x == -3 for x in ids[len(r):]), (
                        f"{where} round {t + 1}: trace {ids} vs {r}")
                want_min = st.stop_logit if gpu_stop else st.group_min
                want_ru = st.runner_up
                for got, want, what in ((float(rec[gsize]), want_min, "taken"),
                                        (float(rec[gsize + 1]), want_ru, "runner-up"),
                                        (float(rec[gsize + 2]), st.stop_logit, "STOP")):
                    assert _close(got, want, tol * scale), (
                        f"{where} round {t + 1}: {what} logit {got!r} vs oracle {want!r} (scale {scale:.3g})")
                    if np.isfinite(want):
                        rep.max_logit_err = max(rep.max_logit_err, abs(got - want) / scale)
            if logits is not None:
                e = check_logit_vector(logits[g, t], st, n, tol, scale, f"{where} round {t + 1}")
                rep.max_logit_err = max(rep.max_logit_err, e)
                rep.logits_checked += int(np.isfinite(st.logits).sum()) + 1
        if exempt_here == 0:
            free = oracle.run_episode(*args, no_history=no_history, keep_steps=False, g=gsize)
            rep.free_running_checked += 1
            assert [sorted(x) for x in free.groups] == [sorted(x) for x in seq if x != [-1]], (
                f"{where}: free-running oracle differs without near-ties")
            rep.free_running_equal += 1
    return rep


TRAJ_TOL = 1e-4


@dataclass
class TrajectoryReport:
    episodes: int = 0
    max_s_err: float = 0.0
    max_kbar_err: float = 0.0
    max_pstop_err: float = 0.0


def check_trajectory(KQV: np.ndarray, ctx: np.ndarray, grp_off, grp_img, caps, b_stop: float,
                     h: int, actions: Sequence[Sequence[int]], s_gpu: np.ndarray,
                     kbar_gpu: np.ndarray, pstop_gpu: Optional[np.ndarray], tau: float,
                     beta: float, ignore_stop: bool = False, no_history: bool = False,
                     groups: Optional[Sequence[int]] = None) -> TrajectoryReport:
    """The trajectory sums of Eqs. 5-7 against the oracle, staged and
    teacher-forced like check_selection: the oracle replays the GPU's actions
    on the GPU's projected rows, so both sides sum over the same steps.

    Tolerance TRAJ_TOL = 1e-4: per group the normwise relative error of s, the
    error of K_bar relative to max(1, K_bar), and the absolute error of every
    p_t(STOP).  Staged logits agree to about 1e-6 of their scale (float32
    against float64), and p_t moves by |dl| / tau, so for tau >= 0.5 and logit
    scales up to ~20 the error stays an order of magnitude below the bar."""
    rep = TrajectoryReport()
    T_vis = KQV.shape[0] - 2
    Kall, Qall, Vall = KQV[:, :h], KQV[:, h:2 * h], KQV[:, 2 * h:3 * h]
    start = (Kall[T_vis], Qall[T_vis], Vall[T_vis])
    k_stop = Kall[T_vis + 1]
    gs = range(len(grp_img)) if groups is None else groups
    for g in gs:
        r0, r1 = int(grp_off[g]), int(grp_off[g + 1])
        n = r1 - r0
        forced = [STOP if a == -1 else a for a in actions[g]]
        tr = oracle.run_trajectory(Kall[r0:r1], Qall[r0:r1], Vall[r0:r1], start, k_stop,
                                   ctx[int(grp_img[g])], int(caps[g]), b_stop, h, tau, beta,
                                   ignore_stop=ignore_stop, no_history=no_history, forced=forced)
        where = f"group {g} (n={n})"
        assert len(tr.pstop) == len(forced), f"{where}: replay length"
        got = np.asarray(s_gpu[r0:r1], np.float64)
        den = max(float(np.linalg.norm(tr.s)), 1e-30)
        e_s = float(np.linalg.norm(got - tr.s)) / den if n else 0.0
        assert e_s <= TRAJ_TOL, f"{where}: s relative error {e_s:.3e}"
        e_k = abs(float(kbar_gpu[g]) - tr.kbar) / max(1.0, tr.kbar)
        assert e_k <= TRAJ_TOL, f"{where}: K_bar {float(kbar_gpu[g])!r} vs {tr.kbar!r}"
        if pstop_gpu is not None:
            row = np.asarray(pstop_gpu[g], np.float64)
            steps = len(tr.pstop)
            if steps:
                e_p = float(np.abs(row[:steps] - np.asarray(tr.pstop)).max())
                assert e_p <= TRAJ_TOL, f"{where}: p(STOP) error {e_p:.3e}"
                rep.max_pstop_err = max(rep.max_pstop_err, e_p)
            assert np.isnan(row[steps:]).all(), f"{where}: p(STOP) past the end"
        rep.episodes += 1
        rep.max_s_err = max(rep.max_s_err, e_s)
        rep.max_kbar_err = max(rep.max_kbar_err, e_k)
    return rep
