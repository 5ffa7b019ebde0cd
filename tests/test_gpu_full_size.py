"""The five paper-shaped batches, and the three high-resolution ones with g = 5
tokens per round (Eq. 11), at full size, launched exactly as bench.py
launches them (one stream, untraced selection kernel), checked against the
oracle on outputs it can compute one by one:

  * projection: a seeded sample of rows plus the START and STOP rows (every
    row is compared in tests/test_gpu_end_to_end.py);
  * text context: a sample of images;
  * selection: EVERY episode replayed in the oracle on the GPU's projected
    rows (tests/parity.py protocol: staged, teacher-forced on the traced
    kernel's actions, free-running when no step is a near-tie), with every
    step's whole logit vector (SP_LOGITS) compared element by element; the
    traced kernel must take the untraced (benchmarked) kernel's decisions,
    and every count and kept set must equal the traced actions;
  * compaction: three feature columns of every output row for the whole batch,
    and every column of the rows of a sample of images, bit-exact.

Tolerances are those of tests/parity.py.
"""
import gc

import numpy as np
import pytest
import torch

import oracle
from paper_2609_13804_amd import binding as sp
from paper_2609_13804_amd import workloads as W
from tests import parity

pytestmark = pytest.mark.gpu

SAMPLE_ROWS = 384
SAMPLE_IMAGES = 3
CHUNK = 64          # episodes per progress line


def _rounds(cap, n, g):
    """Rounds of an episode that never stops: the cap or ceil(n / g)."""
    return min(int(cap), -(-int(n) // g))


@pytest.mark.parametrize("name", W.PAPER_WORKLOADS + W.GROUPED_WORKLOADS)
def test_full_size_parity(gpu_lib, name):
    from paper_2609_13804_amd.runner import DeviceRun
    w = W.WORKLOADS[name]
    lay = W.make_layout(w)
    inp = W.make_inputs(w)
    b_stop = W.stop_bias(w)
    sizes = np.diff(lay.grp_off)
    steps_max = int(max(_rounds(c, n, w.g) for c, n in zip(lay.grp_cap, sizes))) + 1
    print(f"{name}: {lay.batch} images, {lay.groups} groups, {int(lay.img_off[-1])} tokens",
          flush=True)
    run = DeviceRun(w, inp, lay, b_stop, trace_steps=steps_max, logits=True)
    rng = np.random.default_rng([2609, w.cfg_id])

    # ---- the benchmark's launch sequence
    run.project()
    run.select(flags=0)
    if run.out is not None:
        run.compact()
    torch.cuda.synchronize()
    assert run.device_errors() == [0, 0, 0]
    kept = run.kept_lists()
    grp_cnt = run.grp_cnt.cpu().numpy()[:lay.groups]
    T_vis = int(lay.img_off[-1])

    # ---- projection, sampled rows
    rows = np.sort(rng.choice(T_vis, size=min(SAMPLE_ROWS, T_vis), replace=False))
    want = oracle.project(inp["X"][rows], inp["s_start"], inp["s_stop"], inp["W_kqv"], w.dtype)
    idx = torch.from_numpy(np.concatenate([rows, [T_vis, T_vis + 1]])).to(run.KQV.device)
    got = run.KQV[idx].double().cpu().numpy()
    tol = parity.logit_tol(w.dtype)
    assert parity.rows_relerr(got, want) <= tol
    if w.dtype == "bf16":
        assert np.count_nonzero(got != want) / got.size <= 1e-2

    # ---- text context, sampled images
    imgs = sorted({0, lay.batch - 1} | set(int(b) for b in rng.choice(lay.batch, SAMPLE_IMAGES)))
    ctx = run.ctx.double().cpu().numpy()
    for b in imgs:
        t0, t1 = int(lay.text_off[b]), int(lay.text_off[b + 1])
        c = oracle.text_context(inp["E_text"][t0:t1], np.array([0, t1 - t0]), inp["W_text"])
        assert parity.rows_relerr(ctx[b:b + 1], c) <= 1e-5, f"image {b}"

    # ---- selection: the traced kernel (with the logit dump) decides as the
    # benchmarked one did
    run.select(flags=run.flags)
    torch.cuda.synchronize()
    assert run.device_errors() == [0, 0, 0]
    actions = run.trace_actions()
    assert run.kept_lists() == kept
    assert kept == parity.kept_from_actions(actions, lay.grp_off, lay.grp_img, lay.img_off,
                                            lay.batch)
    assert grp_cnt.tolist() == [len(parity._flat(s)) for s in actions]
    stop = -1 if w.g == 1 else [-1]
    for g, s in enumerate(actions):
        r = _rounds(lay.grp_cap[g], sizes[g], w.g)
        assert (s and s[-1] == stop and len(s) <= r + 1) or len(s) == int(lay.grp_cap[g]), g
    steps = np.array([len(s) for s in actions])

    # ---- every episode against the oracle, on the GPU's projected rows
    KQV = run.KQV.float().cpu().numpy()          # exact: bf16 and f32 widen to f32
    trace = run.trace.cpu().numpy()
    logits = run.trace_logits()
    total = parity.SelectReport()
    for c0 in range(0, lay.groups, CHUNK):
        chunk = range(c0, min(lay.groups, c0 + CHUNK))
        if w.g == 1:
            rep = parity.check_selection(KQV, ctx, lay.grp_off, lay.grp_img, lay.grp_cap, b_stop,
                                         w.h, actions, trace, w.dtype, groups=chunk, logits=logits)
        else:
            rep = parity.check_grouped_selection(KQV, ctx, lay.grp_off, lay.grp_img, lay.grp_cap,
                                                 b_stop, w.h, w.g, actions, trace, w.dtype,
                                                 groups=chunk, logits=logits)
        for f in ("episodes", "steps", "exempt_steps", "logits_checked", "free_running_equal",
                  "free_running_checked"):
            setattr(total, f, getattr(total, f) + getattr(rep, f))
        total.max_logit_err = max(total.max_logit_err, rep.max_logit_err)
        total.divergences += rep.divergences
        print(f"{name}: episodes {c0}..{chunk[-1]} checked", flush=True)
    assert total.episodes == lay.groups
    print(f"{name}: checked {total.episodes} of {lay.groups} episodes ({total.steps} steps, longest "
          f"{int(steps.max())}; {total.logits_checked} logits element by element), "
          f"{total.exempt_steps} exempt, max logit err {total.max_logit_err:.2e}, free-running "
          f"equal {total.free_running_equal}/{total.free_running_checked}; kept total "
          f"{sum(map(len, kept))}", flush=True)
    for d in total.divergences:
        print(f"{name}: near-tie {d}", flush=True)
    del KQV, trace, logits

    # ---- compaction
    if run.out is not None:
        cols = [0, w.d // 2, w.d - 1]
        out_cols = run.out[:, cols].float().cpu().numpy()
        want_cols, seq = oracle.compact(inp["X"][:, cols], lay.img_off, inp["E_text"][:, cols],
                                        lay.text_off, kept, w.layout, lay.rows_per_image,
                                        np.zeros((run.out_rows, len(cols))))
        assert np.array_equal(out_cols, want_cols.astype(np.float32))
        assert run.seq_info.cpu().numpy().tolist() == seq.tolist()
        for b in imgs:
            i0, i1 = int(lay.img_off[b]), int(lay.img_off[b + 1])
            t0, t1 = int(lay.text_off[b]), int(lay.text_off[b + 1])
            n_rows = len(kept[b]) + t1 - t0
            base = b * lay.rows_per_image if w.layout == "padded" else int(seq[b])
            got_rows = run.out[base:base + n_rows].float().cpu().numpy()
            want_rows, _ = oracle.compact(inp["X"][i0:i1], np.array([0, i1 - i0]),
                                          inp["E_text"][t0:t1], np.array([0, t1 - t0]), [kept[b]],
                                          "packed", 0, np.zeros((n_rows, w.d)))
            assert np.array_equal(got_rows, want_rows.astype(np.float32)), f"image {b}"
    del run, inp
    gc.collect()
    torch.cuda.empty_cache()
