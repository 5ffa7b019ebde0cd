"""HIP path vs the CPU oracle, element by element, on small workloads that span
several GEMM tiles, ragged groups and ragged tails (oracle in seconds).

All calls go through the C ABI (paper_2609_13804_amd.binding); see
tests/parity.py for the tolerances.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2609_13804_amd import workloads as W
from tests import parity

pytestmark = pytest.mark.gpu

SMALL = W.SMALL_WORKLOADS


def _setup(name, b_stop=None, caps=None, flags=0, trace=True, images=None):
    from paper_2609_13804_amd.runner import DeviceRun
    w = W.WORKLOADS[name]
    inp = W.make_inputs(w, images)
    lay = W.make_layout(w, images)
    b = W.stop_bias(w) if b_stop is None else b_stop
    c = lay.grp_cap if caps is None else np.asarray(caps, np.int32)
    steps = int(max(min(int(x), int(n)) for x, n in zip(c, np.diff(lay.grp_off)))) + 1 if trace else 0
    run = DeviceRun(w, inp, lay, b, trace_steps=steps, flags=flags, caps=c, logits=trace)
    return w, inp, lay, run


def _logits(run):
    """The SP_LOGITS dump of a traced run (every step's whole logit vector)."""
    from paper_2609_13804_amd import binding as sp
    return run.trace_logits() if run.flags & sp.SP_LOGITS else None


def _staged(run):
    KQV = run.KQV.double().cpu().numpy()
    ctx = run.ctx.double().cpu().numpy()
    return KQV, ctx


def _check_errors(run):
    assert run.device_errors() == [0, 0, 0]


@pytest.mark.parametrize("name", SMALL)
def test_projection_parity(gpu_lib, name):
    w, inp, lay, run = _setup(name, trace=False)
    run.project()
    torch.cuda.synchronize()
    _check_errors(run)
    KQV_or = oracle.project(inp["X"], inp["s_start"], inp["s_stop"], inp["W_kqv"], w.dtype)
    ctx_or = oracle.text_context(inp["E_text"], lay.text_off, inp["W_text"])
    KQV, ctx = _staged(run)
    tol = 1e-3 if w.dtype == "bf16" else 1e-5
    assert parity.rows_relerr(KQV, KQV_or) <= tol
    assert parity.rows_relerr(ctx, ctx_or) <= 1e-5
    # Stored values differ from the oracle's single rounding only where the
    # float32 accumulation error crosses a rounding boundary: rarely.
    differ = np.count_nonzero(KQV != KQV_or) / KQV.size
    print(f"{name}: {differ:.2e} of projected values differ from the oracle's rounding")
    if w.dtype == "bf16":
        assert differ <= 1e-2


@pytest.mark.parametrize("name", SMALL)
def test_selection_and_compaction_parity(gpu_lib, name):
    w, inp, lay, run = _setup(name)
    run.run()
    torch.cuda.synchronize()
    _check_errors(run)
    KQV, ctx = _staged(run)
    actions = run.trace_actions()
    tr = run.trace.cpu().numpy()
    rep = parity.check_selection(KQV, ctx, lay.grp_off, lay.grp_img, run.caps_host, run.b_stop,
                                 w.h, actions, tr, w.dtype, logits=_logits(run))
    print(f"{name}: {rep.episodes} episodes, {rep.steps} steps, {rep.exempt_steps} exempt, "
          f"max logit err {rep.max_logit_err:.2e}")
    kept = run.kept_lists()
    assert kept == parity.kept_from_actions(actions, lay.grp_off, lay.grp_img, lay.img_off, lay.batch)
    assert run.grp_cnt.cpu().numpy()[:lay.groups].tolist() == [sum(1 for a in s if a != -1) for s in actions]
    if run.out is not None:
        out_gpu = run.out.float().cpu().numpy()
        out_or, seq_or = oracle.compact(inp["X"], lay.img_off, inp["E_text"], lay.text_off, kept,
                                        w.layout, lay.rows_per_image, np.zeros_like(out_gpu))
        assert np.array_equal(out_gpu, out_or.astype(np.float32))
        assert run.seq_info.cpu().numpy().tolist() == seq_or.tolist()


@pytest.mark.parametrize("name", ["tiny_bf16", "tiny_f32"])
def test_trace_and_plain_kernels_agree(gpu_lib, name):
    """The traced and untraced selection kernels take the same decisions, and a
    second run gives bit-identical results."""
    w, inp, lay, run = _setup(name)
    run.run()
    kept_trace = run.kept_lists()
    run.select(flags=0)
    kept_plain = run.kept_lists()
    out1 = run.out.clone() if run.out is not None else None
    run.run()
    torch.cuda.synchronize()
    assert kept_trace == kept_plain == run.kept_lists()
    if out1 is not None:
        assert torch.equal(out1, run.out)


@pytest.mark.parametrize("name", ["tiny_bf16", "small_packed_bf16"])
def test_two_phase_selection_matches_one_call(gpu_lib, name):
    """SP_GRAM_ONLY then SP_REUSE_GRAM (the pipeline's split) gives the one
    call's kept lists and trace, bit for bit; the first phase writes no output."""
    from paper_2609_13804_amd import binding as sp
    w, inp, lay, run = _setup(name)
    run.run()
    torch.cuda.synchronize()
    kept, tr = run.kept_lists(), run.trace.clone()
    run.kept_cnt.fill_(-7)
    run.select(flags=run.flags | sp.SP_GRAM_ONLY)
    torch.cuda.synchronize()
    assert (run.kept_cnt.cpu().numpy() == -7).all()
    run.select(flags=run.flags | sp.SP_REUSE_GRAM)
    torch.cuda.synchronize()
    _check_errors(run)
    assert run.kept_lists() == kept
    # bitwise: records past an episode's end hold int32 -2, a NaN as float
    assert torch.equal(run.trace.view(torch.int32), tr.view(torch.int32))


def test_immediate_stop(gpu_lib):
    """b_stop = +inf: every episode stops at its first step (K = 0) and the
    prefill holds only the prompt rows."""
    w, inp, lay, run = _setup("tiny_bf16", b_stop=math.inf)
    run.run()
    torch.cuda.synchronize()
    _check_errors(run)
    assert not run.kept_cnt.cpu().numpy().any()
    assert all(s == [-1] for s in run.trace_actions())
    L = np.diff(lay.text_off)
    assert run.seq_info.cpu().numpy().tolist() == L.tolist()


def test_never_stop_is_identity(gpu_lib):
    """b_stop = -inf and caps above the group sizes: every token is kept and the
    compacted sequence of each image is [X_b; E_b] bit for bit."""
    w0 = W.WORKLOADS["tiny_bf16"]
    lay0 = W.make_layout(w0)
    caps = np.diff(lay0.grp_off) + 3
    w, inp, lay, run = _setup("tiny_bf16", b_stop=-math.inf, caps=caps)
    run.run()
    torch.cuda.synchronize()
    _check_errors(run)
    out = run.out.float().cpu().numpy()
    for b in range(lay.batch):
        want = np.vstack([inp["X"][lay.img_off[b]:lay.img_off[b + 1]],
                          inp["E_text"][lay.text_off[b]:lay.text_off[b + 1]]])
        base = b * lay.rows_per_image
        assert np.array_equal(out[base:base + len(want)], want)
    KQV, ctx = _staged(run)
    parity.check_selection(KQV, ctx, lay.grp_off, lay.grp_img, caps, -math.inf, w.h,
                           run.trace_actions(), run.trace.cpu().numpy(), w.dtype,
                           logits=_logits(run))


def test_no_history_is_topk(gpu_lib):
    """SP_NO_HISTORY: the selector collapses to top-K of the first-step logits
    (Eq. 1), checked against torch.topk on the GPU's own first-step logits."""
    from paper_2609_13804_amd import binding as sp
    w, inp, lay, run = _setup("tiny_f32", flags=sp.SP_NO_HISTORY)
    run.run()
    torch.cuda.synchronize()
    _check_errors(run)
    KQV, ctx = _staged(run)
    actions = run.trace_actions()
    parity.check_selection(KQV, ctx, lay.grp_off, lay.grp_img, run.caps_host, run.b_stop, w.h,
                           actions, run.trace.cpu().numpy(), w.dtype, no_history=True,
                           logits=_logits(run))
    h = w.h
    T_vis = KQV.shape[0] - 2
    for g, seq in enumerate(actions):
        r0, r1 = lay.grp_off[g], lay.grp_off[g + 1]
        u = torch.from_numpy(ctx[lay.grp_img[g]] + KQV[T_vis, h:2 * h] + KQV[T_vis, 2 * h:])
        l1 = torch.from_numpy(KQV[r0:r1, :h]) @ u / math.sqrt(h)
        stop = float(torch.from_numpy(KQV[T_vis + 1, :h]) @ u / math.sqrt(h)) + run.b_stop
        k = min(int(run.caps_host[g]), int((l1 > stop).sum()))
        order = torch.sort(l1, descending=True, stable=True).indices[:k].tolist()
        assert [a for a in seq if a != -1] == order


def test_duplicate_rows_identical_logits(gpu_lib):
    """Two tokens with bit-identical rows get bit-identical logits on the GPU, so
    the lower index is taken first (exact tie rule)."""
    w = W.WORKLOADS["tiny_bf16"]
    inp = W.make_inputs(w)
    lay = W.make_layout(w)
    X = inp["X"].copy()
    g0 = int(lay.grp_off[0])
    for dst, src in ((g0 + 5, g0 + 1), (g0 + 40, g0 + 2), (g0 + 41, g0 + 40)):
        X[dst] = X[src]
    inp["X"] = X
    from paper_2609_13804_amd.runner import DeviceRun
    steps = int(lay.grp_cap.max()) + 1
    run = DeviceRun(w, inp, lay, -math.inf, trace_steps=steps)
    run.run()
    torch.cuda.synchronize()
    seq = run.trace_actions()[0]
    for lo, hi in ((1, 5), (2, 40), (2, 41), (40, 41)):
        if hi in seq:
            assert lo in seq and seq.index(lo) < seq.index(hi)
    KQV, ctx = _staged(run)
    parity.check_selection(KQV, ctx, lay.grp_off, lay.grp_img, run.caps_host, -math.inf, w.h,
                           run.trace_actions(), run.trace.cpu().numpy(), w.dtype,
                           logits=_logits(run))


@pytest.mark.parametrize("name", ["mid_bf16", "mid_g5_bf16"])
def test_permutation_equivariance_is_bit_exact(gpu_lib, name):
    """Permuting the tokens inside each group permutes the decisions and leaves
    every traced logit bit-identical (pin P8 on the GPU): a token's projected
    row and its Gram entries are accumulated in the same order wherever the
    token sits, and the history sums run in history order (with g = 5 a
    round's tokens enter it in descending-logit order).  Columns 512 and up of
    a 576-token group are summed in quarters by other lanes, so tokens are
    permuted within [0, 512) and within [512, n) separately."""
    from paper_2609_13804_amd.runner import DeviceRun
    w = W.WORKLOADS[name]
    inp = W.make_inputs(w)
    lay = W.make_layout(w)
    steps = int(lay.grp_cap.max()) + 1
    rng = np.random.default_rng(8808)
    P = np.arange(int(lay.img_off[-1]))
    local = []
    for g in range(lay.groups):
        g0, g1 = int(lay.grp_off[g]), int(lay.grp_off[g + 1])
        perm = np.arange(g1 - g0)
        for lo, hi in ((0, min(512, g1 - g0)), (512, g1 - g0)):
            if hi > lo:
                perm[lo:hi] = lo + rng.permutation(hi - lo)
        P[g0:g1] = g0 + perm
        local.append(perm)              # new position p holds old token perm[p]
    res = []
    for X in (inp["X"], inp["X"][P]):
        run = DeviceRun(w, dict(inp, X=X), lay, W.stop_bias(w), trace_steps=steps)
        run.run()
        torch.cuda.synchronize()
        _check_errors(run)
        res.append((run.trace_actions(), run.trace.cpu().numpy().copy()))
        del run
    (a0, t0), (a1, t1) = res
    k = w.g                             # trace slots holding taken tokens
    for g in range(lay.groups):
        new_pos = np.argsort(local[g])  # old token -> new position
        n = len(a0[g])
        assert n > 1
        # no decision rested on an exact tie: the (smallest) taken logit is
        # strictly above the best candidate left out
        assert np.all(t0[g, :n, k] != t0[g, :n, k + 1]), g
        if k == 1:
            want = [int(new_pos[x]) if x >= 0 else -1 for x in a0[g]]
        else:
            want = [[int(new_pos[x]) if x >= 0 else -1 for x in r] for r in a0[g]]
        assert a1[g] == want, g
        assert np.array_equal(t1[g, :n, k:].view(np.uint32), t0[g, :n, k:].view(np.uint32)), g


def test_zero_caps_and_episode_independence(gpu_lib):
    """Cap 0 gives an empty episode without any step; a sub-batch in another
    order gives the same per-image results (episodes are independent)."""
    w, inp, lay, run = _setup("tiny_bf16")
    run.run()
    torch.cuda.synchronize()
    full = run.kept_lists()
    caps = lay.grp_cap.copy()
    caps[::2] = 0
    w2, inp2, lay2, run2 = _setup("tiny_bf16", caps=caps)
    run2.run()
    torch.cuda.synchronize()
    _check_errors(run2)
    acts = run2.trace_actions()
    for g in range(0, lay.groups, 2):
        assert acts[g] == []
    sub = [3, 1]
    w3, inp3, lay3, run3 = _setup("tiny_bf16", images=sub)
    run3.run()
    torch.cuda.synchronize()
    assert run3.kept_lists() == [full[i] for i in sub]


def test_images_without_groups(gpu_lib):
    """Images of 0 tokens have no group (fixed partitions): their kept counts
    are 0 even over a dirty output, the other images' kept lists match the
    oracle, and a batch with no group at all gives all-zero counts."""
    from paper_2609_13804_amd.runner import DeviceRun
    w = W.Workload("empty_images", 109, batch=6, d=256, d_text=256, h=128, dtype="bf16",
                   text_len=5, tokens=(0, 200, 0, 0, 150, 0), grouping="fixed", group_size=96,
                   cap=20, layout="padded", description="images without tokens")
    lay, inp = W.make_layout(w), W.make_inputs(w)
    assert lay.groups == 5 and list(lay.grp_img) == [1, 1, 1, 4, 4]
    run = DeviceRun(w, inp, lay, 0.5, trace_steps=21)
    run.project()
    run.kept_cnt.fill_(77)
    run.select()
    torch.cuda.synchronize()
    _check_errors(run)
    cnt = run.kept_cnt.cpu().numpy().tolist()
    assert [cnt[b] for b in (0, 2, 3, 5)] == [0, 0, 0, 0]
    KQV, ctx = _staged(run)
    actions = run.trace_actions()
    parity.check_selection(KQV, ctx, lay.grp_off, lay.grp_img, run.caps_host, run.b_stop, w.h,
                           actions, run.trace.cpu().numpy(), w.dtype, logits=_logits(run))
    assert run.kept_lists() == parity.kept_from_actions(actions, lay.grp_off, lay.grp_img,
                                                        lay.img_off, lay.batch)
    w0 = W.Workload("no_groups", 110, batch=2, d=256, d_text=256, h=128, dtype="bf16",
                    text_len=5, tokens=(0, 0), grouping="fixed", group_size=96, cap=20,
                    layout="padded", description="no visual token at all")
    lay0, inp0 = W.make_layout(w0), W.make_inputs(w0)
    assert lay0.groups == 0
    run0 = DeviceRun(w0, inp0, lay0, 0.5)
    run0.project()
    run0.kept_cnt.fill_(77)
    run0.select()
    torch.cuda.synchronize()
    _check_errors(run0)
    assert run0.kept_cnt.cpu().numpy().tolist() == [0, 0]


@pytest.mark.parametrize("dtype,layout", [("bf16", "padded"), ("f32", "packed")])
def test_batch_without_text(gpu_lib, dtype, layout):
    """No text token in the batch (T_txt = 0): no text tile or LayerNorm runs,
    every context is zero (the pooled mean over an empty set, as the oracle
    defines it), and the projection, the selection and the prefill buffer
    (visual rows only) match the oracle.  The STOP bias keeps about half of
    what the caps allow, placed by the oracle's calibration."""
    from paper_2609_13804_amd.runner import DeviceRun
    w = W.Workload(f"no_text_{dtype}", 111 if dtype == "bf16" else 112, batch=3, d=256,
                   d_text=256, h=128, dtype=dtype, text_len=0, tokens=(200, 37, 150), cap=30,
                   layout=layout, description="no text tokens")
    lay, inp = W.make_layout(w), W.make_inputs(w)
    assert int(lay.text_off[-1]) == 0 and inp["E_text"].shape[0] == 0
    KQV_or = oracle.project(inp["X"], inp["s_start"], inp["s_stop"], inp["W_kqv"], w.dtype)
    ctx_or = oracle.text_context(inp["E_text"], lay.text_off, inp["W_text"])
    assert not ctx_or.any()
    pm = oracle.stop_thresholds(KQV_or, ctx_or, lay.grp_off, lay.grp_img, lay.grp_cap, w.h)
    b_stop, _ = oracle.choose_stop_bias(pm, 0.5 * sum(len(x) for x in pm))
    steps = int(max(min(int(c), int(n)) for c, n in zip(lay.grp_cap, np.diff(lay.grp_off)))) + 1
    run = DeviceRun(w, inp, lay, b_stop, trace_steps=steps, logits=True)
    run.run()
    torch.cuda.synchronize()
    _check_errors(run)
    KQV, ctx = _staged(run)
    assert not ctx.any()
    assert parity.rows_relerr(KQV, KQV_or) <= (1e-3 if dtype == "bf16" else 1e-5)
    actions = run.trace_actions()
    rep = parity.check_selection(KQV, ctx, lay.grp_off, lay.grp_img, run.caps_host, run.b_stop, w.h,
                                 actions, run.trace.cpu().numpy(), w.dtype, logits=_logits(run))
    kept = run.kept_lists()
    assert kept == parity.kept_from_actions(actions, lay.grp_off, lay.grp_img, lay.img_off, lay.batch)
    assert 0 < sum(map(len, kept)) < int(lay.img_off[-1])
    out_gpu = run.out.float().cpu().numpy()
    out_or, seq_or = oracle.compact(inp["X"], lay.img_off, inp["E_text"], lay.text_off, kept,
                                    w.layout, lay.rows_per_image, np.zeros_like(out_gpu))
    assert np.array_equal(out_gpu, out_or.astype(np.float32))
    assert run.seq_info.cpu().numpy().tolist() == seq_or.tolist()
    print(f"no text ({dtype}, {layout}): {rep.episodes} episodes, {rep.steps} steps, kept "
          f"{[len(k) for k in kept]}", flush=True)


def test_device_error_on_oversized_group(gpu_lib):
    """A group larger than the stated max_group is reported through the device
    error word and no kernel reads past its buffers."""
    from paper_2609_13804_amd.runner import DeviceRun
    from paper_2609_13804_amd import binding as sp
    w = W.WORKLOADS["tiny_bf16"]
    inp = W.make_inputs(w)
    lay = W.make_layout(w)
    run = DeviceRun(w, inp, lay, 1.0, max_group=int(np.diff(lay.grp_off).max()) - 1)
    run.project()
    run.select()
    torch.cuda.synchronize()
    assert sp.stepprune_read_device_error(run.ws[1]) == sp.SP_DEV_GROUP_TOO_LARGE
    assert sp.stepprune_read_device_error(run.ws[1]) == 0     # read clears it


@pytest.mark.parametrize("case", ["negative_cap", "cap_above_max", "group_outside_image",
                                  "text_offsets_decrease", "packed_output_too_small"])
def test_device_errors_from_bad_data(gpu_lib, case):
    """Data that only the device sees (offsets, caps, counts) and that is
    inconsistent is caught by the kernels' own checks: the stage records the
    documented SP_DEV_* code in its workspace, and reading it clears it.  Each
    case corrupts one device array after a valid set-up; every kernel still
    reads and writes inside its buffers."""
    from paper_2609_13804_amd import binding as sp
    name = "small_packed_bf16" if case == "packed_output_too_small" else "tiny_bf16"
    w, inp, lay, run = _setup(name, trace=False)
    if case == "text_offsets_decrease":
        run.text_off[2] = int(lay.text_off[1]) - 1
        run.project()
        torch.cuda.synchronize()
        assert sp.stepprune_read_device_error(run.ws[0]) == sp.SP_DEV_BAD_OFFSETS
        assert not run.ctx[1].any()          # the image with no valid text gets c = 0
        assert sp.stepprune_read_device_error(run.ws[0]) == 0
        return
    run.project()
    if case == "negative_cap":
        run.grp_cap[1] = -1
        want, stage = sp.SP_DEV_BAD_CAP, 1
    elif case == "cap_above_max":
        run.grp_cap[0] = 10 ** 6             # min(cap, n) exceeds the stated max_cap
        want, stage = sp.SP_DEV_BAD_CAP, 1
    elif case == "group_outside_image":
        run.grp_img[0] = 1                   # group 0's rows lie in image 0
        want, stage = sp.SP_DEV_BAD_OFFSETS, 1
    else:
        run.select()
        torch.cuda.synchronize()
        _check_errors(run)
        run.compact()
        torch.cuda.synchronize()
        need = int(run.seq_info[-1])         # rows the packed buffer needs
        sp.stepprune_compact(run.dims, run.X, run.img_off, run.E, run.text_off, run.kept_idx,
                             run.kept_off, run.kept_cnt, run.sizes.B, run.layout_code, 0,
                             need - 1, run.out, run.seq_info, run.ws[2], run.ws_bytes[2])
        want, stage = sp.SP_DEV_OUTPUT_OVERFLOW, 2
    if stage == 1:
        run.select()
    torch.cuda.synchronize()
    assert sp.stepprune_read_device_error(run.ws[stage]) == want
    assert sp.stepprune_read_device_error(run.ws[stage]) == 0


def test_long_episodes_cross_every_history_tier(gpu_lib):
    """Episodes far longer than the register-resident history: caps of 400 on
    576-token groups with STOP disabled, so the history passes the register
    slots, the LDS rows and the re-read tier; every step still matches the
    oracle (staged, teacher-forced)."""
    w0 = W.WORKLOADS["mid_bf16"]
    lay0 = W.make_layout(w0)
    caps = np.minimum(np.diff(lay0.grp_off), 400)
    w, inp, lay, run = _setup("mid_bf16", b_stop=-math.inf, caps=caps)
    run.run()
    torch.cuda.synchronize()
    _check_errors(run)
    KQV, ctx = _staged(run)
    actions = run.trace_actions()
    assert [len(a) for a in actions] == [int(c) if c <= n else int(n) + 1
                                         for c, n in zip(caps, np.diff(lay.grp_off))]
    rep = parity.check_selection(KQV, ctx, lay.grp_off, lay.grp_img, caps, -math.inf, w.h,
                                 actions, run.trace.cpu().numpy(), w.dtype, logits=_logits(run))
    print(f"long episodes: {rep.steps} steps, {rep.exempt_steps} exempt, "
          f"max logit err {rep.max_logit_err:.2e}")


def test_pipeline_slots_agree_with_one_stream(gpu_lib):
    """runner.Pipeline (projections on one stream, selections and compactions
    on three streams over four buffer slots, events between them) gives every
    slot the single-stream run's kept lists and prefill buffer, bit for bit,
    in both schedules."""
    from paper_2609_13804_amd.runner import Pipeline
    for split in (False, True):
        w, inp, lay, run = _setup("small_packed_bf16", trace=False)
        run.run()
        torch.cuda.synchronize()
        want_kept, want_out = run.kept_lists(), run.out.clone()
        for r_ in [run]:
            r_.kept_idx.fill_(-1)
            r_.out.zero_()
        pipe = Pipeline(run, slots=4, streams=3, split_gram=split)
        for _ in range(9):
            pipe.issue()
        torch.cuda.synchronize()
        for r_ in pipe.runs:
            assert r_.device_errors() == [0, 0, 0]
            assert r_.kept_lists() == want_kept
            assert torch.equal(r_.out, want_out)
