"""Grouped selection on the GPU (Eq. 11; Algorithm 1 step 3c): g tokens per
round, checked round by round against the oracle with the tests/parity.py
protocol (staged, teacher-forced, set equality per round with near-ties
counted; compaction bit-exact).

Covers every launch shape of the grouped kernel (lane columns, second
columns past 512, 16-wave groups past 576), histories long enough to pass
the register slots, the LDS rows and the re-read tier, the traced and
untraced kernels, the no-history variant, and g = 2..5.
"""
import dataclasses
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2609_13804_amd import binding as sp
from paper_2609_13804_amd import workloads as W
from tests import parity

pytestmark = pytest.mark.gpu


def _rounds_bound(caps, sizes, g):
    return int(max(min(int(c), -(-int(n) // g)) for c, n in zip(caps, sizes))) + 1


def _setup(w, b_stop=None, caps=None, flags=0, trace=True):
    from paper_2609_13804_amd.runner import DeviceRun
    inp = W.make_inputs(w)
    lay = W.make_layout(w)
    b = W.stop_bias(w) if b_stop is None else b_stop
    c = lay.grp_cap if caps is None else np.asarray(caps, np.int32)
    steps = _rounds_bound(c, np.diff(lay.grp_off), w.g) if trace else 0
    run = DeviceRun(w, inp, lay, b, trace_steps=steps, flags=flags, caps=c, logits=trace)
    return inp, lay, run


def _check(w, inp, lay, run, no_history=False, compact=True):
    assert run.device_errors() == [0, 0, 0]
    KQV = run.KQV.double().cpu().numpy()
    ctx = run.ctx.double().cpu().numpy()
    rounds = run.trace_actions()
    rep = parity.check_grouped_selection(KQV, ctx, lay.grp_off, lay.grp_img, run.caps_host,
                                         run.b_stop, w.h, w.g, rounds, run.trace.cpu().numpy(),
                                         w.dtype, no_history=no_history,
                                         logits=run.trace_logits() if run.flags & sp.SP_LOGITS
                                         else None)
    kept = run.kept_lists()
    assert kept == parity.kept_from_actions(rounds, lay.grp_off, lay.grp_img, lay.img_off, lay.batch)
    assert run.grp_cnt.cpu().numpy()[:lay.groups].tolist() == [len(parity._flat(s)) for s in rounds]
    if compact and run.out is not None:
        out_gpu = run.out.float().cpu().numpy()
        out_or, seq_or = oracle.compact(inp["X"], lay.img_off, inp["E_text"], lay.text_off, kept,
                                        w.layout, lay.rows_per_image, np.zeros_like(out_gpu))
        assert np.array_equal(out_gpu, out_or.astype(np.float32))
        assert run.seq_info.cpu().numpy().tolist() == seq_or.tolist()
    print(f"{w.name} g={w.g}: {rep.episodes} episodes, {rep.steps} rounds, {rep.exempt_steps} exempt, "
          f"max logit err {rep.max_logit_err:.2e}, kept {[len(k) for k in kept]}")
    return rounds, kept


@pytest.mark.parametrize("name", W.GROUPED_SMALL_WORKLOADS)
def test_grouped_selection_and_compaction_parity(gpu_lib, name):
    w = W.WORKLOADS[name]
    inp, lay, run = _setup(w)
    run.run()
    torch.cuda.synchronize()
    _check(w, inp, lay, run)


@pytest.mark.parametrize("name", W.GROUPED_SMALL_WORKLOADS)
def test_grouped_trace_and_plain_kernels_agree(gpu_lib, name):
    """The untraced kernel (the benchmark's; it ranks g candidates per wave,
    the traced one g + 1) takes the same decisions, bit for bit on reruns."""
    from paper_2609_13804_amd import binding as sp
    w = W.WORKLOADS[name]
    inp, lay, run = _setup(w)
    run.run()
    torch.cuda.synchronize()
    traced = run.kept_lists()
    run.select(flags=0)
    torch.cuda.synchronize()
    assert run.device_errors() == [0, 0, 0]
    plain = run.kept_lists()
    run.select(flags=run.flags)
    torch.cuda.synchronize()
    assert traced == plain == run.kept_lists()


@pytest.mark.parametrize("g", [2, 3, 4, 5])
def test_every_group_size(gpu_lib, g):
    """g = 2..5 on the ragged tiny fp32 batch (a 3-token image: g >= n)."""
    w = dataclasses.replace(W.WORKLOADS["tiny_g5_f32"], g=g)
    inp, lay, run = _setup(w, b_stop=W.stop_bias(W.WORKLOADS["tiny_g5_f32"]))
    run.run()
    torch.cuda.synchronize()
    _check(w, inp, lay, run)


def test_grouped_long_rounds_cross_every_history_tier(gpu_lib):
    """STOP disabled and caps past ceil(n / g): every token is taken, 5 per
    round, so a 576-token group's history passes the register slots, the LDS
    rows and the re-read tier, and ends with a STOP round with no candidate
    left."""
    w = W.WORKLOADS["mid_g5_bf16"]
    lay0 = W.make_layout(w)
    sizes = np.diff(lay0.grp_off)
    caps = np.full(len(sizes), 130, np.int32)
    inp, lay, run = _setup(w, b_stop=-math.inf, caps=caps)
    run.run()
    torch.cuda.synchronize()
    rounds, kept = _check(w, inp, lay, run)
    assert [len(r) for r in rounds] == [-(-int(n) // 5) + 1 for n in sizes]
    assert kept == [list(range(int(n))) for n in sizes]


def test_grouped_no_history(gpu_lib):
    """SP_NO_HISTORY: the query stays START's, so every round takes the next
    g tokens of one fixed order."""
    from paper_2609_13804_amd import binding as sp
    w = W.WORKLOADS["small_g5_bf16"]
    inp, lay, run = _setup(w, flags=sp.SP_NO_HISTORY)
    run.run()
    torch.cuda.synchronize()
    _check(w, inp, lay, run, no_history=True)


GROUP_SHAPES = [
    # (name, cfg id, tokens per image, round cap, STOP bias)
    ("g5_wide_1000", 111, (1000, 700, 33), 30, -math.inf),
    ("g5_wide_1000_stop", 111, (1000, 700, 33), 30, 0.64),   # STOPs after 5 and 30 tokens
    ("g5_second_cols_576", 112, (576, 513, 512, 65), 40, 0.25),
    ("g5_second_cols_deep", 113, (513, 576), 110, -math.inf),
    ("g5_lanes_512", 114, (512, 448, 64, 1), 20, 0.1),
]


@pytest.mark.parametrize("name,cfg,tokens,cap,b_stop", GROUP_SHAPES, ids=[c[0] for c in GROUP_SHAPES])
def test_grouped_group_shapes(gpu_lib, name, cfg, tokens, cap, b_stop):
    """The grouped kernel at each launch shape, traced and untraced."""
    from paper_2609_13804_amd import binding as sp
    w = W.Workload(name, cfg, batch=len(tokens), d=256, d_text=256, h=128, dtype="bf16",
                   text_len=5, tokens=tokens, cap=cap, g=5, layout="padded",
                   description="grouped group-shape edge case")
    inp, lay, run = _setup(w, b_stop=b_stop)
    run.project()
    run.select(flags=0)
    torch.cuda.synchronize()
    assert run.device_errors() == [0, 0, 0]
    plain = run.kept_lists()
    run.select(flags=run.flags)
    run.compact()
    torch.cuda.synchronize()
    _, kept = _check(w, inp, lay, run)
    assert kept == plain
