"""Seeded random batch shapes through the C ABI against the oracle.

Sixteen cases drawn once from a fixed seed mix what the fixed workloads keep
apart: float32 and bfloat16, widths d and h, one to three images of 1 to
1500 tokens, single, fixed-size and balanced groups (up to 1022 tokens, so
all three of the selection kernel's layouts occur), caps from 1 round to
every token, 1 to 5 tokens per round, padded and packed prefill buffers.
Each case's STOP bias is placed by the oracle's calibration (on its own
projection) between two adjacent breakpoints, at a random retained fraction.

Per case (tests/parity.py protocol): the untraced and traced kernels take the
same decisions; the oracle replays every episode on the GPU's projected rows
with every step's whole logit vector compared element by element; the kept
lists follow from the traced actions; the prefill buffer matches the oracle's
compaction exactly.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_13804_amd import workloads as W
from tests import parity

pytestmark = pytest.mark.gpu


def _cases(n=16, seed=20260913):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        dtype = "f32" if rng.random() < 0.35 else "bf16"
        d = int(rng.choice([128, 192, 256, 320, 512]))
        h = int(rng.choice([64, 128, 192, 256, 512]))
        grouping = str(rng.choice(["single", "fixed", "balanced"]))
        group_size = int(rng.choice([64, 200, 256, 512, 520, 576, 700, 1022]))
        B = int(rng.integers(1, 4))
        hi = 1022 if grouping == "single" else 1500
        sizes = tuple(int(x) for x in rng.integers(1, hi + 1, size=B))
        if grouping == "balanced":
            sizes = tuple(max(4, 4 * (s // 4)) for s in sizes)
        g = int(rng.choice([1, 1, 1, 2, 3, 5]))
        cap = int(rng.integers(1, 121))
        out.append(dict(name=f"rand{i:02d}", cfg=400 + i, dtype=dtype, d=d, h=h, grouping=grouping,
                        group_size=group_size, tokens=sizes, g=g, cap=cap,
                        text_len=int(rng.integers(1, 25)),
                        layout=str(rng.choice(["padded", "packed"])),
                        keep=float(rng.uniform(0.05, 0.9))))
    return out


CASES = _cases()


def _workload(c):
    return W.Workload(c["name"], c["cfg"], batch=len(c["tokens"]), d=c["d"], d_text=c["d"], h=c["h"],
                      dtype=c["dtype"], text_len=c["text_len"], tokens=c["tokens"],
                      grouping=c["grouping"], group_size=c["group_size"], cap=c["cap"], g=c["g"],
                      layout=c["layout"], description="seeded random shape")


def _stop_bias(w, lay, inp, keep):
    """A bias retaining about ``keep`` of the tokens the caps allow, halfway
    between two adjacent breakpoints of the oracle's own selection."""
    KQV = oracle.project(inp["X"], inp["s_start"], inp["s_stop"], inp["W_kqv"], w.dtype)
    ctx = oracle.text_context(inp["E_text"], lay.text_off, inp["W_text"])
    pm = oracle.stop_thresholds(KQV, ctx, lay.grp_off, lay.grp_img, lay.grp_cap, w.h, g=w.g)
    allowed = int(sum(len(p) for p in pm))
    b, _ = oracle.choose_stop_bias(pm, keep * allowed)
    return b


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_random_shape(gpu_lib, case):
    from paper_2609_13804_amd import binding as sp
    from paper_2609_13804_amd.runner import DeviceRun
    w = _workload(case)
    lay = W.make_layout(w)
    inp = W.make_inputs(w)
    b_stop = _stop_bias(w, lay, inp, case["keep"])
    sizes = np.diff(lay.grp_off)
    steps = int(max(min(int(c), -(-int(n) // w.g)) for c, n in zip(lay.grp_cap, sizes))) + 1
    print(f"{case['name']}: {case}", flush=True)
    run = DeviceRun(w, inp, lay, b_stop, trace_steps=steps, logits=True)
    run.project()
    run.select(flags=0)
    run.compact()
    torch.cuda.synchronize()
    assert run.device_errors() == [0, 0, 0]
    plain = run.kept_lists()
    out_gpu = run.out.float().cpu().numpy()
    seq_gpu = run.seq_info.cpu().numpy().tolist()
    run.select(flags=sp.SP_TRACE | sp.SP_LOGITS)
    torch.cuda.synchronize()
    assert run.device_errors() == [0, 0, 0]
    assert run.kept_lists() == plain
    actions = run.trace_actions()
    KQV = run.KQV.double().cpu().numpy()
    ctx = run.ctx.double().cpu().numpy()
    tr = run.trace.cpu().numpy()
    if w.g == 1:
        rep = parity.check_selection(KQV, ctx, lay.grp_off, lay.grp_img, lay.grp_cap, b_stop, w.h,
                                     actions, tr, w.dtype, logits=run.trace_logits())
    else:
        rep = parity.check_grouped_selection(KQV, ctx, lay.grp_off, lay.grp_img, lay.grp_cap,
                                             b_stop, w.h, w.g, actions, tr, w.dtype,
                                             logits=run.trace_logits())
    assert plain == parity.kept_from_actions(actions, lay.grp_off, lay.grp_img, lay.img_off,
                                             lay.batch)
    # the prefill buffer starts zero-filled; rows a step does not write stay so
    out_or, seq_or = oracle.compact(inp["X"], lay.img_off, inp["E_text"], lay.text_off, plain,
                                    w.layout, lay.rows_per_image, np.zeros_like(out_gpu))
    assert seq_gpu == seq_or.tolist()
    assert np.array_equal(out_gpu, out_or.astype(np.float32))
    print(f"{case['name']}: {rep.episodes} episodes, {rep.steps} steps, {rep.exempt_steps} exempt, "
          f"max logit err {rep.max_logit_err:.2e}, kept {[len(k) for k in plain]}", flush=True)
