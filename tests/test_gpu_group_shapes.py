"""Group sizes at the edges of the selection kernel's launch shapes, checked
element by element against the oracle (tests/parity.py protocol):

  * up to 512 tokens: one lane per token column;
  * 513-576 tokens: waves 0-3 also own the columns past 512, a quarter of
    each column's history per lane;
  * more than 576 tokens: 16 waves with fewer history registers per lane;
  * a largest group of 256 or 512 tokens: the Gram products' edge layout;

with caps that keep the history in registers, and caps that push it through
the LDS rows and the re-read tier.  Each case runs the untraced kernel (the
benchmark's) and the traced one, which must take the same decisions; the
traced run dumps every step's whole logit vector (SP_LOGITS), compared with
the oracle's element by element.
"""
import math

import numpy as np
import pytest
import torch

from paper_2609_13804_amd import workloads as W
from tests import parity

pytestmark = pytest.mark.gpu

CASES = [
    # (name, cfg id, tokens per image, cap, STOP bias)
    ("wide_1000", 105, (1000, 700, 33), 48, -math.inf),
    ("wide_1000_stop", 105, (1000, 700, 33), 48, 0.25),
    ("second_cols_576", 106, (576, 513, 512, 65), 64, 0.25),
    ("second_cols_deep", 107, (513, 520), 300, -math.inf),
    ("lanes_512", 108, (512, 448, 64, 1), 40, 0.1),
    # largest group a multiple of 256: the Gram tiles cover the token blocks
    # only and a separate kernel computes the START / STOP / context entries
    ("edge_256", 115, (256, 100, 255, 1, 254), 40, 0.1),
    ("edge_256_deep", 116, (256, 256), 200, -math.inf),
    ("edge_512", 117, (512, 300), 48, 0.1),
]


def _workload(name, cfg, tokens, cap):
    return W.Workload(name, cfg, batch=len(tokens), d=256, d_text=256, h=128, dtype="bf16",
                      text_len=5, tokens=tokens, cap=cap, layout="padded",
                      description="group-shape edge case")


@pytest.mark.parametrize("name,cfg,tokens,cap,b_stop", CASES, ids=[c[0] for c in CASES])
def test_group_shape(gpu_lib, name, cfg, tokens, cap, b_stop):
    from paper_2609_13804_amd.runner import DeviceRun
    from paper_2609_13804_amd import binding as sp
    w = _workload(name, cfg, tokens, cap)
    lay = W.make_layout(w)
    inp = W.make_inputs(w)
    sizes = np.diff(lay.grp_off)
    steps = int(max(min(int(c), int(n)) for c, n in zip(lay.grp_cap, sizes))) + 1
    run = DeviceRun(w, inp, lay, b_stop, trace_steps=steps, logits=True)
    run.project()
    run.select(flags=0)
    run.compact()
    torch.cuda.synchronize()
    assert run.device_errors() == [0, 0, 0]
    plain = run.kept_lists()
    run.select(flags=sp.SP_TRACE | sp.SP_LOGITS)
    torch.cuda.synchronize()
    assert run.device_errors() == [0, 0, 0]
    assert run.kept_lists() == plain
    actions = run.trace_actions()
    KQV = run.KQV.double().cpu().numpy()
    ctx = run.ctx.double().cpu().numpy()
    rep = parity.check_selection(KQV, ctx, lay.grp_off, lay.grp_img, lay.grp_cap, b_stop, w.h,
                                 actions, run.trace.cpu().numpy(), w.dtype,
                                 logits=run.trace_logits())
    assert plain == parity.kept_from_actions(actions, lay.grp_off, lay.grp_img, lay.img_off,
                                             lay.batch)
    print(f"{name}: {rep.episodes} episodes, {rep.steps} steps, {rep.exempt_steps} exempt, "
          f"max logit err {rep.max_logit_err:.2e}, kept {[len(k) for k in plain]}")
