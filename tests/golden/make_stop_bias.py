"""Calibrate the STOP bias of every workload with the CPU oracle.

Writes paper_2609_13804_amd/stop_bias.json.  The bias is an input of the
selector (an additive scalar on the STOP logit) chosen so that each
workload retains its target count: the paper's operating points (mean
retained 64 of 576 for LLaVA-1.5, 32 per 576-token group for the
LLaVA-NeXT-shaped batch, 88.9% and 90% pruning for the Qwen2.5-VL- and
InternVL3-shaped batches).  Only the oracle and the seeded generator run here.

    python tests/golden/make_stop_bias.py [workload ...]
"""
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2609_13804_amd import workloads as W  # noqa: E402


def calibrate(w):
    inp = W.make_inputs(w)
    lay = W.make_layout(w)
    KQV = oracle.project(inp["X"], inp["s_start"], inp["s_stop"], inp["W_kqv"], w.dtype)
    ctx = oracle.text_context(inp["E_text"], lay.text_off, inp["W_text"])
    del inp
    pm = oracle.stop_thresholds(KQV, ctx, lay.grp_off, lay.grp_img, lay.grp_cap, w.h, g=w.g)
    kind, val = w.stop_target
    n_tok = int(lay.img_off[-1])
    if kind == "mean_k":
        target = val * lay.groups
    elif kind == "ratio":
        target = val * n_tok
    elif kind == "k_each":
        target = val * lay.groups
    else:
        raise ValueError(kind)
    b, total = oracle.choose_stop_bias(pm, target, stop_inside_cap=(kind == "k_each"))
    per_group = [int(np.count_nonzero(p >= b)) for p in pm]
    return dict(b_stop=b, target=kind, target_value=val, target_total=target,
                retained_total=total, groups=lay.groups, tokens=n_tok,
                mean_per_group=total / lay.groups, ratio=total / n_tok,
                per_group_min=min(per_group), per_group_max=max(per_group))


def main(names):
    path = W.STOP_BIAS_FILE
    table = json.load(open(path)) if os.path.exists(path) else {}
    for name in names:
        t0 = time.time()
        table[name] = calibrate(W.WORKLOADS[name])
        print(name, json.dumps(table[name]), "%.1fs" % (time.time() - t0), flush=True)
        with open(path, "w") as f:
            json.dump(table, f, indent=1, sort_keys=True)


if __name__ == "__main__":
    main(sys.argv[1:] or (W.SMALL_WORKLOADS + W.PAPER_WORKLOADS + W.GROUPED_SMALL_WORKLOADS
                          + W.GROUPED_WORKLOADS))
