"""HIP graphs of the selection path: a captured step, and the pipeline's
per-slot stage graphs, replayed several times with eager work and device
synchronisations between the replays; every replay must reproduce the eager
result bit for bit (projected rows, context, kept lists, counts and the
prefill buffer)."""
import numpy as np
import pytest
import torch

from paper_2609_13804_amd import workloads as W
from paper_2609_13804_amd.runner import DeviceRun, Pipeline

pytestmark = pytest.mark.gpu


def _outputs(run):
    """What a step writes: projected rows, context, each image's kept list and
    count, the per-group counts and the prefill rows the step fills."""
    lay = run.layout
    res = [run.KQV.view(torch.uint8).cpu().numpy().tobytes(), run.ctx.cpu().numpy().tobytes(),
           run.kept_lists(), run.kept_cnt.cpu().numpy().tolist(),
           run.grp_cnt.cpu().numpy()[:lay.groups].tolist()]
    if run.out is not None:
        seq = run.seq_info.cpu().numpy()
        out = run.out.view(torch.uint8).cpu().numpy()
        if run.w.layout == "padded":
            rows = [out[b * lay.rows_per_image: b * lay.rows_per_image + int(seq[b])]
                    for b in range(lay.batch)]
        else:
            rows = [out[:int(seq[-1])]]
        res += [seq.tolist(), b"".join(r.tobytes() for r in rows)]
    return res


def _clear(run):
    """Poison everything a step rewrites in full."""
    run.KQV.fill_(float("nan"))
    run.ctx.fill_(float("nan"))
    run.kept_cnt.fill_(-3)
    run.kept_idx.fill_(-3)
    if run.out is not None:
        run.out.fill_(float("nan"))
        run.seq_info.fill_(-3)


def _same(a, b):
    return all(x == y for x, y in zip(a, b)) and len(a) == len(b)


@pytest.mark.parametrize("name", ["tiny_f32", "small_packed_bf16", "single_f32", "llava15_bf16"])
def test_captured_step_replays_match_eager(gpu_lib, name):
    w = W.WORKLOADS[name]
    run = DeviceRun(w, W.make_inputs(w), W.make_layout(w), W.stop_bias(w))
    run.run()
    torch.cuda.synchronize()
    assert run.device_errors() == [0, 0, 0]
    ref = _outputs(run)
    g = run.capture()
    for rep in range(3):
        _clear(run)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert run.device_errors() == [0, 0, 0], rep
        assert _same(_outputs(run), ref), f"replay {rep} differs from the eager step"
        # eager work between replays
        _clear(run)
        run.run()
        torch.cuda.synchronize()
        assert _same(_outputs(run), ref)


def test_pipeline_graphs_match_one_stream(gpu_lib):
    w = W.WORKLOADS["llava15_bf16"]
    lay = W.make_layout(w)
    run = DeviceRun(w, W.make_inputs(w), lay, W.stop_bias(w))
    pipe = Pipeline(run, slots=4, streams=3,
                    inputs=[W.make_inputs(w, batch_index=k) for k in range(1, 4)])
    refs = []
    for r in pipe.runs:
        r.run()
        torch.cuda.synchronize()
        refs.append(_outputs(r))
    pipe.use_graphs()
    for rnd in range(3):
        for r in pipe.runs:
            _clear(r)
        torch.cuda.synchronize()
        for _ in range(len(pipe.runs)):
            pipe.issue()
        torch.cuda.synchronize()
        for k, r in enumerate(pipe.runs):
            assert r.device_errors() == [0, 0, 0]
            assert _same(_outputs(r), refs[k]), f"round {rnd}, slot {k}"
