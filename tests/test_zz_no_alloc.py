"""stepprune_select_noalloc (the selection with its scratch in the library's
fixed device array) against stepprune_select (caller workspace), through the
C ABI, on two calls in a row: the 16 x 576 x 4096 bf16 batch (42.9 MB of
scratch, near the 64 MiB limit), then a smaller ragged batch, so the second
call runs on the first one's leftovers.  The two entry points run the same
kernels, so kept indices, counts and the per-step trace must be bit-identical.
Also: the error word is the caller's, a data error lands in it, and
stepprune_select decides alike when its workspace holds garbage past the
header (nothing else in it has to start at zero).
"""
import numpy as np
import pytest
import torch

from paper_2609_13804_amd import binding as sp
from paper_2609_13804_amd import workloads as W

pytestmark = pytest.mark.gpu


def _noalloc(run, err, flags=None, caps=None):
    s = run.sizes
    return sp.stepprune_select_noalloc(
        run.dims, run.KQV, run.ctx, s.T_vis, run.img_off, s.B, run.grp_off, run.grp_img,
        run.grp_cap if caps is None else caps, s.G, s.max_group, s.max_cap, run.kept_off,
        run.b_stop, run.g, run.flags if flags is None else flags, run.kept_idx, run.kept_cnt,
        run.grp_cnt, run.trace, run.trace_steps, err, raise_on_error=False)


def _outputs(run):
    torch.cuda.synchronize()
    out = [run.kept_idx.clone(), run.kept_cnt.clone(), run.grp_cnt.clone()]
    if run.trace is not None:
        out.append(run.trace.clone())
    return out


def _reset(run):
    run.kept_idx.fill_(-7)
    run.kept_cnt.fill_(-7)
    run.grp_cnt.fill_(-7)
    if run.trace is not None:
        run.trace.fill_(float("nan"))


def _same(a, b):
    return all(torch.equal(x.view(torch.int32), y.view(torch.int32)) for x, y in zip(a, b))


def _device_run(name, trace=True):
    from paper_2609_13804_amd.runner import DeviceRun
    w = W.WORKLOADS[name]
    lay = W.make_layout(w)
    steps = int(max(lay.grp_cap.max(), 1)) + 1 if trace else 0
    run = DeviceRun(w, W.make_inputs(w), lay, W.stop_bias(w), trace_steps=steps)
    run.project()
    torch.cuda.synchronize()
    assert run.device_errors()[0] == 0
    return run


@pytest.mark.parametrize("first,second", [("llava15_bf16", "mid_bf16"),
                                          ("llava15_bf16", "small_g5_bf16"),
                                          ("tiny_f32", "tiny_bf16")])
def test_noalloc_matches_select(gpu_lib, first, second):
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    for name in (first, second):
        run = _device_run(name)
        s = run.sizes
        need = sp.stepprune_workspace_bytes(1, run.dims, s.T_vis, s.T_txt, s.B, s.G, s.max_group,
                                            s.max_cap)
        assert need <= sp.NOALLOC_SCRATCH_BYTES, (name, need)
        print(f"{name}: {s.B} images, {s.G} groups, scratch {need / 2**20:.1f} MiB", flush=True)
        for flags in (sp.SP_TRACE, 0):
            _reset(run)
            run.select(flags=flags)
            want = _outputs(run)
            assert run.device_errors()[1] == 0
            _reset(run)
            assert _noalloc(run, err, flags=flags) == sp.SP_OK
            got = _outputs(run)
            assert sp.stepprune_read_device_error(err) == 0
            assert _same(got, want), f"{name} flags {flags}: outputs differ"
        del run
        torch.cuda.empty_cache()


def test_noalloc_error_word_and_limits(gpu_lib):
    run = _device_run("tiny_bf16", trace=False)
    s = run.sizes
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    # a data error (a negative cap) lands in the caller's error word, which
    # keeps it until it is read
    caps = run.grp_cap.clone()
    caps[0] = -1
    assert _noalloc(run, err, flags=0, caps=caps) == sp.SP_OK
    assert _noalloc(run, err, flags=0) == sp.SP_OK
    assert sp.stepprune_read_device_error(err) == sp.SP_DEV_BAD_CAP
    assert sp.stepprune_read_device_error(err) == 0
    # sizes beyond the fixed scratch are refused before any launch
    big_g = sp.NOALLOC_SCRATCH_BYTES // (2 * 1000 * 1000 * 4) + 1
    st = sp.stepprune_select_noalloc(run.dims, run.KQV, run.ctx, s.T_vis, run.img_off, s.B,
                                     run.grp_off, run.grp_img, run.grp_cap, big_g, 1000, 8,
                                     run.kept_off, run.b_stop, 1, 0, run.kept_idx, run.kept_cnt,
                                     run.grp_cnt, None, 0, err, raise_on_error=False)
    assert st == sp.SP_EWORKSPACE
    # no error word, or a misaligned one
    assert _noalloc(run, None, flags=0) == sp.SP_EINVAL
    assert _noalloc(run, err.data_ptr() + 2, flags=0) == sp.SP_EINVAL
    torch.cuda.synchronize()
    assert sp.stepprune_read_device_error(err) == 0


def test_select_workspace_garbage_past_header(gpu_lib):
    """stepprune_select needs only the workspace header zeroed (the fixed
    scratch is never cleared, so this is what makes it valid to reuse)."""
    run = _device_run("mid_bf16")
    _reset(run)
    run.select(flags=sp.SP_TRACE)
    want = _outputs(run)
    ws = run.ws[1]
    ws.fill_(0xFF)              # float32 NaN everywhere
    ws[:256].zero_()
    _reset(run)
    run.select(flags=sp.SP_TRACE)
    got = _outputs(run)
    assert run.device_errors()[1] == 0
    assert _same(got, want)
