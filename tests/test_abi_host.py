"""The C ABI on the host: the library loads, exports every entry point the
header declares, and rejects invalid arguments before any device work.

Every call here fails host-side validation, so no GPU is needed: the
pointers passed are fake (never dereferenced) and the stream is 0.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "stepprune.h")


@pytest.fixture(scope="module")
def sp():
    from paper_2609_13804_amd import binding
    return binding


def test_header_symbols_are_exported(sp):
    text = open(HEADER).read()
    declared = set(re.findall(r"\b(stepprune_\w+)\s*\(", text))
    assert declared == set(sp.EXPORTS)
    lib = sp.library()
    for name in declared:
        assert hasattr(lib, name), name


def test_status_strings(sp):
    for code in range(6):
        assert sp.status_string(code) != "unknown status"
    assert sp.status_string(99) == "unknown status"


FAKE = 0x10000          # aligned, never dereferenced
MISALIGNED = 0x10008


def _dims(sp, d=256, dt=256, h=128, dtype=None):
    return sp.dims(d, dt, h, sp.SP_BF16 if dtype is None else dtype)


def test_workspace_bytes(sp):
    dm = _dims(sp)
    assert sp.stepprune_workspace_bytes(0, dm, 100, 10, 2, 3, 50, 10) >= 256 + 10 * 128 * 4
    sel = sp.stepprune_workspace_bytes(1, dm, 100, 10, 2, 3, 50, 10)
    assert sel >= 256 + 3 * 2 * 51 * 52 * 4
    assert sp.stepprune_workspace_bytes(2, dm, 100, 10, 2, 3, 50, 10) == 256
    assert sp.stepprune_workspace_bytes(1, dm, 100, 10, 2, 3, 5000, 10) == 0   # group too large
    gate = sp.stepprune_workspace_bytes(3, dm, 100, 10, 2, 3, 50, 10)   # T = 100 tokens, d = 256
    assert gate >= 256 + 100 * 256 * (4 + 2 + 2 + 8)
    assert sp.stepprune_workspace_bytes(3, _dims(sp, dtype=sp.SP_F32), 100, 10, 2, 3, 50, 10) == 0
    assert sp.stepprune_workspace_bytes(4, dm, 100, 10, 2, 3, 50, 10) > 0       # the encoder
    assert sp.stepprune_workspace_bytes(5, dm, 100, 10, 2, 3, 50, 10) == 0
    assert sp.stepprune_workspace_bytes(0, _dims(sp, h=100), 100, 10, 2, 3, 50, 10) == 0


def _project(sp, dm=None, **kw):
    args = dict(X=FAKE, T_vis=10, s_start=FAKE, s_stop=FAKE, W_kqv=FAKE, E_text=FAKE,
                text_off=FAKE, B=1, T_txt=4, W_text=FAKE, g_text=1.0, ln_eps=1e-5, KQV=FAKE,
                ctx=FAKE, ws=FAKE, ws_bytes=0)
    args.update(kw)
    return sp.stepprune_project(dm or _dims(sp), stream=0, raise_on_error=False, **args)


def test_project_validation(sp):
    assert _project(sp, _dims(sp, h=96)) == sp.SP_EINVAL                 # h not a multiple of 64
    assert _project(sp, _dims(sp, d=0)) == sp.SP_EINVAL
    assert _project(sp, _dims(sp, dtype=7)) == sp.SP_EUNSUPPORTED
    assert _project(sp, _dims(sp, h=2048)) == sp.SP_EUNSUPPORTED
    # float32 takes h <= 512; bfloat16 h <= 1024
    assert _project(sp, _dims(sp, h=576, dtype=sp.SP_F32)) == sp.SP_EUNSUPPORTED
    assert _project(sp, _dims(sp, h=1024, dtype=sp.SP_F32)) == sp.SP_EUNSUPPORTED
    assert _project(sp, _dims(sp, h=512, dtype=sp.SP_F32)) == sp.SP_EWORKSPACE
    assert _project(sp, _dims(sp, h=1024)) == sp.SP_EWORKSPACE
    assert _select(sp, _dims(sp, h=576, dtype=sp.SP_F32)) == sp.SP_EUNSUPPORTED
    assert sp.stepprune_workspace_bytes(1, _dims(sp, h=576, dtype=sp.SP_F32), 100, 10, 2, 3, 50,
                                        10) == 0
    assert _project(sp, X=None) == sp.SP_EINVAL
    assert _project(sp, KQV=None) == sp.SP_EINVAL
    assert _project(sp, W_kqv=MISALIGNED) == sp.SP_EINVAL
    assert _project(sp, B=0) == sp.SP_EINVAL
    assert _project(sp, ln_eps=-1.0) == sp.SP_EINVAL
    assert _project(sp) == sp.SP_EWORKSPACE                              # ws_bytes = 0


def _select(sp, dm=None, **kw):
    args = dict(KQV=FAKE, ctx=FAKE, T_vis=10, img_off=FAKE, B=1, grp_off=FAKE, grp_img=FAKE,
                grp_cap=FAKE, G=1, max_group=10, max_cap=4, kept_off=FAKE, b_stop=0.0, g=1,
                flags=0, kept_idx=FAKE, kept_cnt=FAKE, grp_cnt=None, trace=None, trace_steps=0,
                ws=FAKE, ws_bytes=0)
    args.update(kw)
    return sp.stepprune_select(dm or _dims(sp), stream=0, raise_on_error=False, **args)


def test_select_validation(sp):
    assert _select(sp, g=0) == sp.SP_EINVAL
    assert _select(sp, g=6) == sp.SP_EUNSUPPORTED                       # g <= 5
    assert _select(sp, g=5) == sp.SP_EWORKSPACE                         # accepted up to the workspace
    assert _select(sp, max_group=1023) == sp.SP_EUNSUPPORTED
    assert _select(sp, max_group=-1) == sp.SP_EINVAL
    assert _select(sp, flags=32) == sp.SP_EINVAL                        # unknown flag
    assert _select(sp, flags=sp.SP_TRACE, trace_steps=5, trace=None) == sp.SP_EINVAL
    assert _select(sp, b_stop=float("nan")) == sp.SP_EINVAL
    assert _select(sp, KQV=None) == sp.SP_EINVAL
    assert _select(sp, grp_off=None) == sp.SP_EINVAL
    assert _select(sp, ws=MISALIGNED) == sp.SP_EINVAL
    assert _select(sp, B=0) == sp.SP_EINVAL
    assert _select(sp) == sp.SP_EWORKSPACE


def _select_noalloc(sp, **kw):
    args = dict(KQV=FAKE, ctx=FAKE, T_vis=10, img_off=FAKE, B=1, grp_off=FAKE, grp_img=FAKE,
                grp_cap=FAKE, G=1, max_group=10, max_cap=4, kept_off=FAKE, b_stop=0.0, g=1,
                flags=0, kept_idx=FAKE, kept_cnt=FAKE, grp_cnt=None, trace=None, trace_steps=0,
                err=FAKE)
    args.update(kw)
    return sp.stepprune_select_noalloc(_dims(sp), stream=0, raise_on_error=False, **args)


def test_select_noalloc_validation(sp):
    """Only calls that host validation refuses: a valid call would reach the
    device."""
    assert _select_noalloc(sp, err=None) == sp.SP_EINVAL               # the error word is required
    assert _select_noalloc(sp, err=FAKE + 2) == sp.SP_EINVAL           # and 4-byte aligned
    assert _select_noalloc(sp, g=6) == sp.SP_EUNSUPPORTED
    assert _select_noalloc(sp, KQV=None) == sp.SP_EINVAL
    assert _select_noalloc(sp, flags=32) == sp.SP_EINVAL
    # sizes whose workspace exceeds the fixed scratch: 9 groups of 1000 tokens
    # need 9 x 8.05 MB of Gram blocks
    dm = _dims(sp)
    assert sp.stepprune_workspace_bytes(1, dm, 9000, 0, 1, 9, 1000, 8) > sp.NOALLOC_SCRATCH_BYTES
    assert _select_noalloc(sp, T_vis=9000, G=9, max_group=1000, max_cap=8) == sp.SP_EWORKSPACE
    # the 16 x 576 batch at h = 1024 fits, with 24 such groups the most
    big = sp.dims(4096, 4096, 1024, sp.SP_BF16)
    fits = [G for G in range(1, 40)
            if sp.stepprune_workspace_bytes(1, big, 576 * G, 64 * G, G, G, 576, 192)
            <= sp.NOALLOC_SCRATCH_BYTES]
    assert max(fits) == 24 and fits == list(range(1, 25))


def _select_traj(sp, traj, **kw):
    args = dict(KQV=FAKE, ctx=FAKE, T_vis=10, img_off=FAKE, B=1, grp_off=FAKE, grp_img=FAKE,
                grp_cap=FAKE, G=1, max_group=10, max_cap=4, kept_off=FAKE, b_stop=0.0, g=1,
                flags=0, kept_idx=FAKE, kept_cnt=FAKE, grp_cnt=None, trace=None, trace_steps=0,
                traj=traj, ws=FAKE, ws_bytes=0)
    args.update(kw)
    return sp.stepprune_select_trajectory(_dims(sp), stream=0, raise_on_error=False, **args)


def test_gate_denoise_validation(sp):
    names = ["ln1_g", "ln1_b", "W_v", "b_v", "W_o", "b_o", "ln2_g", "ln2_b", "W_1", "b_1",
             "W_2", "b_2"]
    full = sp.sp_denoiser(**{n: FAKE for n in names})
    dm = _dims(sp)
    ws_bytes = sp.stepprune_workspace_bytes(3, dm, 10, 0, 1, 0, 0, 0)

    def call(dm=dm, X=FAKE, T=10, alpha=FAKE, eps=FAKE, p=full, out=FAKE + 0x100000, ws=FAKE,
             ws_bytes=ws_bytes):
        return sp.stepprune_gate_denoise(dm, X, T, alpha, eps, p, out, ws, ws_bytes, stream=0,
                                         raise_on_error=False)
    assert call(dm=_dims(sp, dtype=sp.SP_F32)) == sp.SP_EUNSUPPORTED
    assert call(dm=_dims(sp, d=4160, dt=4160)) == sp.SP_EUNSUPPORTED
    assert call(T=-1) == sp.SP_EINVAL
    assert call(X=None) == sp.SP_EINVAL
    assert call(out=FAKE) == sp.SP_EINVAL                  # aliases X
    assert call(X=MISALIGNED) == sp.SP_EINVAL
    assert call(ws_bytes=ws_bytes - 1) == sp.SP_EWORKSPACE
    assert call(p=sp.sp_denoiser(**{m: (MISALIGNED if m == "b_1" else FAKE) for m in names})) \
        == sp.SP_EINVAL
    for n in names:
        part = sp.sp_denoiser(**{m: (None if m == n else FAKE) for m in names})
        assert call(p=part) == sp.SP_EINVAL, n


def test_select_trajectory_validation(sp):
    ok = sp.trajectory(1.0, 0.9, FAKE, FAKE)
    assert _select_traj(sp, ok) == sp.SP_EWORKSPACE                    # accepted up to the workspace
    assert _select_traj(sp, None) == sp.SP_EINVAL
    assert _select_traj(sp, sp.trajectory(0.0, 0.9, FAKE, FAKE)) == sp.SP_EINVAL      # tau <= 0
    assert _select_traj(sp, sp.trajectory(1.0, 0.0, FAKE, FAKE)) == sp.SP_EINVAL      # beta <= 0
    assert _select_traj(sp, sp.trajectory(1.0, 1.5, FAKE, FAKE)) == sp.SP_EINVAL      # beta > 1
    assert _select_traj(sp, sp.trajectory(1.0, 0.9, None, FAKE)) == sp.SP_EINVAL
    assert _select_traj(sp, sp.trajectory(1.0, 0.9, FAKE, None)) == sp.SP_EINVAL
    assert _select_traj(sp, sp.trajectory(1.0, 0.9, FAKE, FAKE, None, 3)) == sp.SP_EINVAL
    assert _select_traj(sp, ok, g=2) == sp.SP_EUNSUPPORTED
    assert _select_traj(sp, ok, flags=sp.SP_FULL_ROLLOUT | sp.SP_TRACE, trace=FAKE,
                        trace_steps=3) == sp.SP_EWORKSPACE
    assert _select(sp, flags=sp.SP_FULL_ROLLOUT) == sp.SP_EWORKSPACE
    assert _select(sp, flags=sp.SP_GRAM_ONLY) == sp.SP_EWORKSPACE
    assert _select(sp, flags=sp.SP_REUSE_GRAM) == sp.SP_EWORKSPACE
    assert _select(sp, flags=sp.SP_GRAM_ONLY | sp.SP_REUSE_GRAM) == sp.SP_EINVAL
    assert _select_traj(sp, ok, flags=sp.SP_GRAM_ONLY) == sp.SP_EINVAL
    assert _select(sp, flags=32) == sp.SP_EINVAL                        # unknown flag


def _compact(sp, dm=None, **kw):
    args = dict(X=FAKE, img_off=FAKE, E_text=FAKE, text_off=FAKE, kept_idx=FAKE, kept_off=FAKE,
                kept_cnt=FAKE, B=2, layout=sp.SP_LAYOUT_PADDED, rows_per_image=8, out_rows=16,
                out=FAKE, seq_info=FAKE, ws=FAKE, ws_bytes=0)
    args.update(kw)
    return sp.stepprune_compact(dm or _dims(sp), stream=0, raise_on_error=False, **args)


def test_compact_validation(sp):
    assert _compact(sp, _dims(sp, d=256, dt=128)) == sp.SP_EUNSUPPORTED   # text rows must match
    assert _compact(sp, layout=7) == sp.SP_EINVAL
    assert _compact(sp, rows_per_image=9) == sp.SP_EINVAL               # 2 * 9 > out_rows
    assert _compact(sp, out=None) == sp.SP_EINVAL
    assert _compact(sp, out=MISALIGNED) == sp.SP_EINVAL
    assert _compact(sp) == sp.SP_EWORKSPACE


def test_read_device_error_rejects_null(sp):
    code = ctypes.c_int32(0)
    assert sp.library().stepprune_read_device_error(None, None, ctypes.byref(code)) == sp.SP_EINVAL


C_PROGRAM = r"""
#include <stdio.h>
#include "stepprune.h"
int main(void) {
  sp_dims d = {4096, 4096, 1024, SP_BF16};
  for (int s = SP_OK; s <= SP_EDEVICE; ++s) printf("%s\n", stepprune_status_string((sp_status)s));
  printf("%zu\n", stepprune_workspace_bytes(1, &d, 9216, 1024, 16, 16, 576, 192));
  /* host validation only: a null dims pointer and null buffers never reach the device */
  printf("%d\n", (int)stepprune_project(NULL, NULL, 0, NULL, NULL, NULL, NULL, NULL, 1, 0, NULL,
                                        1.0f, 1e-5f, NULL, NULL, NULL, 0, NULL, 0));
  printf("%d\n", (int)stepprune_compact(&d, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 1,
                                        SP_LAYOUT_PADDED, 640, 0, NULL, NULL, NULL, 0, NULL, 0));
  return 0;
}
"""


def test_header_is_plain_c(sp, tmp_path):
    """A C99 program compiled by gcc against the header alone links the library
    and gets the same answers the Python binding gets."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    rocm_inc = "/opt/rocm/include"
    if gcc is None or not os.path.isdir(rocm_inc):
        pytest.skip("gcc or the ROCm headers are not available")
    src = tmp_path / "abi.c"
    src.write_text(C_PROGRAM)
    lib_dir = os.path.dirname(sp.LIB_PATH)
    exe = tmp_path / "abi"
    subprocess.run([gcc, "-std=c99", "-Wall", "-Werror=implicit-function-declaration",
                    "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I", rocm_inc,
                    str(src), "-o", str(exe), "-L", lib_dir, "-lstepprune",
                    f"-Wl,-rpath,{lib_dir}"], check=True, capture_output=True, timeout=120)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True,
                         timeout=60).stdout.split("\n")
    assert out[:6] == [sp.status_string(s) for s in range(6)]
    assert int(out[6]) == sp.stepprune_workspace_bytes(1, sp.dims(4096, 4096, 1024, sp.SP_BF16),
                                                       9216, 1024, 16, 16, 576, 192)
    assert int(out[7]) == sp.SP_EINVAL
    assert int(out[8]) == sp.SP_EINVAL


def test_encode_validation(sp):
    blk = sp.encoder_blocks([{k: FAKE for k in sp.ENCODER_FIELDS}] * 2)
    dm = _dims(sp, d=256, dt=192)

    def call(dm=dm, blocks=blk, max_seq=64, flags=0, ws_bytes=0, X=FAKE, W_p=FAKE):
        return sp.stepprune_encode(dm, X, 10, FAKE, 1, FAKE, FAKE, 4, W_p, 1.0, blocks, max_seq,
                                   flags, FAKE + 0x100000, FAKE, ws_bytes, stream=0,
                                   raise_on_error=False)
    assert call() == sp.SP_EWORKSPACE                                     # accepted up to the workspace
    assert call(dm=_dims(sp, d=320, dt=192)) == sp.SP_EUNSUPPORTED       # heads of 128
    assert call(dm=_dims(sp, d=4224, dt=192)) == sp.SP_EUNSUPPORTED      # d <= 4096
    assert call(dm=_dims(sp, d=256, dt=192, dtype=sp.SP_F32)) == sp.SP_EUNSUPPORTED
    assert call(blocks=None) == sp.SP_EINVAL
    part = sp.encoder_blocks([{k: FAKE for k in sp.ENCODER_FIELDS},
                              {k: (None if k == "b_2" else FAKE) for k in sp.ENCODER_FIELDS}])
    assert call(blocks=part) == sp.SP_EINVAL
    assert call(max_seq=0) == sp.SP_EINVAL
    assert call(flags=2) == sp.SP_EINVAL
    assert call(X=None) == sp.SP_EINVAL
    assert call(W_p=MISALIGNED) == sp.SP_EINVAL
    need = sp.stepprune_workspace_bytes(4, dm, 10, 4, 1, 0, 64, 0)
    assert need >= 256 + 14 * 256 * (4 + 2 + 2 + 6 + 8)
    assert call(ws_bytes=need - 1) == sp.SP_EWORKSPACE
    assert sp.stepprune_workspace_bytes(4, dm, 10, 4, 1, 0, 0, 0) == 0     # max_seq >= 1
