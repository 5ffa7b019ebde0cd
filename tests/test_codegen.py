"""Properties of the generated gfx950 code that the sources rely on.  Every
translation unit of the library is compiled here to device assembly with the
library's own flags (hipcc cross-compiles; no GPU is needed).

  * Packed float32: no kernel contains a packed float32 ALU instruction
    (v_pk_fma_f32, v_pk_mul_f32, v_pk_add_f32); the build disables them.
  * M0: the direct-to-LDS load (csrc/lds_dma.h) is an inline-assembly
    statement that sets M0 itself immediately before its load.  The compiler
    treats M0 as reserved and does not preserve it across inline assembly, so
    in the files that use the statement no compiler-generated instruction may
    hold a value in M0: every write of M0 there must be one of the statement's
    own, directly followed by its load, and none of the instructions that read
    M0 implicitly (register indexing, messages) may appear.
"""
import concurrent.futures
import os
import re
import subprocess

import pytest

from paper_2609_13804_amd import build as B

DMA_USERS = ["gemm.hip", "encode.hip"]
PACKED_F32 = re.compile(r"\bv_pk_(fma|mul|add)_f32\b")
IMPLICIT_M0 = re.compile(r"^\s*(s_set_gpr_idx_\w+|v_movre\w+|s_movre\w+|s_sendmsg\w*|v_interp_\w+)\b")


@pytest.fixture(scope="module")
def device_asm(tmp_path_factory):
    hipcc = B._hipcc()
    out = tmp_path_factory.mktemp("asm")
    sources = list(B.SOURCES) + [B.PROBE_SOURCE]

    def compile_one(src):
        dst = str(out / src.replace(".hip", ".s"))
        flags = [f for f in B.HIPCC_FLAGS if f != "-fPIC"]
        cmd = [hipcc, *flags, *B.EXTRA_FLAGS.get(src, []), "--cuda-device-only", "-S",
               os.path.join(B.CSRC, src), "-o", dst]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        return src, open(dst).read().splitlines()

    with concurrent.futures.ThreadPoolExecutor(max_workers=4) as ex:
        return dict(ex.map(compile_one, sources))


def _instructions(lines):
    for i, line in enumerate(lines):
        s = line.split(";")[0].strip()
        if s and not s.startswith(".") and not s.endswith(":"):
            yield i, s


def test_no_packed_fp32(device_asm):
    for src, lines in device_asm.items():
        bad = [s for _, s in _instructions(lines) if PACKED_F32.search(s)]
        assert not bad, (src, bad[:5])


@pytest.mark.parametrize("src", DMA_USERS)
def test_m0_is_written_only_by_the_lds_load(device_asm, src):
    ins = list(_instructions(device_asm[src]))
    writes = 0
    for k, (_, s) in enumerate(ins):
        assert not IMPLICIT_M0.match(s), (src, s)
        ops = s.split(None, 1)
        if len(ops) == 2 and re.match(r"m0\s*,", ops[1]):
            # the statement's own: s_mov_b32 m0, sN ; s_nop 0 ; global_load_lds_dwordx4
            assert re.fullmatch(r"s_mov_b32\s+m0,\s*s\d+", s), (src, s)
            assert ins[k + 1][1] == "s_nop 0", (src, ins[k + 1][1])
            assert ins[k + 2][1].startswith("global_load_lds_dwordx4"), (src, ins[k + 2][1])
            writes += 1
    assert writes > 0, src
