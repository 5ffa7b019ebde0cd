"""The cross-modal input encoder on the GPU (stepprune_encode, Eq. 3) against
the oracle (oracle/encoder.py), through the C ABI.

Small batches are checked on every row of H, with ragged sequences (lengths
that are not multiples of the 32-key blocks, more than one 128-query block,
an image without text, an image with one visual token), both attention
directions and three widths (at d = 384 the q/k/v product's columns end in
a partial tile, so its bias epilogue runs on a ragged edge); the 16 x
640-token batch at d = 4096 is checked on two whole images.

Tolerance.  The oracle's exact mode is the definition; its mirror mode rounds
to bfloat16 where the GPU stores bfloat16.  Per row of H the GPU must be within
MIRROR_TOL of the mirror (normwise relative): both round the same values at the
same points, the GPU computing in float32 between them and the oracle in
float64, so a value within float32 error of a rounding boundary may round the
other way and the flip propagates through the later products.  Against the
exact block the GPU may then differ by no more than the mirror does plus
MIRROR_TOL (triangle inequality): |gpu - exact| <= |mirror - exact| + MIRROR_TOL.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle.encoder import EncoderBlock
from paper_2609_13804_amd import binding as sp
from paper_2609_13804_amd import workloads as W

pytestmark = pytest.mark.gpu

MIRROR_TOL = 1e-2


def _dev_bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to("cuda", torch.bfloat16)


def _dev_f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()


def _run(d, d_text, X, img_off, E, text_off, params, g_text=1.0, causal=False, max_seq=None,
         expect_error=0):
    B = len(img_off) - 1
    T_vis, T_txt = int(img_off[-1]), int(text_off[-1])
    seqs = np.diff(img_off) + np.diff(text_off)
    max_seq = int(seqs.max()) if max_seq is None else max_seq
    dm = sp.dims(d, d_text, 128, sp.SP_BF16)
    ws_bytes = sp.stepprune_workspace_bytes(sp.STAGE_ENCODE, dm, T_vis, T_txt, B, 0, max_seq, 0)
    assert ws_bytes > 0
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    Xd, Ed = _dev_bf16(X), _dev_bf16(E) if T_txt else None
    io = torch.from_numpy(np.asarray(img_off, np.int32)).cuda()
    to = torch.from_numpy(np.asarray(text_off, np.int32)).cuda()
    Wp = _dev_bf16(params["W_p"])
    blk = [{k: (_dev_bf16(v) if k.startswith("W_") else _dev_f32(v)) for k, v in b.items()}
           for b in params["blocks"]]
    H = torch.full((max(1, T_vis), d), float("nan"), dtype=torch.bfloat16, device="cuda")
    sp.stepprune_encode(dm, Xd, T_vis, io, B, Ed, to, T_txt, Wp, g_text, sp.encoder_blocks(blk),
                        max_seq, sp.SP_ENC_CAUSAL if causal else 0, H, ws, ws_bytes)
    torch.cuda.synchronize()
    assert sp.stepprune_read_device_error(ws) == expect_error
    return H[:T_vis].float().cpu().numpy().astype(np.float64)


def _oracle(X, img_off, E, text_off, params, g_text=1.0, causal=False, mirror=False, images=None):
    blocks = [EncoderBlock(**{k: np.asarray(v, np.float64) for k, v in b.items()})
              for b in params["blocks"]]
    if images is None:
        return oracle.encode(X, img_off, E, text_off, params["W_p"], blocks, g_text, causal, mirror)
    out = {}
    for b in images:
        i0, i1, t0, t1 = img_off[b], img_off[b + 1], text_off[b], text_off[b + 1]
        out[b] = oracle.encode(X[i0:i1], [0, i1 - i0], E[t0:t1], [0, t1 - t0], params["W_p"],
                               blocks, g_text, causal, mirror)
    return out


def _rel(got, want):
    return np.linalg.norm(got - want, axis=1) / np.maximum(np.linalg.norm(want, axis=1), 1e-30)


def _check(name, got, exact, mirror):
    assert np.all(np.isfinite(got)), name
    e_m = _rel(got, mirror)
    e_x = _rel(got, exact)
    m_x = _rel(mirror, exact)
    print(f"{name}: rows {len(got)}; GPU vs mirror max {e_m.max():.2e} mean {e_m.mean():.2e}; "
          f"GPU vs exact max {e_x.max():.2e} mean {e_x.mean():.2e}; mirror vs exact max "
          f"{m_x.max():.2e} mean {m_x.mean():.2e}; bit-equal to mirror {np.mean(got == mirror):.3f}",
          flush=True)
    assert e_m.max() <= MIRROR_TOL, name
    assert np.all(e_x <= m_x + MIRROR_TOL), name


def _case(seed, d, d_text, sizes, texts):
    rng = np.random.default_rng([2609, 3, seed])
    n, L = sum(sizes), sum(texts)
    # clustered visual tokens (the selector's inputs) and N(0, 1) text, in bfloat16
    centres = rng.standard_normal((12, d)).astype(np.float32)
    X = centres[rng.integers(0, 12, n)] + 0.05 * rng.standard_normal((n, d)).astype(np.float32)
    X = oracle.round_bf16(X)
    E = oracle.round_bf16(rng.standard_normal((L, d_text)))
    img_off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    text_off = np.concatenate([[0], np.cumsum(texts)]).astype(np.int64)
    w = W.Workload(f"enc{seed}", 300 + seed, batch=len(sizes), d=d, d_text=d_text, h=128,
                   dtype="bf16", text_len=1, tokens=tuple(sizes))
    return X, img_off, E, text_off, W.make_encoder_inputs(w)


SMALL = [
    # (name, seed, d, d_text, visual tokens per image, text tokens per image)
    ("ragged_d256", 1, 256, 192, (70, 33, 200, 1), (5, 0, 12, 40)),
    ("d512", 2, 512, 256, (129, 64, 17), (31, 64, 3)),
    # three heads: the q/k/v product's 1152 columns end in half a 256-column tile
    ("d384", 3, 384, 128, (90, 300), (20, 7)),
]


@pytest.mark.parametrize("causal", [False, True], ids=["bidirectional", "causal"])
@pytest.mark.parametrize("name,seed,d,d_text,sizes,texts", SMALL, ids=[c[0] for c in SMALL])
def test_encoder_every_row(gpu_lib, name, seed, d, d_text, sizes, texts, causal):
    X, img_off, E, text_off, params = _case(seed, d, d_text, sizes, texts)
    got = _run(d, d_text, X, img_off, E, text_off, params, g_text=0.8, causal=causal)
    exact = _oracle(X, img_off, E, text_off, params, 0.8, causal)
    mirror = _oracle(X, img_off, E, text_off, params, 0.8, causal, mirror=True)
    _check(f"{name} {'causal' if causal else 'bidirectional'}", got, exact, mirror)


def test_encoder_padding_and_errors(gpu_lib):
    X, img_off, E, text_off, params = _case(1, 256, 192, (70, 33, 200, 1), (5, 0, 12, 40))
    # a larger max_seq than needed gives the same H
    a = _run(256, 192, X, img_off, E, text_off, params)
    b = _run(256, 192, X, img_off, E, text_off, params, max_seq=400)
    np.testing.assert_array_equal(a, b)
    # an image longer than max_seq is a device error
    _run(256, 192, X, img_off, E, text_off, params, max_seq=100,
         expect_error=sp.SP_DEV_GROUP_TOO_LARGE)


def test_encoder_full_size_two_images(gpu_lib):
    """The 16 x (576 + 64) batch at d = 4096 (32 heads), as the bench runs it;
    the first and the last image against the oracle."""
    w = W.WORKLOADS["llava15_bf16"]
    lay = W.make_layout(w)
    inp = W.make_inputs(w)
    params = W.make_encoder_inputs(w)
    print("encoder full size: inputs ready", flush=True)
    got = _run(w.d, w.d_text, inp["X"], lay.img_off, inp["E_text"], lay.text_off, params)
    print("encoder full size: GPU done", flush=True)
    for b in (0, lay.batch - 1):
        i0, i1 = lay.img_off[b], lay.img_off[b + 1]
        exact = _oracle(inp["X"], lay.img_off, inp["E_text"], lay.text_off, params, images=[b])[b]
        mirror = _oracle(inp["X"], lay.img_off, inp["E_text"], lay.text_off, params, mirror=True,
                         images=[b])[b]
        _check(f"llava15 encoder image {b}", got[i0:i1], exact, mirror)
