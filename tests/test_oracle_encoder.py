"""Pins for the oracle's cross-modal input encoder (oracle/encoder.py, Eq. 3).

The exact mode is checked against torch's own pre-norm transformer encoder
layer in float64 (a library implementation of the block R24 reads), against
torch's LayerNorm for the text projection, and against properties the
definition fixes: the identity when both residual branches are zero, images
independent of each other, visual rows permuted with the visual tokens, text
tokens interchangeable under bidirectional attention, and under causal
attention a visual token that sees only the tokens before it.  Each of these
fails for a plausible slip: a transposed weight, a missing bias, the wrong
LayerNorm eps or affine, tanh GELU, a scale of 1/d instead of 1/sqrt(128),
heads taking interleaved columns, text appended before the visual tokens, the
text rows kept, images attending to each other, or a mask on the wrong side.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle.encoder import EncoderBlock, block, encode, text_projection, HEAD_DIM

D, DT = 256, 192          # two heads of 128


def _block(rng, d=D, scale=1.0):
    f = lambda *s, sd=1.0: rng.standard_normal(s) * sd
    return EncoderBlock(ln1_g=1 + 0.1 * f(d), ln1_b=0.1 * f(d),
                        W_qkv=f(3 * d, d, sd=scale / np.sqrt(d)), b_qkv=0.1 * f(3 * d),
                        W_o=f(d, d, sd=1 / np.sqrt(d)), b_o=0.1 * f(d),
                        ln2_g=1 + 0.1 * f(d), ln2_b=0.1 * f(d),
                        W_1=f(4 * d, d, sd=1 / np.sqrt(d)), b_1=0.1 * f(4 * d),
                        W_2=f(d, 4 * d, sd=1 / np.sqrt(4 * d)), b_2=0.1 * f(d))


def _torch_layer(p: EncoderBlock, d=D):
    layer = torch.nn.TransformerEncoderLayer(d, d // HEAD_DIM, dim_feedforward=4 * d, dropout=0.0,
                                             activation="gelu", layer_norm_eps=1e-6,
                                             batch_first=True, norm_first=True,
                                             dtype=torch.float64)
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    with torch.no_grad():
        layer.self_attn.in_proj_weight.copy_(t(p.W_qkv))
        layer.self_attn.in_proj_bias.copy_(t(p.b_qkv))
        layer.self_attn.out_proj.weight.copy_(t(p.W_o))
        layer.self_attn.out_proj.bias.copy_(t(p.b_o))
        layer.linear1.weight.copy_(t(p.W_1))
        layer.linear1.bias.copy_(t(p.b_1))
        layer.linear2.weight.copy_(t(p.W_2))
        layer.linear2.bias.copy_(t(p.b_2))
        layer.norm1.weight.copy_(t(p.ln1_g))
        layer.norm1.bias.copy_(t(p.ln1_b))
        layer.norm2.weight.copy_(t(p.ln2_g))
        layer.norm2.bias.copy_(t(p.ln2_b))
    return layer.eval()


def _inputs(rng, sizes=(7, 5, 9), text=(3, 4, 0)):
    X = rng.standard_normal((sum(sizes), D))
    E = rng.standard_normal((sum(text), DT))
    W_p = rng.standard_normal((D, DT)) / np.sqrt(DT)
    img_off = np.concatenate([[0], np.cumsum(sizes)])
    text_off = np.concatenate([[0], np.cumsum(text)])
    return X, img_off, E, text_off, W_p


@pytest.mark.parametrize("causal", [False, True])
def test_encoder_matches_torch_transformer_layers(causal):
    rng = np.random.default_rng(3)
    X, img_off, E, text_off, W_p = _inputs(rng)
    blocks = [_block(rng), _block(rng)]
    H = encode(X, img_off, E, text_off, W_p, blocks, g_text=0.7, causal=causal)
    layers = [_torch_layer(p) for p in blocks]
    Et = torch.nn.functional.layer_norm(torch.from_numpy(E @ W_p.T), (D,), eps=1e-5).numpy() * 0.7
    for b in range(len(img_off) - 1):
        i0, i1 = img_off[b], img_off[b + 1]
        seq = np.concatenate([X[i0:i1], Et[text_off[b]:text_off[b + 1]]])
        x = torch.from_numpy(seq)[None]
        mask = (torch.nn.Transformer.generate_square_subsequent_mask(len(seq), dtype=torch.float64)
                if causal else None)
        with torch.no_grad():
            for layer in layers:
                x = layer(x, src_mask=mask, is_causal=causal)
        np.testing.assert_allclose(H[i0:i1], x[0, :i1 - i0].numpy(), rtol=1e-11, atol=1e-11)


def test_text_projection_is_layer_norm_of_the_product():
    rng = np.random.default_rng(4)
    E = rng.standard_normal((6, DT))
    W_p = rng.standard_normal((D, DT))
    want = 0.25 * torch.nn.functional.layer_norm(torch.from_numpy(E) @ torch.from_numpy(W_p).T,
                                                 (D,), eps=1e-5).numpy()
    np.testing.assert_allclose(text_projection(E, W_p, 0.25), want, rtol=1e-12, atol=1e-12)


def test_zero_branches_give_the_identity():
    """W_o = W_2 = 0 and b_o = b_2 = 0: each block returns its input, so H = X
    (the visual rows, in order, whatever the text)."""
    rng = np.random.default_rng(5)
    X, img_off, E, text_off, W_p = _inputs(rng)
    blocks = []
    for _ in range(2):
        p = _block(rng)
        p.W_o[:] = 0
        p.b_o[:] = 0
        p.W_2[:] = 0
        p.b_2[:] = 0
        blocks.append(p)
    for causal in (False, True):
        H = encode(X, img_off, E, text_off, W_p, blocks, causal=causal)
        np.testing.assert_array_equal(H, X)


def test_images_are_independent():
    rng = np.random.default_rng(6)
    X, img_off, E, text_off, W_p = _inputs(rng)
    blocks = [_block(rng), _block(rng)]
    H = encode(X, img_off, E, text_off, W_p, blocks)
    for b in range(len(img_off) - 1):
        i0, i1, t0, t1 = img_off[b], img_off[b + 1], text_off[b], text_off[b + 1]
        alone = encode(X[i0:i1], [0, i1 - i0], E[t0:t1], [0, t1 - t0], W_p, blocks)
        np.testing.assert_allclose(H[i0:i1], alone, rtol=1e-12, atol=1e-12)


def test_permutations():
    """Bidirectional attention: permuting an image's visual tokens permutes its
    rows of H, and permuting its text tokens changes nothing."""
    rng = np.random.default_rng(7)
    X, img_off, E, text_off, W_p = _inputs(rng, sizes=(8,), text=(5,))
    blocks = [_block(rng), _block(rng)]
    H = encode(X, img_off, E, text_off, W_p, blocks)
    pv, pt = rng.permutation(8), rng.permutation(5)
    np.testing.assert_allclose(encode(X[pv], img_off, E, text_off, W_p, blocks), H[pv],
                               rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(encode(X, img_off, E[pt], text_off, W_p, blocks), H,
                               rtol=1e-11, atol=1e-11)
    # causal attention is order-dependent: the same text permutation changes H
    Hc = encode(X, img_off, E, text_off, W_p, blocks, causal=True)
    assert not np.allclose(encode(X[pv], img_off, E, text_off, W_p, blocks, causal=True), Hc[pv])


def test_causal_token_sees_only_its_prefix():
    """Under causal attention visual token i's output is the encoder's output
    on the sequence of visual tokens 0..i alone (text comes after them)."""
    rng = np.random.default_rng(8)
    X, img_off, E, text_off, W_p = _inputs(rng, sizes=(6,), text=(4,))
    blocks = [_block(rng), _block(rng)]
    H = encode(X, img_off, E, text_off, W_p, blocks, causal=True)
    for i in range(6):
        x = X[:i + 1]
        for p in blocks:
            x = block(x, p, causal=True)
        np.testing.assert_allclose(H[i], x[i], rtol=1e-11, atol=1e-11)


def test_mirror_mode_stores_bfloat16_and_stays_near_exact():
    """Mirror mode (the GPU's storage points) returns bfloat16 values, within a
    few bfloat16 ulps of the exact block."""
    rng = np.random.default_rng(9)
    X, img_off, E, text_off, W_p = _inputs(rng)
    X = oracle.round_bf16(X)
    blocks = [_block(rng), _block(rng)]
    Hm = encode(X, img_off, E, text_off, W_p, blocks, mirror=True)
    He = encode(X, img_off, E, text_off, W_p, blocks)
    np.testing.assert_array_equal(Hm, oracle.round_bf16(Hm))
    rel = np.linalg.norm(Hm - He, axis=1) / np.linalg.norm(He, axis=1)
    assert rel.max() < 2e-2
