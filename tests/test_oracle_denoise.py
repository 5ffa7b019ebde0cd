"""Pins of the oracle's noise gate and locally masked denoiser (Eq. 9 and the
denoiser paragraph of Section "Trajectory-Aware Differentiable
Optimization"; readings R21-R23 in oracle/denoise.py).

The block is checked against torch's own pre-norm transformer encoder layer
run in float64 with a diagonal attention mask, which fixes the reading that
diagonal attention leaves only the value projection, the pre-norm order, the
exact GELU and the residual placement independently of the oracle's code.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle.denoise import DenoiserParams, denoise, gate_denoise, gelu, layer_norm_affine, vp_gate


def _params(rng, d, scale=1.0):
    f = lambda *s: rng.standard_normal(s) * scale
    return DenoiserParams(
        ln1_g=1.0 + 0.1 * f(d), ln1_b=0.1 * f(d), W_v=f(d, d) / np.sqrt(d), b_v=0.1 * f(d),
        W_o=f(d, d) / np.sqrt(d), b_o=0.1 * f(d), ln2_g=1.0 + 0.1 * f(d), ln2_b=0.1 * f(d),
        W_1=f(4 * d, d) / np.sqrt(d), b_1=0.1 * f(4 * d), W_2=f(d, 4 * d) / np.sqrt(4 * d),
        b_2=0.1 * f(d))


def _torch_layer(p, d, nhead, rng):
    layer = torch.nn.TransformerEncoderLayer(d, nhead, dim_feedforward=4 * d, dropout=0.0,
                                             activation="gelu", layer_norm_eps=1e-6,
                                             batch_first=True, norm_first=True).double().eval()
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    with torch.no_grad():
        # W_Q and W_K are random: under the diagonal mask they must not matter
        layer.self_attn.in_proj_weight.copy_(torch.cat([t(rng.standard_normal((d, d))),
                                                        t(rng.standard_normal((d, d))),
                                                        t(p.W_v)]))
        layer.self_attn.in_proj_bias.copy_(torch.cat([t(rng.standard_normal(d)),
                                                      t(rng.standard_normal(d)), t(p.b_v)]))
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
    return layer


@pytest.mark.parametrize("nhead", [1, 4])
def test_denoiser_is_torch_prenorm_layer_with_diagonal_mask(nhead):
    rng = np.random.default_rng([9, nhead])
    d, T = 32, 11
    p = _params(rng, d)
    x = rng.standard_normal((T, d))
    layer = _torch_layer(p, d, nhead, rng)
    mask = torch.full((T, T), float("-inf"), dtype=torch.float64)
    mask.fill_diagonal_(0.0)
    with torch.no_grad():
        want = layer(torch.from_numpy(x)[None], src_mask=mask)[0].numpy()
    got = denoise(x, p, mirror=False)
    assert np.max(np.abs(got - want)) <= 1e-12 * max(1.0, np.max(np.abs(want)))


def test_rows_are_independent_under_the_diagonal_mask():
    rng = np.random.default_rng(17)
    d, T = 16, 9
    p = _params(rng, d)
    x = rng.standard_normal((T, d))
    full = denoise(x, p, mirror=False)
    for i in (0, 4, 8):      # equal up to the order a library product sums in
        assert np.max(np.abs(denoise(x[i:i + 1], p, mirror=False)[0] - full[i])) <= 1e-12


def test_gate_end_points_and_variance():
    rng = np.random.default_rng(23)
    x = rng.standard_normal((4000, 256))
    e = rng.standard_normal((4000, 256))
    assert np.array_equal(vp_gate(x, np.ones(4000), e), x)
    assert np.array_equal(vp_gate(x, np.zeros(4000), e), e)
    a = rng.uniform(0.0, 1.0, 4000)
    xt = vp_gate(x, a, e)
    # unit-variance x and eps, independent: every gated entry has variance 1
    assert abs(np.mean(xt ** 2) - 1.0) < 0.02
    # the mixture weights: E[x~ x] = sqrt(a) per row
    corr = np.mean(xt * x, axis=1)
    assert np.corrcoef(corr, np.sqrt(a))[0, 1] > 0.95


def test_layer_norm_and_gelu_against_torch():
    rng = np.random.default_rng(31)
    x = rng.standard_normal((7, 48)) * 3 + 1
    g, b = rng.standard_normal(48), rng.standard_normal(48)
    want = torch.nn.functional.layer_norm(torch.from_numpy(x), (48,), torch.from_numpy(g),
                                          torch.from_numpy(b), eps=1e-6).numpy()
    assert np.max(np.abs(layer_norm_affine(x, g, b) - want)) <= 1e-12
    v = np.linspace(-8, 8, 1001)
    assert np.max(np.abs(gelu(v) - torch.nn.functional.gelu(torch.from_numpy(v)).numpy())) <= 1e-12


def test_mirror_rounds_only_where_the_gpu_stores_bfloat16():
    rng = np.random.default_rng(41)
    d, T = 64, 20
    p = _params(rng, d)
    x = oracle.round_bf16(rng.standard_normal((T, d)))
    e = oracle.round_bf16(rng.standard_normal((T, d)))
    a = rng.uniform(0, 1, T)
    exact = gate_denoise(x, a, e, p, mirror=False)
    mir = gate_denoise(x, a, e, p, mirror=True)
    assert np.array_equal(mir, oracle.round_bf16(mir))            # output stored in bf16
    rel = np.linalg.norm(mir - exact, axis=1) / np.linalg.norm(exact, axis=1)
    assert rel.max() < 2e-2 and rel.max() > 0                      # a few bf16 roundings
