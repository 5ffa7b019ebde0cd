"""The training pathway's noise gate and locally masked denoiser (TEST
INFRASTRUCTURE ONLY; plain float64 NumPy).

Section "Trajectory-Aware Differentiable Optimization", paragraphs on the
variance-preserving noise gate (Eq. 9) and the locally masked denoiser:

    x~_i  = sqrt(a_i) x_i + sqrt(1 - a_i) eps_i                     (Eq. 9)
    X^    = Denoise(X~; mask = diag)

Readings taken here (the paper gives the block's type, not its details):

  R21  a_i in [0, 1] is an input.  In the paper it comes from the
       differentiable top-k of Eq. 8, which is out of scope; eps is the
       caller's N(0, I) draw, passed in.
  R22  Denoise is one pre-norm Vision Transformer block of width d:
           h  = x~ + Attn(LN1(x~)),     X^ = h + MLP(LN2(h)),
       LayerNorm with affine parameters and eps 1e-6, MLP(z) =
       W2 GELU(W1 z + b1) + b2 with hidden width 4d and the exact (erf)
       GELU, every linear map with a bias.  Restricting self-attention to
       the diagonal leaves each token one key, its own, so its softmax
       weight is exactly 1 and Attn(z) = W_O (W_V z + b_V) + b_O whatever
       the number of heads; W_Q and W_K never reach the output.
  R23  Storage: the GPU keeps the residual stream (x~, h) in float32 and
       rounds every matrix-product operand and result to bfloat16 once
       (LN outputs, the four products, the biased V output, the GELU
       output, the block output).  ``mirror=True`` rounds at the same
       points; ``mirror=False`` is the exact float64 block.

Weights use nn.Linear's layout, [out_features, in_features].
"""
from dataclasses import dataclass

import numpy as np
from scipy.special import erf

from .rounding import round_bf16

LN_EPS = 1e-6


@dataclass
class DenoiserParams:
    ln1_g: np.ndarray   # [d]
    ln1_b: np.ndarray   # [d]
    W_v: np.ndarray     # [d, d]
    b_v: np.ndarray     # [d]
    W_o: np.ndarray     # [d, d]
    b_o: np.ndarray     # [d]
    ln2_g: np.ndarray   # [d]
    ln2_b: np.ndarray   # [d]
    W_1: np.ndarray     # [4d, d]
    b_1: np.ndarray     # [4d]
    W_2: np.ndarray     # [d, 4d]
    b_2: np.ndarray     # [d]


def vp_gate(X, alpha, eps):
    """Eq. 9, row by row: sqrt(a_i) x_i + sqrt(1 - a_i) eps_i."""
    a = np.asarray(alpha, np.float64)[:, None]
    return np.sqrt(a) * np.asarray(X, np.float64) + np.sqrt(1.0 - a) * np.asarray(eps, np.float64)


def layer_norm_affine(x, g, b, eps=LN_EPS):
    """LayerNorm over the last axis (biased variance) with scale g and shift b."""
    x = np.asarray(x, np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def gelu(x):
    """The exact GELU, x * Phi(x)."""
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def denoise(Xt, p: DenoiserParams, mirror=True):
    """R22's block on the gated rows Xt [T, d] (float64 values)."""
    r = round_bf16 if mirror else (lambda v: v)
    xt = np.asarray(Xt, np.float64)
    z1 = r(layer_norm_affine(xt, p.ln1_g, p.ln1_b))
    u1 = r(r(z1 @ p.W_v.T) + p.b_v)              # V projection (the only attended value)
    h = xt + r(u1 @ p.W_o.T) + p.b_o             # residual stream, float32 on the GPU
    z2 = r(layer_norm_affine(h, p.ln2_g, p.ln2_b))
    a = r(gelu(r(z2 @ p.W_1.T) + p.b_1))
    return r(h + r(a @ p.W_2.T) + p.b_2)


def gate_denoise(X, alpha, eps, p: DenoiserParams, mirror=True):
    """Eq. 9 followed by the locally masked denoiser."""
    return denoise(vp_gate(X, alpha, eps), p, mirror)
