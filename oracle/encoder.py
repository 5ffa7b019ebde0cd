"""Eq. 3: the cross-modal input encoder (TEST INFRASTRUCTURE ONLY; plain
float64 NumPy).

Section "Conditional Sequential Pointer Policy", paragraph "Cross-Modal Input
Encoder", and Table "component-ablation" (a):

    E~   = g_text * LN(E_text W_p^T)               text projected into R^D
    H    = Enc([X; E~])[visual positions]          two pre-norm ViT blocks

For each image the visual tokens X_b and its projected text tokens E~_b form
one sequence [X_b; E~_b] of N_b + L_b tokens; the blocks attend over the whole
sequence (bidirectionally by default, as the paper's default; causally as its
ablation row), and only the first N_b outputs are kept.  Images never see each
other.

Readings taken here (the paper names the block type, not its sizes):

  R24  Enc is two pre-norm Vision Transformer blocks of width D = d:
           h = x + W_o MHA(LN1(x)) + b_o,     y = h + W_2 GELU(W_1 LN2(h) + b_1) + b_2,
       LayerNorm with scale and shift and eps 1e-6, multi-head attention with
       heads of width 128 (d / 128 heads) over q, k, v = LN1(x) W_qkv^T + b_qkv
       (rows [0, d) query, [d, 2d) key, [2d, 3d) value; head j takes columns
       [128 j, 128 j + 128) of each), scores scaled by 128^(-1/2), the MLP
       4d wide with the exact GELU, every linear map with a bias.
  R25  The text projection's LN is the pointer context's: no scale or shift,
       biased variance, eps 1e-5; g_text = 1 at inference.  W_p is stored
       [d, d_text] (output-major, x -> x W_p^T).
  R26  Bidirectional attention unless ``causal``: then token i attends to
       tokens j <= i of its own sequence (visual tokens first).
  R27  Storage (mirror mode only): the GPU keeps the residual stream in
       float32 and rounds once to bfloat16 the text projection's product, the
       LayerNorm outputs, each product's result, the biased query/key/value,
       the attention probabilities that weight the values, each head's
       output, the biased GELU output and H.  ``mirror=True`` rounds at those
       points (the probabilities taken against the row's final maximum);
       ``mirror=False`` is the exact float64 block.

Weights use nn.Linear's layout, [out_features, in_features].
"""
from dataclasses import dataclass
from typing import List, Sequence

import numpy as np
from scipy.special import erf

from .rounding import round_bf16

ENC_LN_EPS = 1e-6          # the blocks' LayerNorms (R24)
TEXT_LN_EPS = 1e-5         # the text projection's LayerNorm (R25)
HEAD_DIM = 128


@dataclass
class EncoderBlock:
    ln1_g: np.ndarray   # [d]
    ln1_b: np.ndarray   # [d]
    W_qkv: np.ndarray   # [3d, d]
    b_qkv: np.ndarray   # [3d]
    W_o: np.ndarray     # [d, d]
    b_o: np.ndarray     # [d]
    ln2_g: np.ndarray   # [d]
    ln2_b: np.ndarray   # [d]
    W_1: np.ndarray     # [4d, d]
    b_1: np.ndarray     # [4d]
    W_2: np.ndarray     # [d, 4d]
    b_2: np.ndarray     # [d]


def _ln(x, g=None, b=None, eps=ENC_LN_EPS):
    x = np.asarray(x, np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    y = (x - mu) / np.sqrt(var + eps)
    return y if g is None else y * g + b


def _gelu(x):
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def text_projection(E, W_p, g_text=1.0, mirror=False):
    """E~ = g_text * LN(E W_p^T) (Eq. 3's first line, R25)."""
    r = round_bf16 if mirror else (lambda v: v)
    P = r(np.asarray(E, np.float64) @ np.asarray(W_p, np.float64).T)
    return g_text * _ln(P, eps=TEXT_LN_EPS)


def attention(z_q, z_k, z_v, causal=False, mirror=False):
    """softmax(q k^T / sqrt(128)) v for one sequence, head by head (R24, R26).
    z_q, z_k, z_v: [S, d] (d a multiple of 128)."""
    r = round_bf16 if mirror else (lambda v: v)
    S, d = z_q.shape
    out = np.empty((S, d))
    scale = 1.0 / np.sqrt(HEAD_DIM)
    mask = np.triu(np.ones((S, S), bool), 1) if causal else None
    for hd in range(d // HEAD_DIM):
        c = slice(HEAD_DIM * hd, HEAD_DIM * (hd + 1))
        s = (z_q[:, c] @ z_k[:, c].T) * scale
        if mask is not None:
            s = np.where(mask, -np.inf, s)
        e = np.exp(s - s.max(axis=1, keepdims=True))
        out[:, c] = r((r(e) @ z_v[:, c]) / e.sum(axis=1, keepdims=True))
    return out


def block(x, p: EncoderBlock, causal=False, mirror=False):
    """One pre-norm block (R24) on one sequence x [S, d] (float64 values)."""
    r = round_bf16 if mirror else (lambda v: v)
    d = x.shape[1]
    z = r(_ln(x, p.ln1_g, p.ln1_b))
    qkv = r(r(z @ p.W_qkv.T) + p.b_qkv)
    a = attention(qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:], causal, mirror)
    h = x + r(a @ p.W_o.T) + p.b_o
    z2 = r(_ln(h, p.ln2_g, p.ln2_b))
    m = r(_gelu(r(z2 @ p.W_1.T) + p.b_1))
    return h + r(m @ p.W_2.T) + p.b_2


def encode(X, img_off, E, text_off, W_p, blocks: Sequence[EncoderBlock], g_text=1.0,
           causal=False, mirror=False) -> np.ndarray:
    """H for every image (Eq. 3): [X_b; E~_b] through the blocks, the first N_b
    rows kept.  X [T_vis, d] packed by img_off [B+1]; E [T_txt, d_text] packed
    by text_off [B+1]; returns H [T_vis, d]."""
    r = round_bf16 if mirror else (lambda v: v)
    X = np.asarray(X, np.float64)
    Et = text_projection(E, W_p, g_text, mirror) if len(E) else np.zeros((0, X.shape[1]))
    H = np.empty_like(X)
    for b in range(len(img_off) - 1):
        i0, i1 = int(img_off[b]), int(img_off[b + 1])
        t0, t1 = int(text_off[b]), int(text_off[b + 1])
        x = np.concatenate([X[i0:i1], Et[t0:t1]], axis=0)
        for p in blocks:
            x = block(x, p, causal, mirror)
        H[i0:i1] = r(x[:i1 - i0])
    return H
