"""Algorithm 1, step 1: project the visual tokens and the text context once.

Paper: Section "Conditional Sequential Pointer Policy" (text projection
W_p E_text followed by LayerNorm and the gain g_text; the encoder of Eq. 3),
and the pointer decoder's attention projections (Eq. 4).

Readings taken here (the paper leaves these open):
* The two-block encoder of Eq. 3 is not on this path: H = X.  The pointer
  decoder is one layer with one head of width h and no normalisation, so its
  key / query / value projections are row-wise linear maps of the candidate
  memory M = [X; s_stop] and of the START embedding, computed once:
  [k | q | v] = x W_kqv^T, W_kqv of shape [3h, d] (rows: key, query and
  value output features).
* The text projection maps into the pointer query space (width h):
  c_b = g_text * mean_l LN(E_{b,l} W_text^T), LayerNorm without affine
  parameters, biased variance, eps = 1e-5, g_text = 1 at inference.  An image
  with no text tokens gets c_b = 0.
* Projected rows are stored in the workload dtype, rounded once from the exact
  product; the context is stored in float32.
"""
import numpy as np

from .rounding import round_to, round_f32


def project(X, s_start, s_stop, W_kqv, dtype):
    """Projected rows [T_vis + 2, 3h]: the visual rows, then START, then STOP.

    X: [T_vis, d] visual tokens of all images, packed; s_start, s_stop: [d];
    W_kqv: [3h, d].  Columns [0:h] are keys, [h:2h] queries, [2h:3h] values.
    """
    X_aug = np.vstack([np.asarray(X, np.float64),
                       np.asarray(s_start, np.float64)[None, :],
                       np.asarray(s_stop, np.float64)[None, :]])
    exact = X_aug @ np.asarray(W_kqv, np.float64).T
    return round_to(exact, dtype)


def layer_norm(T, eps):
    """LayerNorm over the last axis without affine parameters (biased variance)."""
    T = np.asarray(T, np.float64)
    mu = T.mean(axis=-1, keepdims=True)
    var = ((T - mu) ** 2).mean(axis=-1, keepdims=True)
    return (T - mu) / np.sqrt(var + eps)


def text_context(E_text, text_off, W_text, g_text=1.0, ln_eps=1e-5):
    """Per-image pooled text context c_b, [B, h], float32 values as float64.

    E_text: [T_txt, d_text] text rows of all images, packed by text_off[B+1];
    W_text: [h, d_text].
    """
    E = np.asarray(E_text, np.float64)
    W = np.asarray(W_text, np.float64)
    B = len(text_off) - 1
    h = W.shape[0]
    ctx = np.zeros((B, h), np.float64)
    for b in range(B):
        rows = E[text_off[b]:text_off[b + 1]]
        if rows.shape[0] == 0:
            continue
        ctx[b] = g_text * layer_norm(rows @ W.T, ln_eps).mean(axis=0)
    return round_f32(ctx)
