"""Algorithm 1, step 5: physically gather the kept tokens ahead of the prompt.

Paper: Train-Inference Alignment (the hard subset, in native visual order, is
gathered before prefill) and the Introduction (the visual tokens are
prepended to the text prompt).

Readings taken here: each image's prefill sequence is its kept visual rows in
ascending index order followed by its text rows.  "padded": image b owns rows
[b*R, (b+1)*R) of the output and rows past K_b + L_b are left untouched;
seq_info[b] = K_b + L_b.  "packed": sequences are back to back,
seq_info = cu_seqlens[B+1] with cu[b+1] = cu[b] + K_b + L_b.
"""
import numpy as np


def compact(X, img_off, E_text, text_off, kept, layout: str, rows_per_image: int, out):
    """Return (out, seq_info).  ``out`` is copied, then written; ``kept`` lists
    image-local ascending indices per image."""
    out = np.array(out, copy=True)
    B = len(img_off) - 1
    if layout == "padded":
        seq = np.zeros(B, np.int32)
        for b in range(B):
            k = np.asarray(kept[b], np.int64)
            L = int(text_off[b + 1] - text_off[b])
            base = b * rows_per_image
            out[base:base + len(k)] = X[int(img_off[b]) + k]
            out[base + len(k):base + len(k) + L] = E_text[int(text_off[b]):int(text_off[b + 1])]
            seq[b] = len(k) + L
        return out, seq
    if layout == "packed":
        cu = np.zeros(B + 1, np.int32)
        for b in range(B):
            k = np.asarray(kept[b], np.int64)
            L = int(text_off[b + 1] - text_off[b])
            base = int(cu[b])
            out[base:base + len(k)] = X[int(img_off[b]) + k]
            out[base + len(k):base + len(k) + L] = E_text[int(text_off[b]):int(text_off[b + 1])]
            cu[b + 1] = cu[b] + len(k) + L
        return out, cu
    raise ValueError(f"unknown layout {layout!r}")
