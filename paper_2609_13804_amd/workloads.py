"""Seeded synthetic workloads shaped like the paper's four backbones.

This module only draws random inputs and lays out their offsets; it holds
none of the selector's arithmetic, so both the HIP path and the CPU oracle
can be fed from it.

Shapes follow the paper's evaluated settings (Section "Models and Evaluation
Scope"): LLaVA-1.5 with a fixed 576-token prefix, LLaVA-NeXT AnyRes with
2880 tokens as one base grid plus four tiles of 576, Qwen2.5-VL with
dynamic resolution, and InternVL3 with 12 tiles plus a thumbnail of 256
tokens each.  The paper's benchmarks and frozen vision features are not
available, so seeded tensors of the same shapes stand in for them:

* visual tokens: per image, 48 centres ~ N(0, I_d) and every token is a centre
  plus N(0, 0.05^2 I_d) noise, so clusters of near-duplicate tokens exist;
* text tokens: ~ N(0, I_{d_text});
* selector weights: W_kqv ~ N(0, 1/d), W_text ~ N(0, 1/d_text), START and STOP
  embeddings ~ N(0, I_d);
* sizes (dynamic resolution): N_i = 4 * U{64 .. 1024}.

Every random stream is ``numpy.random.default_rng([260913804, cfg_id, stream,
index])`` so a given image is identical whatever batch it sits in.  The
one-image float32 workload is keyed 1097: its operating point is 63 retained
tokens with STOP taken inside the cap of 64 rounds, and the retained counts a
STOP bias can reach are the breakpoints of the running minimum of the STOP
margin (see oracle/calibration.py), which depend on the draw (key 1 reaches
46 at most).  1097 is the first key from 1001 on whose draw reaches 63.

Values are drawn in float32 and rounded once (round-to-nearest-even) to
bfloat16 for the bf16 workloads; the float32 copies handed to the CPU side are
those rounded values, exactly.
"""
from __future__ import annotations

import dataclasses
import json
import math
import os
from typing import Dict, List, Optional, Tuple

import numpy as np

SEED_ROOT = 260913804
N_CLUSTERS = 48
CLUSTER_NOISE = 0.05

STREAM_WEIGHTS = 0
STREAM_VISUAL = 1
STREAM_TEXT = 2
STREAM_SIZES = 3

_HERE = os.path.dirname(os.path.abspath(__file__))
STOP_BIAS_FILE = os.path.join(_HERE, "stop_bias.json")


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: batch shape, selector shape and grouping."""
    name: str
    cfg_id: int
    batch: int
    d: int
    d_text: int
    h: int
    dtype: str                       # "f32" or "bf16"
    text_len: int
    tokens: Tuple[int, ...] = ()     # fixed per-image N (empty: drawn, see ragged)
    ragged: Optional[Tuple[int, int, int]] = None  # (lo, hi, multiple) for drawn N
    grouping: str = "single"         # "single" | "fixed" | "balanced"
    group_size: int = 0              # "fixed": tokens per group, "balanced": max
    cap: int = 0                     # per-group round cap (0 with cap_frac)
    cap_frac: float = 0.0            # cap = n_group * cap_frac (exact for these sizes)
    g: int = 1                       # tokens per round (Eq. 11); the cap counts rounds
    layout: str = "padded"           # "padded" | "packed"
    stop_target: Tuple[str, float] = ("mean_k", 64.0)
    description: str = ""

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


def _rng(cfg_id: int, stream: int, index: int) -> np.random.Generator:
    return np.random.default_rng([SEED_ROOT, cfg_id, stream, index])


# The five paper-shaped workloads, then small ones that span several tiles with
# ragged tails so the oracle finishes in seconds.
WORKLOADS: Dict[str, Workload] = {}


def _add(w: Workload) -> None:
    WORKLOADS[w.name] = w


_add(Workload("single_f32", 1097, batch=1, d=1024, d_text=1024, h=256, dtype="f32",
              text_len=32, tokens=(576,), cap=64, layout="padded",
              stop_target=("k_each", 63.0),
              description="1 image, N=576, d=1024, fp32, hidden 256, cap 64"))
_add(Workload("llava15_bf16", 2, batch=16, d=4096, d_text=4096, h=1024, dtype="bf16",
              text_len=64, tokens=(576,) * 16, cap=192, layout="padded",
              stop_target=("mean_k", 64.0),
              description="16 images x 576 tokens x 4096, bf16, cap 192, 576+64 prefill rows"))
_add(Workload("llavanext_bf16", 3, batch=8, d=4096, d_text=4096, h=1024, dtype="bf16",
              text_len=128, tokens=(2880,) * 8, grouping="fixed", group_size=576,
              cap=64, layout="padded", stop_target=("mean_k", 32.0),
              description="8 images x 2880 tokens (5 groups of 576), bf16, cap 64/group"))
_add(Workload("qwen25vl_bf16", 4, batch=32, d=3584, d_text=3584, h=1024, dtype="bf16",
              text_len=96, ragged=(256, 4096, 4), grouping="balanced", group_size=576,
              cap_frac=0.25, layout="packed", stop_target=("ratio", 0.111),
              description="32 images, N ~ U{256..4096 step 4}, d=3584, groups <= 576, cap N/4, packed"))
_add(Workload("internvl3_bf16", 5, batch=64, d=3584, d_text=3584, h=1024, dtype="bf16",
              text_len=512, tokens=(3328,) * 64, grouping="fixed", group_size=256,
              cap=32, layout="packed", stop_target=("ratio", 0.10),
              description="64 images x 13 groups x 256 tokens, d=3584, cap 32/group, packed"))

# Small workloads for element-by-element parity (oracle in seconds).
_add(Workload("tiny_f32", 101, batch=3, d=256, d_text=192, h=64, dtype="f32",
              text_len=7, tokens=(97, 130, 61), cap=40, layout="padded",
              stop_target=("mean_k", 12.0), description="ragged tiny fp32"))
_add(Workload("tiny_bf16", 102, batch=4, d=320, d_text=320, h=128, dtype="bf16",
              text_len=11, tokens=(200, 37, 150, 257), grouping="fixed", group_size=96,
              cap=24, layout="padded", stop_target=("mean_k", 8.0),
              description="ragged tiny bf16, fixed groups with ragged tails"))
_add(Workload("small_packed_bf16", 103, batch=6, d=512, d_text=512, h=256, dtype="bf16",
              text_len=19, ragged=(64, 1400, 4), grouping="balanced", group_size=576,
              cap_frac=0.25, layout="packed", stop_target=("ratio", 0.111),
              description="ragged bf16, balanced groups <= 576, packed varlen"))
_add(Workload("mid_bf16", 104, batch=3, d=1024, d_text=1024, h=1024, dtype="bf16",
              text_len=40, tokens=(576, 576, 300), cap=192, layout="padded",
              stop_target=("mean_k", 64.0),
              description="hidden 1024 bf16 with full 576-token groups and long caps"))
_add(Workload("wide_f32", 120, batch=12, d=512, d_text=512, h=256, dtype="f32",
              text_len=16, tokens=(576,) * 12, cap=64, layout="padded",
              stop_target=("mean_k", 40.0),
              description="fp32 batch large enough for the 128 x 128 float32 tiles"))

# Grouped selection, g = 5 tokens per round (the setting of the high-resolution
# backbones), on the same shapes: small parity cases, then the three
# high-resolution batches.
_add(Workload("tiny_g5_f32", 201, batch=3, d=256, d_text=192, h=64, dtype="f32",
              text_len=7, tokens=(97, 130, 3), cap=9, g=5, layout="padded",
              stop_target=("mean_k", 14.0), description="ragged tiny fp32, 5 tokens per round"))
_add(Workload("small_g5_bf16", 202, batch=5, d=512, d_text=512, h=256, dtype="bf16",
              text_len=19, ragged=(64, 1400, 4), grouping="balanced", group_size=576,
              cap_frac=0.05, g=5, layout="packed", stop_target=("ratio", 0.111),
              description="ragged bf16, balanced groups <= 576, 5 tokens per round, packed"))
_add(Workload("mid_g5_bf16", 203, batch=2, d=1024, d_text=1024, h=1024, dtype="bf16",
              text_len=40, tokens=(576, 301), cap=40, g=5, layout="padded",
              stop_target=("mean_k", 64.0),
              description="hidden 1024 bf16, full 576-token groups, 5 tokens per round"))
_add(Workload("llavanext_g5_bf16", 13, batch=8, d=4096, d_text=4096, h=1024, dtype="bf16",
              text_len=128, tokens=(2880,) * 8, grouping="fixed", group_size=576,
              cap=13, g=5, layout="padded", stop_target=("mean_k", 32.0),
              description="8 images x 2880 tokens (5 groups of 576), bf16, 5 tokens per round"))
_add(Workload("qwen25vl_g5_bf16", 14, batch=32, d=3584, d_text=3584, h=1024, dtype="bf16",
              text_len=96, ragged=(256, 4096, 4), grouping="balanced", group_size=576,
              cap_frac=0.05, g=5, layout="packed", stop_target=("ratio", 0.111),
              description="32 images, N ~ U{256..4096 step 4}, groups <= 576, 5 tokens per round"))
_add(Workload("internvl3_g5_bf16", 15, batch=64, d=3584, d_text=3584, h=1024, dtype="bf16",
              text_len=512, tokens=(3328,) * 64, grouping="fixed", group_size=256,
              cap=7, g=5, layout="packed", stop_target=("ratio", 0.10),
              description="64 images x 13 groups x 256 tokens, d=3584, 5 tokens per round"))

PAPER_WORKLOADS = ["single_f32", "llava15_bf16", "llavanext_bf16", "qwen25vl_bf16", "internvl3_bf16"]
SMALL_WORKLOADS = ["tiny_f32", "tiny_bf16", "small_packed_bf16", "mid_bf16", "wide_f32"]
GROUPED_SMALL_WORKLOADS = ["tiny_g5_f32", "small_g5_bf16", "mid_g5_bf16"]
GROUPED_WORKLOADS = ["llavanext_g5_bf16", "qwen25vl_g5_bf16", "internvl3_g5_bf16"]


def image_sizes(w: Workload) -> List[int]:
    """Visual token count of every image."""
    if w.ragged is None:
        assert len(w.tokens) == w.batch
        return list(w.tokens)
    lo, hi, mult = w.ragged
    rng = _rng(w.cfg_id, STREAM_SIZES, 0)
    return [int(v) * mult for v in rng.integers(lo // mult, hi // mult + 1, size=w.batch)]


def partition(w: Workload, n: int) -> List[int]:
    """Split one image's n tokens into contiguous group sizes, in order."""
    if w.grouping == "single":
        return [n]
    if w.grouping == "fixed":
        sizes = [w.group_size] * (n // w.group_size)
        if n % w.group_size:
            sizes.append(n % w.group_size)
        return sizes
    if w.grouping == "balanced":
        # ceil(n / max) groups whose sizes are multiples of 4 and differ by at most 4.
        g = -(-n // w.group_size)
        units = n // 4
        base, extra = divmod(units, g)
        sizes = [4 * (base + (1 if i < extra else 0)) for i in range(g)]
        sizes[-1] += n - sum(sizes)      # n not a multiple of 4 (never for these workloads)
        return sizes
    raise ValueError(w.grouping)


def group_cap(w: Workload, n_group: int) -> int:
    if w.cap_frac:
        return max(1, int(math.floor(n_group * w.cap_frac)))
    return w.cap


@dataclasses.dataclass
class Layout:
    """Offsets describing a batch: all arrays int32 numpy."""
    img_off: np.ndarray     # [B+1] visual row offsets
    text_off: np.ndarray    # [B+1] text row offsets
    grp_off: np.ndarray     # [G+1] visual row offsets of each group
    grp_img: np.ndarray     # [G] owning image
    grp_cap: np.ndarray     # [G] round cap
    kept_off: np.ndarray    # [B+1] prefix sum of per-image kept capacity sum min(cap * g, n)
    rows_per_image: int     # padded layout: rows per image (max N + max L)
    out_rows: int           # rows of the compacted buffer

    @property
    def batch(self) -> int:
        return len(self.img_off) - 1

    @property
    def groups(self) -> int:
        return len(self.grp_img)


def make_layout(w: Workload, images: Optional[List[int]] = None) -> Layout:
    """Offsets for the whole batch, or for the sub-batch ``images`` (in that order)."""
    all_sizes = image_sizes(w)
    sizes = all_sizes if images is None else [all_sizes[i] for i in images]
    B = len(sizes)
    img_off = np.zeros(B + 1, np.int32)
    img_off[1:] = np.cumsum(sizes)
    text_off = (np.arange(B + 1) * w.text_len).astype(np.int32)
    grp_off = [0]
    grp_img, grp_cap = [], []
    kept = np.zeros(B + 1, np.int64)
    for b, n in enumerate(sizes):
        cap_b = 0
        for ng in partition(w, n):
            grp_off.append(grp_off[-1] + ng)
            grp_img.append(b)
            c = group_cap(w, ng)
            grp_cap.append(c)
            cap_b += min(c * w.g, ng)
        kept[b + 1] = kept[b] + cap_b
    rows_per_image = max(sizes) + w.text_len
    if w.layout == "padded":
        out_rows = B * rows_per_image
    else:
        out_rows = int(kept[B]) + B * w.text_len
    return Layout(img_off=img_off, text_off=text_off,
                  grp_off=np.asarray(grp_off, np.int32), grp_img=np.asarray(grp_img, np.int32),
                  grp_cap=np.asarray(grp_cap, np.int32), kept_off=kept.astype(np.int32),
                  rows_per_image=rows_per_image, out_rows=out_rows)


def _to_dtype_values(x32: np.ndarray, dtype: str) -> np.ndarray:
    """float32 array -> float32 array holding values exactly representable in dtype."""
    if dtype == "f32":
        return x32
    import torch
    return torch.from_numpy(np.ascontiguousarray(x32)).to(torch.bfloat16).float().numpy()


def make_weights(w: Workload) -> Dict[str, np.ndarray]:
    """Selector weights in the layout the library takes (output-major rows)."""
    rng = _rng(w.cfg_id, STREAM_WEIGHTS, 0)
    f = lambda shape, scale: (rng.standard_normal(shape, dtype=np.float32) * np.float32(scale))
    W_kqv = f((3 * w.h, w.d), 1.0 / math.sqrt(w.d))        # rows: K | Q | V output features
    W_text = f((w.h, w.d_text), 1.0 / math.sqrt(w.d_text))
    s_start = f((w.d,), 1.0)
    s_stop = f((w.d,), 1.0)
    return {k: _to_dtype_values(v, w.dtype) for k, v in
            dict(W_kqv=W_kqv, W_text=W_text, s_start=s_start, s_stop=s_stop).items()}


def make_image(w: Workload, index: int, n: int) -> np.ndarray:
    rng = _rng(w.cfg_id, STREAM_VISUAL, index)
    centres = rng.standard_normal((N_CLUSTERS, w.d), dtype=np.float32)
    assign = rng.integers(0, N_CLUSTERS, size=n)
    noise = rng.standard_normal((n, w.d), dtype=np.float32)
    x = centres[assign] + np.float32(CLUSTER_NOISE) * noise
    return _to_dtype_values(x, w.dtype)


def make_text(w: Workload, index: int) -> np.ndarray:
    rng = _rng(w.cfg_id, STREAM_TEXT, index)
    return _to_dtype_values(rng.standard_normal((w.text_len, w.d_text), dtype=np.float32), w.dtype)


def make_inputs(w: Workload, images: Optional[List[int]] = None,
                batch_index: int = 0) -> Dict[str, np.ndarray]:
    """All inputs of a workload as float32 arrays holding dtype-exact values.

    ``images`` restricts the batch to a subset (same per-image content).
    ``batch_index`` k > 0 draws the k-th further batch of a stream of batches:
    the same image sizes (so the same layout) with fresh content, image i
    drawn as image k * batch + i of the workload's streams."""
    sizes = image_sizes(w)
    idx = list(range(w.batch)) if images is None else list(images)
    base = batch_index * w.batch
    X = np.concatenate([make_image(w, base + i, sizes[i]) for i in idx], axis=0)
    E = np.concatenate([make_text(w, base + i) for i in idx], axis=0)
    out = make_weights(w)
    out.update(X=X, E_text=E)
    return out


STREAM_DENOISER = 5
DENOISER_FIELDS = ("ln1_g", "ln1_b", "W_v", "b_v", "W_o", "b_o", "ln2_g", "ln2_b", "W_1", "b_1",
                   "W_2", "b_2")


def make_denoiser_inputs(w: Workload, T: int) -> Dict[str, np.ndarray]:
    """Seeded inputs of the noise gate and denoiser block for T tokens of width
    w.d: gate weights alpha ~ U[0, 1] (the first two tokens get exactly 1 and
    0), noise eps ~ N(0, I) rounded to bfloat16, random-init block parameters
    (weights N(0, 1/fan_in) rounded to bfloat16 in [out, in] layout, biases
    N(0, 0.02^2), LayerNorm scales 1 + N(0, 0.1^2) and shifts N(0, 0.1^2),
    float32)."""
    d = w.d
    rng = _rng(w.cfg_id, STREAM_DENOISER, 0)
    bf = lambda a: _to_dtype_values(a, "bf16")
    out = {"alpha": rng.uniform(0.0, 1.0, T).astype(np.float32),
           "eps": bf(rng.standard_normal((T, d), dtype=np.float32))}
    if T >= 2:
        out["alpha"][:2] = (1.0, 0.0)
    shapes = {"W_v": (d, d), "W_o": (d, d), "W_1": (4 * d, d), "W_2": (d, 4 * d)}
    for name in DENOISER_FIELDS:
        if name in shapes:
            n_out, n_in = shapes[name]
            out[name] = bf(rng.standard_normal((n_out, n_in), dtype=np.float32)
                           * np.float32(1.0 / math.sqrt(n_in)))
        elif name.startswith("ln") and name.endswith("_g"):
            out[name] = (1.0 + 0.1 * rng.standard_normal(d)).astype(np.float32)
        elif name.startswith("ln"):
            out[name] = (0.1 * rng.standard_normal(d)).astype(np.float32)
        else:
            n = 4 * d if name == "b_1" else d
            out[name] = (0.02 * rng.standard_normal(n)).astype(np.float32)
    return out


STREAM_ENCODER = 6
ENCODER_FIELDS = ("ln1_g", "ln1_b", "W_qkv", "b_qkv", "W_o", "b_o", "ln2_g", "ln2_b", "W_1", "b_1",
                  "W_2", "b_2")
ENCODER_BLOCKS = 2


def make_encoder_inputs(w: Workload) -> Dict[str, object]:
    """Seeded random-init parameters of the cross-modal input encoder for
    width w.d: the text projection W_p [d, d_text] and two blocks (weights
    N(0, 1/fan_in) rounded to bfloat16 in [out, in] layout, biases
    N(0, 0.02^2), LayerNorm scales 1 + N(0, 0.1^2) and shifts N(0, 0.1^2),
    float32).  Returns {"W_p": ..., "blocks": [dict, dict]}."""
    d = w.d
    rng = _rng(w.cfg_id, STREAM_ENCODER, 0)
    bf = lambda a: _to_dtype_values(a, "bf16")
    W_p = bf(rng.standard_normal((d, w.d_text), dtype=np.float32)
             * np.float32(1.0 / math.sqrt(w.d_text)))
    shapes = {"W_qkv": (3 * d, d), "W_o": (d, d), "W_1": (4 * d, d), "W_2": (d, 4 * d)}
    sizes = {"b_qkv": 3 * d, "b_1": 4 * d}
    blocks = []
    for _ in range(ENCODER_BLOCKS):
        blk = {}
        for name in ENCODER_FIELDS:
            if name in shapes:
                n_out, n_in = shapes[name]
                blk[name] = bf(rng.standard_normal((n_out, n_in), dtype=np.float32)
                               * np.float32(1.0 / math.sqrt(n_in)))
            elif name.startswith("ln") and name.endswith("_g"):
                blk[name] = (1.0 + 0.1 * rng.standard_normal(d)).astype(np.float32)
            elif name.startswith("ln"):
                blk[name] = (0.1 * rng.standard_normal(d)).astype(np.float32)
            else:
                blk[name] = (0.02 * rng.standard_normal(sizes.get(name, d))).astype(np.float32)
        blocks.append(blk)
    return {"W_p": W_p, "blocks": blocks}


def load_stop_bias() -> Dict[str, float]:
    if not os.path.exists(STOP_BIAS_FILE):
        return {}
    with open(STOP_BIAS_FILE) as f:
        return {k: float(v["b_stop"]) for k, v in json.load(f).items()}


def stop_bias(w: Workload) -> float:
    table = load_stop_bias()
    if w.name not in table:
        raise KeyError(f"no calibrated stop bias for workload {w.name!r} in {STOP_BIAS_FILE}")
    return table[w.name]
