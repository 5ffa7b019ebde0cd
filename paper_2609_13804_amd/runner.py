"""Device buffers for one batch and the three library calls in order
(DeviceRun), and a stream of batches overlapped across streams (Pipeline).

Plumbing only: torch allocates HBM and provides the streams and events; every
stage runs in libstepprune's kernels through the binding.
"""
import copy
import os
from dataclasses import dataclass
from typing import Dict, Optional

import numpy as np
import torch

from . import binding as sp
from . import workloads as W


def torch_dtype(dtype: str):
    return torch.float32 if dtype == "f32" else torch.bfloat16


@dataclass
class Sizes:
    T_vis: int
    T_txt: int
    B: int
    G: int
    max_group: int
    max_cap: int
    kept_total: int


def _storage_rows(a: np.ndarray) -> np.ndarray:
    """The text rows as uploaded: a batch without text still gets one zero row
    of storage, because the ABI takes a valid E_text pointer (no kernel reads
    a row outside the ones text_off spans)."""
    return a if a.shape[0] > 0 else np.zeros((1,) + a.shape[1:], a.dtype)


class DeviceRun:
    """All inputs, outputs and workspaces of one batch, resident on the GPU."""

    def __init__(self, w: W.Workload, inputs: Dict[str, np.ndarray], layout: W.Layout,
                 b_stop: float, device="cuda", trace_steps: int = 0, flags: int = 0,
                 caps: Optional[np.ndarray] = None, max_group: Optional[int] = None,
                 logits: bool = False):
        """trace_steps > 0 allocates the per-step trace (SP_TRACE); with
        ``logits`` every record also holds the step's whole logit vector
        (SP_LOGITS)."""
        self.w = w
        self.layout = layout
        self.b_stop = float(b_stop)
        logits = logits and trace_steps > 0
        self.flags = flags | (sp.SP_TRACE if trace_steps > 0 else 0) | (sp.SP_LOGITS if logits else 0)
        self.trace_steps = trace_steps
        self.g = w.g
        self.trace_base = 4 if w.g == 1 else w.g + 3
        self.trace_width = self.trace_base
        dev = torch.device(device)
        tdt = torch_dtype(w.dtype)
        up = lambda a, dt=tdt: torch.from_numpy(np.ascontiguousarray(a)).to(device=dev, dtype=dt)
        upi = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)
        self.X = up(inputs["X"])
        self.E = up(_storage_rows(inputs["E_text"]))
        self.W_kqv = up(inputs["W_kqv"])
        self.W_text = up(inputs["W_text"])
        self.s_start = up(inputs["s_start"])
        self.s_stop = up(inputs["s_stop"])
        caps = layout.grp_cap if caps is None else np.asarray(caps, np.int32)
        sizes = np.diff(layout.grp_off)
        self.caps_host = caps
        kept_per_img = np.zeros(layout.batch + 1, np.int64)
        for g in range(layout.groups):
            kept_per_img[layout.grp_img[g] + 1] += min(int(caps[g]) * w.g, int(sizes[g]))
        kept_off = np.cumsum(kept_per_img).astype(np.int32)
        self.img_off = upi(layout.img_off)
        self.text_off = upi(layout.text_off)
        self.grp_off = upi(layout.grp_off)
        self.grp_img = upi(layout.grp_img)
        self.grp_cap = upi(caps)
        self.kept_off = upi(kept_off)
        self.kept_off_host = kept_off
        self.sizes = Sizes(T_vis=int(layout.img_off[-1]), T_txt=int(layout.text_off[-1]),
                           B=layout.batch, G=layout.groups,
                           max_group=int(max_group if max_group is not None else
                                         (sizes.max() if sizes.size else 0)),
                           max_cap=int(max(1, max((min(int(c) * w.g, int(n)) for c, n in zip(caps, sizes)),
                                                  default=1))),
                           kept_total=int(kept_off[-1]))
        s = self.sizes
        if logits:
            self.trace_width = self.trace_base + s.max_group + 1
        self.dims = sp.dims(w.d, w.d_text, w.h, sp.SP_F32 if w.dtype == "f32" else sp.SP_BF16)
        if w.layout == "padded":
            self.layout_code = sp.SP_LAYOUT_PADDED
            self.rows_per_image = layout.rows_per_image
            self.out_rows = s.B * layout.rows_per_image
        else:
            self.layout_code = sp.SP_LAYOUT_PACKED
            self.rows_per_image = 0
            self.out_rows = s.kept_total + s.T_txt
        nb = lambda which: sp.stepprune_workspace_bytes(which, self.dims, s.T_vis, s.T_txt, s.B,
                                                        s.G, s.max_group, s.max_cap)
        self.ws_bytes = [nb(sp.STAGE_PROJECT), nb(sp.STAGE_SELECT), nb(sp.STAGE_COMPACT)]
        if min(self.ws_bytes) == 0:
            raise ValueError("workspace size query rejected the sizes")
        self._alloc_outputs()

    def _alloc_outputs(self):
        """Outputs and workspaces (zero-filled workspaces: their error words start clear)."""
        s, w, dev, tdt = self.sizes, self.w, self.X.device, self.X.dtype
        self.KQV = torch.empty((s.T_vis + 2, 3 * w.h), dtype=tdt, device=dev)
        self.ctx = torch.empty((s.B, w.h), dtype=torch.float32, device=dev)
        self.kept_idx = torch.full((max(1, s.kept_total),), -1, dtype=torch.int32, device=dev)
        self.kept_cnt = torch.zeros(s.B, dtype=torch.int32, device=dev)
        self.grp_cnt = torch.zeros(max(1, s.G), dtype=torch.int32, device=dev)
        self.trace = (torch.empty((s.G, self.trace_steps, self.trace_width), dtype=torch.float32,
                                  device=dev)
                      if self.trace_steps > 0 else None)
        self.seq_info = torch.zeros(s.B + (self.layout_code == sp.SP_LAYOUT_PACKED), dtype=torch.int32,
                                    device=dev)
        self.out = (torch.zeros((self.out_rows, w.d), dtype=tdt, device=dev)
                    if w.d_text == w.d else None)
        self.ws = [torch.zeros(n, dtype=torch.uint8, device=dev) for n in self.ws_bytes]

    def sibling(self, inputs: Optional[Dict[str, np.ndarray]] = None):
        """Another run with outputs and workspaces of its own, for work on a
        second stream.  It shares the weights and offsets (read only), and the
        visual and text tokens too unless ``inputs`` gives a batch of the same
        shape (X and E_text are then uploaded for it)."""
        other = copy.copy(self)
        if inputs is not None:
            up = lambda a, ref: torch.from_numpy(np.ascontiguousarray(a)).to(device=ref.device,
                                                                             dtype=ref.dtype)
            E = _storage_rows(inputs["E_text"])
            if inputs["X"].shape != tuple(self.X.shape) or E.shape != tuple(self.E.shape):
                raise ValueError("a sibling's batch must have the same shape")
            other.X = up(inputs["X"], self.X)
            other.E = up(E, self.E)
        other._alloc_outputs()
        return other

    # ---------------------------------------------------------------- stages
    def project(self, stream=None, g_text: float = 1.0, ln_eps: float = 1e-5, events=None):
        s = self.sizes
        return sp.stepprune_project(self.dims, self.X, s.T_vis, self.s_start, self.s_stop,
                                    self.W_kqv, self.E, self.text_off, s.B, s.T_txt, self.W_text,
                                    g_text, ln_eps, self.KQV, self.ctx, self.ws[0],
                                    self.ws_bytes[0], stream, events=events)

    def select(self, stream=None, b_stop: Optional[float] = None, flags: Optional[int] = None,
               events=None):
        s = self.sizes
        return sp.stepprune_select(self.dims, self.KQV, self.ctx, s.T_vis, self.img_off, s.B,
                                   self.grp_off, self.grp_img, self.grp_cap, s.G, s.max_group,
                                   s.max_cap, self.kept_off,
                                   self.b_stop if b_stop is None else b_stop, self.g,
                                   self.flags if flags is None else flags, self.kept_idx,
                                   self.kept_cnt, self.grp_cnt, self.trace, self.trace_steps,
                                   self.ws[1], self.ws_bytes[1], stream, events=events)

    def trajectory_outputs(self, pstop_steps: int = 0):
        """Buffers for select_trajectory: (s [T_vis], kbar [G], pstop [G, steps] or None)."""
        s_, dev = self.sizes, self.X.device
        ts = torch.zeros(max(1, s_.T_vis), dtype=torch.float32, device=dev)
        kb = torch.zeros(max(1, s_.G), dtype=torch.float32, device=dev)
        ps = (torch.empty((s_.G, pstop_steps), dtype=torch.float32, device=dev)
              if pstop_steps > 0 else None)
        return ts, kb, ps

    def select_trajectory(self, tau: float, beta: float, flags: Optional[int] = None,
                          pstop_steps: int = 0, stream=None, out=None, events=None):
        """The selection and the trajectory sums of Eqs. 5-7 along it (g = 1);
        returns (s [T_vis], kbar [G], pstop [G, pstop_steps] or None), in
        ``out`` (from trajectory_outputs) when given."""
        s_ = self.sizes
        ts, kb, ps = out if out is not None else self.trajectory_outputs(pstop_steps)
        pstop_steps = 0 if ps is None else int(ps.shape[1])
        tj = sp.trajectory(tau, beta, ts, kb, ps, pstop_steps)
        sp.stepprune_select_trajectory(self.dims, self.KQV, self.ctx, s_.T_vis, self.img_off, s_.B,
                                       self.grp_off, self.grp_img, self.grp_cap, s_.G,
                                       s_.max_group, s_.max_cap, self.kept_off, self.b_stop, self.g,
                                       self.flags if flags is None else flags, self.kept_idx,
                                       self.kept_cnt, self.grp_cnt, self.trace, self.trace_steps, tj,
                                       self.ws[1], self.ws_bytes[1], stream, events=events)
        return ts, kb, ps

    def compact(self, stream=None, events=None):
        s = self.sizes
        return sp.stepprune_compact(self.dims, self.X, self.img_off, self.E, self.text_off,
                                    self.kept_idx, self.kept_off, self.kept_cnt, s.B,
                                    self.layout_code, self.rows_per_image, self.out_rows, self.out,
                                    self.seq_info, self.ws[2], self.ws_bytes[2], stream,
                                    events=events)

    def run(self, stream=None):
        self.project(stream)
        self.select(stream)
        if self.out is not None:
            self.compact(stream)

    # ---------------------------------------------------------------- graphs
    def capture(self, stages=("project", "select", "compact")):
        """A HIP graph of the given stages on this run's buffers (one step by
        default), replayed with ``g.replay()`` on the current stream.  Every
        entry point only launches kernels, so a step captures whole; the
        stages are run once eagerly on the capture stream first."""
        todo = [getattr(self, st) for st in stages if st != "compact" or self.out is not None]
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for f in todo:
                f()
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for f in todo:
                f()
        return g

    def device_errors(self):
        return [sp.stepprune_read_device_error(ws) for ws in self.ws]

    # ---------------------------------------------------------------- results
    def kept_lists(self):
        cnt = self.kept_cnt.cpu().numpy()
        idx = self.kept_idx.cpu().numpy()
        off = self.kept_off_host
        return [idx[off[b]:off[b] + cnt[b]].tolist() for b in range(self.sizes.B)]

    def trace_logits(self):
        """SP_LOGITS: [G, trace_steps, max_group + 1] float32, every step's logit
        of each token slot (-inf where masked or past the group) and STOP last."""
        return self.trace[..., self.trace_base:].cpu().numpy()

    def trace_actions(self):
        """Per group: the taken candidates in order (-1 = STOP); with g > 1 per
        round the list of taken tokens, [-1] for STOP."""
        tr = self.trace.cpu().numpy()
        ids = np.ascontiguousarray(tr[..., :self.g]).view(np.int32)
        out = []
        for g in range(self.sizes.G):
            seq = []
            for t in range(self.trace_steps):
                a = int(ids[g, t, 0])
                if a == -2:
                    break
                if self.g == 1:
                    seq.append(a)
                else:
                    seq.append([int(x) for x in ids[g, t] if x != -3])
            out.append(seq)
        return out


class Pipeline:
    """A stream of batches through the three stages with the matrix-core work
    of later batches overlapping the recurrences of earlier ones.

    The recurrence of one batch occupies one compute unit per episode for
    most of a batch's time while the projection and Gram products need the
    whole chip, so batches are staggered: batch k's projection runs on one
    stream, in batch order, and its selection and compaction on select stream
    k mod ``streams``.  With ``split_gram`` the selection's Gram products
    (SP_GRAM_ONLY) join the projection stream and only the recurrence
    (SP_REUSE_GRAM) runs on the select stream; measured on the 16 x 576 batch
    this is slower (38K against 44K images/s): concurrent GEMMs of two
    batches fill each other's last tile rounds.  Batch k uses buffer slot k mod ``slots``, a
    DeviceRun with its own outputs and workspaces (and its own tokens when
    ``inputs`` are given; the weights are shared read-only):
    a slot's projection waits for the slot's previous select + compact, and
    its recurrence waits for its projection and Gram products.  More slots
    than select streams let the GEMM stream run ahead.  All streams use the
    default priority.

    The GEMM work goes to the caller's current stream, so the pipeline uses
    streams + 1 streams in all: at most three select streams keep every
    stream on a hardware queue of its own under HIP's default of four per
    process."""

    @staticmethod
    def max_streams() -> int:
        """Select streams that keep every stream of the pipeline (plus the
        caller's) on a hardware queue of its own: GPU_MAX_HW_QUEUES - 1 (HIP's
        default of four queues gives three)."""
        return max(1, int(os.environ.get("GPU_MAX_HW_QUEUES", "4")) - 1)

    def __init__(self, run: DeviceRun, slots: int = 4, streams: int = 3, split_gram: bool = False,
                 inputs=None):
        """``inputs``: None (every slot reads ``run``'s tokens) or one input
        dict per further slot (slots - 1 of them), so that the stream of
        batches reads fresh tokens from HBM rather than cached ones."""
        if not 1 <= streams <= self.max_streams():
            raise ValueError(f"streams must be 1..{self.max_streams()}")
        if slots < streams:
            raise ValueError("need at least one slot per select stream")
        if inputs is not None and len(inputs) != slots - 1:
            raise ValueError("one input batch per further slot")
        self.runs = [run] + [run.sibling(None if inputs is None else inputs[k])
                             for k in range(slots - 1)]
        self.proj_stream = torch.cuda.current_stream()
        self.sel_streams = [torch.cuda.Stream() for _ in range(streams)]
        self.projected = [torch.cuda.Event() for _ in self.runs]
        self.done = [torch.cuda.Event() for _ in self.runs]
        self.split_gram = split_gram
        self.k = 0
        self.graphs = None

    def use_graphs(self):
        """Replay each slot's stages from HIP graphs (the projection, and the
        selection with compaction) instead of enqueuing their kernels one by
        one; the streams and events between them stay as they are."""
        if self.split_gram:
            raise ValueError("graphs replay whole stages")
        self.graphs = [(r.capture(("project",)), r.capture(("select", "compact"))) for r in self.runs]
        torch.cuda.synchronize()

    def issue(self):
        """Queue the next batch (nothing waits on the host)."""
        s = self.k % len(self.runs)
        r, ps = self.runs[s], self.proj_stream
        ss = self.sel_streams[self.k % len(self.sel_streams)]
        if self.k >= len(self.runs):
            ps.wait_event(self.done[s])
        if self.graphs is not None:
            gp, gs = self.graphs[s]
            with torch.cuda.stream(ps):
                gp.replay()
            self.projected[s].record(ps)
            ss.wait_event(self.projected[s])
            with torch.cuda.stream(ss):
                gs.replay()
            self.done[s].record(ss)
            self.k += 1
            return
        r.project(ps.cuda_stream)
        if self.split_gram:
            r.select(ps.cuda_stream, flags=r.flags | sp.SP_GRAM_ONLY)
        self.projected[s].record(ps)
        ss.wait_event(self.projected[s])
        r.select(ss.cuda_stream, flags=r.flags | (sp.SP_REUSE_GRAM if self.split_gram else 0))
        if r.out is not None:
            r.compact(ss.cuda_stream)
        self.done[s].record(ss)
        self.k += 1
