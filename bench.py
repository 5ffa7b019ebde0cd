#!/usr/bin/env python3
"""Throughput of StepPrune's inference-time selection path on one MI355X.

One step is the whole path (Algorithm 1) over one batch already resident in
HBM: stepprune_project (projection GEMM + text context), stepprune_select
(per-group Gram products + the pointer recurrence with STOP) and
stepprune_compact (gather into the prefill buffer).  The default batch is
the LLaVA-1.5-shaped one: 16 images x 576 tokens x 4096, bf16, selector
hidden width 1024, cap 192, STOP bias set so that the mean retained count is
about 64, compaction into 576 + 64 prefill rows.

Two timed passes over K steps each, after W untimed warm-up steps:

  * single stream: the batches one after another on one stream, with per-stage
    and per-kernel times from HIP events the library records on that stream
    ("single_stream", "stages_us", "kernels_us", "stage_roofline");
  * pipelined (the reported "value", whole-job throughput): projections on one
    stream in batch order and each batch's select + compact on one of S select
    streams over a ring of buffer slots (runner.Pipeline), so that one batch's
    projection and Gram products run beside earlier batches' recurrences; each
    slot holds its own seeded batch of the same shape (over 256 MB of tokens in
    all on the default batch, more than the Infinity Cache holds); at least 64
    untimed batches fill and warm the pipeline first.

Prints one JSON line.  "roofline" covers the kernel with the largest share of
the GPU (kernel time x fraction of the compute units it occupies), with its HBM
traffic from the committed counter summary; "measured_peaks" adds rates this
GPU reaches on library work; "cpu_baseline" is the float64 oracle timed on this
host's cores over a bounded sample of the same batch.

    python bench.py [--gpus 1] [--steps 50] [--warmup 10] [--streams 3] [--slots 6]
                    [--workload llava15_bf16] [--trajectory TAU BETA] [--steady R] [--denoise]
                    [--encoder] [--lds-probe] [--shared-inputs]
"""
import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "images/sec and µs/image through selector+compaction (N=576, bf16), % roofline"

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 matrix
PEAK_F32_MATRIX_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
# float32 FMA without packed instructions: 256 CU x 4 SIMD x 16 lanes x 2 flop x 2.4 GHz
PEAK_F32_VALU_TFLOPS = 78.6
# LDS reads: 256 B/clk per CU x 256 CUs x 2.4 GHz, the rate the LDS probe
# (csrc/probe.hip, bench.py --lds-probe) measures on gfx950 with 16-byte reads;
# every run also reports its own probe measurement in measured_peaks
PEAK_LDS_GBS = 157286.0
NOMINAL_CLOCK_HZ = 2.4e9
N_CU = 256

# minimum untimed warm-up of the pipelined pass, in batches (about 25 ms of
# overlapped work on the 16-image batch)
PIPE_WARMUP_BATCHES = 64


class HipEvents:
    """Raw hipEvent_t handles through libamdhip64 (the library records them on the
    stream it launches on)."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        ev = ctypes.c_void_p()
        if self.hip.hipEventCreate(ctypes.byref(ev)) != 0:
            raise RuntimeError("hipEventCreate failed")
        return ev.value

    def record(self, ev, stream):
        if self.hip.hipEventRecord(ev, stream) != 0:
            raise RuntimeError("hipEventRecord failed")

    def ms(self, a, b):
        out = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(out), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(out.value)

    def destroy(self, ev):
        self.hip.hipEventDestroy(ev)


def _ensure_built():
    lib = os.path.join(ROOT, "paper_2609_13804_amd", "libstepprune.so")
    if not os.path.exists(lib):
        from paper_2609_13804_amd import build
        build.build()


def _episode_steps(caps, sizes, kept, g=1):
    """Rounds per episode: ceil(kept / g) token rounds, plus the STOP round
    unless the episode ended at its cap."""
    steps = []
    for c, n, k in zip(caps, sizes, kept):
        r = -(-int(k) // g)
        steps.append(r if r == int(c) else r + 1)
    return steps


def cpu_baseline(w, lay, b_stop, budget_s, single_thread=False, gpu_kept=None):
    """The oracle (float64 NumPy, as written) over a bounded sample of the batch:
    chunks of up to 4 images, passing over the batch again until the oracle has
    run for the time budget.  With single_thread the BLAS pool is limited to
    one thread (the selection loop is single-threaded Python either way).
    With gpu_kept (the GPU's kept lists of the batch) the sampled images'
    oracle sets are compared with them, outside the timed region."""
    import contextlib
    limit = contextlib.nullcontext()
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
        if single_thread:
            limit = threadpool_limits(1)
            threads = 1
    except Exception:
        threads = 1 if single_thread else (os.cpu_count() or 1)
    with limit:
        return _oracle_sample(w, b_stop, budget_s, threads, gpu_kept)


def _oracle_sample(w, b_stop, budget_s, threads, gpu_kept=None):
    import numpy as np
    import oracle
    from paper_2609_13804_amd import workloads as W
    done = 0
    elapsed = 0.0
    chunk = max(1, min(4, w.batch))
    images = list(range(w.batch))
    chunks = [images[i:i + chunk] for i in range(0, w.batch, chunk)]
    k = 0
    equal = {}                                 # image -> oracle set == GPU set
    while elapsed < budget_s:
        sub = chunks[k % len(chunks)]
        k += 1
        inp, sl = W.make_inputs(w, sub), W.make_layout(w, sub)     # not timed
        t0 = time.perf_counter()
        KQV = oracle.project(inp["X"], inp["s_start"], inp["s_stop"], inp["W_kqv"], w.dtype)
        ctx = oracle.text_context(inp["E_text"], sl.text_off, inp["W_text"])
        res = oracle.select(KQV, ctx, sl.img_off, sl.grp_off, sl.grp_img, sl.grp_cap, b_stop, w.h,
                            keep_steps=False, g=w.g)
        if w.d_text == w.d:
            oracle.compact(inp["X"], sl.img_off, inp["E_text"], sl.text_off, res.kept, w.layout,
                           sl.rows_per_image, np.zeros((sl.out_rows, w.d)))
        elapsed += time.perf_counter() - t0
        done += len(sub)
        if gpu_kept is not None:
            for i, b in enumerate(sub):
                equal[b] = list(res.kept[i]) == list(gpu_kept[b])
    out = {"value": done / elapsed, "unit": "images/s", "cores": int(threads), "kind": "oracle",
           "sample": f"{done} images ({done / w.batch:.2f} passes over the {w.batch}-image "
                     f"{w.name} batch, chunks of {chunk}) of project + select + compact in "
                     f"float64, {elapsed:.1f} s"}
    if gpu_kept is not None:
        out["parity"] = {"images_compared": len(equal), "kept_sets_equal": int(sum(equal.values())),
                         "how": "the oracle end to end from the raw inputs (its own float64 "
                                "projection) against the GPU's kept lists of the same images; "
                                "bfloat16 sets may differ at near-ties that the stored-value "
                                "rounding flips (the parity tests check each such divergence)"}
    return out


def steady_pass(w, R, b_stop, hip, stream, t_scan_roof, ref_kept, longest, steps=10, warmup=2):
    """Secondary, labelled steady-state figure for the selection stage: R copies
    of the batch in one call of each stage, so the recurrence runs R times as
    many episodes at once (up to one per compute unit) and the per-batch select
    time approaches its throughput rather than the longest episode's latency."""
    import numpy as np
    from paper_2609_13804_amd import workloads as W
    from paper_2609_13804_amd.runner import DeviceRun
    inp = W.make_inputs(w)
    inp["X"] = np.tile(inp["X"], (R, 1))
    inp["E_text"] = np.tile(inp["E_text"], (R, 1))
    lay = W.make_layout(w, list(range(w.batch)) * R)
    run = DeviceRun(w, inp, lay, b_stop)
    run.flags = 0
    del inp
    for _ in range(warmup):
        run.run(stream)
    names = ["sel0", "gram0", "gram1", "rec0", "rec1", "sel1"]
    evs = [{n: hip.create() for n in names} for _ in range(steps)]
    for e in evs:
        run.project(stream)
        hip.record(e["sel0"], stream)
        run.select(stream, events=[e["gram0"], e["gram1"], e["rec0"], e["rec1"]])
        hip.record(e["sel1"], stream)
        run.compact(stream)
    import torch
    torch.cuda.synchronize()
    if any(run.device_errors()):
        raise RuntimeError(f"device error words {run.device_errors()}")
    kept = run.kept_lists()
    if any(kept[r * w.batch:(r + 1) * w.batch] != ref_kept for r in range(R)):
        raise RuntimeError("a copy of the batch selected differently from the batch alone")
    mean = lambda a, b: float(np.mean([1e3 * hip.ms(e[a], e[b]) for e in evs]))
    sel, gram, rec = mean("sel0", "sel1"), mean("gram0", "gram1"), mean("rec0", "rec1")
    for e in evs:
        for ev in e.values():
            hip.destroy(ev)
    return {"copies": R, "images": R * w.batch, "episodes": int(lay.grp_off.size - 1),
            "select_us": round(sel, 2), "gram_us": round(gram, 2), "recurrence_us": round(rec, 2),
            "select_us_per_batch": round(sel / R, 2),
            "recurrence_us_per_step_longest_episode": round(rec / max(1, longest), 3),
            "frac_keyscan_roofline": round(R * t_scan_roof / (sel * 1e-6), 4),
            "note": "secondary figure: R copies of the batch per call of each stage; "
                    "not the headline value"}


def gate_denoise_pass(w, K, hip, stream, mfma_peak):
    """The training pathway's noise gate and masked denoiser (stepprune_gate_denoise)
    on the batch's visual tokens: mean time of the whole block over K calls
    (HIP events around it) and its matrix throughput; 20 T d^2 flop (value and
    output projections, the 4d MLP)."""
    import numpy as np
    import torch
    from paper_2609_13804_amd import binding as sp
    from paper_2609_13804_amd import workloads as W
    T = int(W.make_layout(w).img_off[-1])
    dev = torch.device("cuda")
    inp = W.make_denoiser_inputs(w, T)
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev, torch.bfloat16)
    f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev)
    t = {k: (bf(v) if k.startswith("W_") else f32(v)) for k, v in inp.items()
         if k in W.DENOISER_FIELDS}
    X = bf(W.make_inputs(w)["X"])
    eps, alpha = bf(inp["eps"]), f32(inp["alpha"])
    del inp
    dm = sp.dims(w.d, w.d_text, w.h, sp.SP_BF16)
    ws_bytes = sp.stepprune_workspace_bytes(sp.STAGE_GATE, dm, T, 0, 1, 0, 0, 0)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device=dev)
    out = torch.empty((T, w.d), dtype=torch.bfloat16, device=dev)
    params = sp.denoiser(**t)
    for _ in range(3):
        sp.stepprune_gate_denoise(dm, X, T, alpha, eps, params, out, ws, ws_bytes, stream)
    evs = [(hip.create(), hip.create()) for _ in range(K)]
    for e in evs:
        sp.stepprune_gate_denoise(dm, X, T, alpha, eps, params, out, ws, ws_bytes, stream,
                                  events=[e[0], e[1]])
    torch.cuda.synchronize()
    if sp.stepprune_read_device_error(ws):
        raise RuntimeError("device error in the gate and denoiser")
    us = float(np.mean([1e3 * hip.ms(a, b) for a, b in evs]))
    for a, b in evs:
        hip.destroy(a)
        hip.destroy(b)
    flop = 20.0 * T * w.d * w.d
    achieved = flop / (us * 1e-6) / 1e12
    return {"tokens": T, "d": w.d, "us": round(us, 2), "algorithmic": f"{flop * 1e-12:.4f} TFLOP",
            "achieved_tflops": round(achieved, 2), "frac": round(achieved / mfma_peak, 4),
            "bound": "mfma"}


def encoder_pass(w, K, hip, stream, mfma_peak, causal=False):
    """The cross-modal input encoder (stepprune_encode, Eq. 3) on the batch:
    mean time of the whole call over K calls (HIP events around it) and its
    matrix throughput.  Algorithmic flop: the text product 2 T_txt d_text d;
    per block 24 S d^2 for the four products over the S = T_vis + T_txt
    sequence rows and 4 S_b^2 d for each image's attention (q k^T and p v;
    half of it when causal)."""
    import numpy as np
    import torch
    from paper_2609_13804_amd import binding as sp
    from paper_2609_13804_amd import workloads as W
    lay = W.make_layout(w)
    inp = W.make_inputs(w)
    params = W.make_encoder_inputs(w)
    dev = torch.device("cuda")
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev, torch.bfloat16)
    f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev)
    B = lay.batch
    T_vis, T_txt = int(lay.img_off[-1]), int(lay.text_off[-1])
    seqs = np.diff(lay.img_off).astype(np.int64) + np.diff(lay.text_off)
    max_seq = int(seqs.max())
    X, E, Wp = bf(inp["X"]), bf(inp["E_text"]), bf(params["W_p"])
    blk = [{k: (bf(v) if k.startswith("W_") else f32(v)) for k, v in b.items()}
           for b in params["blocks"]]
    del inp, params
    io = torch.from_numpy(lay.img_off.astype(np.int32)).to(dev)
    to = torch.from_numpy(lay.text_off.astype(np.int32)).to(dev)
    dm = sp.dims(w.d, w.d_text, w.h, sp.SP_BF16)
    ws_bytes = sp.stepprune_workspace_bytes(sp.STAGE_ENCODE, dm, T_vis, T_txt, B, 0, max_seq, 0)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device=dev)
    H = torch.empty((T_vis, w.d), dtype=torch.bfloat16, device=dev)
    blocks = sp.encoder_blocks(blk)
    flags = sp.SP_ENC_CAUSAL if causal else 0
    call = lambda ev=None: sp.stepprune_encode(dm, X, T_vis, io, B, E, to, T_txt, Wp, 1.0, blocks,
                                               max_seq, flags, H, ws, ws_bytes, stream, events=ev)
    for _ in range(3):
        call()
    evs = [(hip.create(), hip.create()) for _ in range(K)]
    for e in evs:
        call([e[0], e[1]])
    torch.cuda.synchronize()
    if sp.stepprune_read_device_error(ws):
        raise RuntimeError("device error in the encoder")
    us = float(np.mean([1e3 * hip.ms(a, b) for a, b in evs]))
    for a, b in evs:
        hip.destroy(a)
        hip.destroy(b)
    S = T_vis + T_txt
    attn = float((seqs.astype(np.float64) ** 2).sum()) * 4.0 * w.d * (0.5 if causal else 1.0)
    flop = 2.0 * T_txt * w.d_text * w.d + W.ENCODER_BLOCKS * (24.0 * S * w.d * w.d + attn)
    achieved = flop / (us * 1e-6) / 1e12
    return {"images": B, "sequence_rows": S, "d": w.d, "heads": w.d // 128, "us": round(us, 2),
            "us_per_image": round(us / B, 2), "attention": "causal" if causal else "bidirectional",
            "algorithmic": f"{flop * 1e-12:.4f} TFLOP", "achieved_tflops": round(achieved, 2),
            "frac": round(achieved / mfma_peak, 4), "bound": "mfma"}


def host_info():
    """The host the CPU baseline ran on: CPU model, cores visible to this
    process, and the BLAS library NumPy's products use with its thread count."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    info = {"cpu_model": model, "cpu_count": os.cpu_count(),
            "affinity": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None}
    try:
        from threadpoolctl import threadpool_info
        info["blas"] = [{"api": i.get("internal_api"), "threads": i.get("num_threads")}
                        for i in threadpool_info() if i.get("user_api") == "blas"]
    except Exception:
        info["blas"] = None
    return info


def measured_peaks():
    """Rates this GPU reaches on plain library work, the second denominator for
    the stage fractions: HBM from a 1 GiB device-to-device copy (bytes read plus
    bytes written), bf16 matrix throughput from the best of torch's bf16
    matmuls (hipBLASLt) over three shapes.  Timed with events on torch's
    current stream, where they run."""
    import torch
    res = {}
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda").random_(0, 255)
    dst = torch.empty_like(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(3):
        dst.copy_(src)
    e0.record()
    for _ in range(10):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    res["hbm_copy_GBs"] = round(2 * n * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e9, 1)
    del src, dst
    # a square shape, a tall one, and the 16-image batch's projection (without
    # its START / STOP rows); X [M, K] times W^T with W stored [N, K], the
    # layout the library's projection takes (a two-dimensional product, no batch)
    rates = {}
    for (mm, kk, nn) in [(8192, 8192, 8192), (16384, 4096, 4096), (9216, 4096, 3072)]:
        a = torch.randn(mm, kk, device="cuda").to(torch.bfloat16)
        b = torch.randn(nn, kk, device="cuda").to(torch.bfloat16)
        for _ in range(3):
            c = a @ b.t()
        e0.record()
        for _ in range(10):
            c = a @ b.t()
        e1.record()
        torch.cuda.synchronize()
        rates[f"{mm}x{kk}x{nn}"] = round(2.0 * mm * kk * nn * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e12, 1)
        del a, b, c
    torch.cuda.empty_cache()
    res.update(lds_probe())
    res["bf16_matmul_TFLOPs"] = max(rates.values())
    res["bf16_matmul_by_shape"] = rates
    res["how"] = ("1 GiB device copy (read + write bytes); the best torch bf16 matmul rate "
                  "(M x K x N) of the shapes listed; the LDS read probe; 10 launches each "
                  "after 3 warm-up")
    return res


def lds_probe(launches=10, warmup=3, iters=2048):
    """LDS read bandwidth of the whole chip: the probe kernel of
    libstepprune_probe.so (16-byte reads, two 512-thread workgroups per
    compute unit, 64 KB of LDS each), timed with events on torch's current
    stream, where it is launched."""
    import torch
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2609_13804_amd", "libstepprune_probe.so"))
    lib.stepprune_probe_lds.restype = ctypes.c_int
    lib.stepprune_probe_lds.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                        ctypes.c_void_p]
    threads = int(lib.stepprune_probe_lds_threads())
    blocks = 8 * N_CU
    out = torch.empty(blocks * threads, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream

    def launch():
        if lib.stepprune_probe_lds(out.data_ptr(), blocks, iters, stream) != 0:
            raise RuntimeError("LDS probe launch failed")
    for _ in range(warmup):
        launch()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(launches):
        launch()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / launches
    nbytes = blocks * threads * iters * 8 * 16
    gbs = nbytes / (us * 1e-6) / 1e9
    return {"lds_read_GBs": round(gbs, 1), "lds_probe_us": round(us, 2),
            "lds_read_B_per_clk_per_cu_at_2.4GHz": round(gbs * 1e9 / (N_CU * NOMINAL_CLOCK_HZ), 1),
            "lds_probe": f"{blocks} workgroups x {threads} threads x {iters} rounds of 8 "
                         f"16-byte reads ({nbytes / 1e9:.1f} GB a launch)"}


def copy_probe(mib):
    """A plain device-to-device copy of a known size: under rocprofv3 --pmc its
    FETCH_SIZE and WRITE_SIZE readings calibrate the same counters taken on the
    library's kernels (bytes counted per byte moved)."""
    import torch
    n = mib << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda").random_(0, 255)
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n, "launches": 5}), flush=True)
    return 0


def hbm_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter summary,
    or None when there is none or the kernel's source has changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{kernel}_{workload}.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            rec[k.strip()] = v.strip()
    digest = hashlib.sha256()
    for name in rec.get("source", "").split():
        src = os.path.join(ROOT, "paper_2609_13804_amd", "csrc", name)
        if not os.path.isfile(src):
            return None
        digest.update(open(src, "rb").read())
    if not rec.get("source") or digest.hexdigest() != rec.get("source_sha256"):
        return None
    return float(rec["bytes_per_launch"])


def trajectory_pass(run, tb, K, hip):
    """Select-stage time with the trajectory sums over the full rollout, beside
    the plain selection and the plain full rollout (g = 1 workloads), single
    stream, HIP events around each call."""
    import numpy as np
    import torch
    from paper_2609_13804_amd import binding as sp
    tau, beta = tb
    stream = torch.cuda.current_stream().cuda_stream
    outs = run.trajectory_outputs()
    variants = {
        "plain_select_us": lambda e: run.select(stream, flags=0, events=e),
        "full_rollout_select_us": lambda e: run.select(stream, flags=sp.SP_FULL_ROLLOUT, events=e),
        "traced_full_rollout_select_us": lambda e: run.select(
            stream, flags=sp.SP_FULL_ROLLOUT | (sp.SP_TRACE if run.trace is not None else 0),
            events=e),
        "trajectory_select_us": lambda e: run.select_trajectory(tau, beta, flags=sp.SP_FULL_ROLLOUT,
                                                                stream=stream, out=outs, events=e),
    }
    res = {"tau": tau, "beta": beta, "rollout": "full (SP_FULL_ROLLOUT)"}
    for name, fn in variants.items():
        for _ in range(3):
            fn(None)
        torch.cuda.synchronize()
        evs = [[hip.create() for _ in range(6)] for _ in range(K)]
        for e in evs:
            hip.record(e[0], stream)
            fn([e[1], e[2], e[3], e[4]])
            hip.record(e[5], stream)
        torch.cuda.synchronize()
        res[name] = round(float(np.mean([1e3 * hip.ms(e[0], e[5]) for e in evs])), 2)
        res[name.replace("select_us", "recurrence_us")] = round(
            float(np.mean([1e3 * hip.ms(e[3], e[4]) for e in evs])), 2)
        for e in evs:
            for ev in e:
                hip.destroy(ev)
    if any(run.device_errors()):
        raise RuntimeError(f"device error words {run.device_errors()}")
    res["kbar_mean"] = round(float(outs[1][:run.sizes.G].mean()), 4)
    return res


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llava15_bf16")
    ap.add_argument("--streams", type=int, default=3,
                    help="streams of the pipelined pass: select streams (staggered, at most 3) "
                         "or round-robin streams (rr); 1: no pipelined pass")
    ap.add_argument("--hw-queues", type=int, default=0,
                    help="set GPU_MAX_HW_QUEUES (at most 32) for this process before HIP starts, "
                         "to run more pipelined streams on queues of their own (0: leave it)")
    ap.add_argument("--slots", type=int, default=6,
                    help="buffer slots of the staggered pipelined pass (batches in flight)")
    ap.add_argument("--schedule", choices=["staggered", "staggered-gram", "rr"], default="staggered",
                    help="pipelined pass: projections on one stream ahead of select (Gram "
                         "products + recurrence) and compaction on per-slot streams "
                         "(staggered), the Gram products on the projection stream too "
                         "(staggered-gram: SP_GRAM_ONLY / SP_REUSE_GRAM), or whole batches "
                         "round-robin (rr)")
    ap.add_argument("--trajectory", type=float, nargs=2, metavar=("TAU", "BETA"), default=None,
                    help="also time the selection with the trajectory sums of Eqs. 5-7 over the "
                         "full rollout (stepprune_select_trajectory) against the plain selection")
    ap.add_argument("--steady", type=int, default=-1, metavar="R",
                    help="also time the selection stage on R copies of the batch in one call "
                         "(R x the episodes at once): a secondary steady-state figure; -1 (the "
                         "default): 256 / episodes copies when the batch has fewer than 128 "
                         "episodes (16 for the 16 x 576 batch), none otherwise; 0: none")
    ap.add_argument("--encoder", action="store_true",
                    help="also time the cross-modal input encoder of Eq. 3 (stepprune_encode, two "
                         "blocks over each image's visual and text tokens) on the batch")
    ap.add_argument("--denoise", action="store_true",
                    help="also time the training pathway's noise gate and masked denoiser "
                         "(stepprune_gate_denoise) on the batch's visual tokens")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=12.0,
                    help="seconds of oracle work for the CPU baseline sample")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB (5 launches), the "
                         "calibration for the FETCH_SIZE / WRITE_SIZE counters, and exit")
    ap.add_argument("--lds-probe", action="store_true",
                    help="only run the LDS read probe (10 timed launches), print its rate and exit")
    ap.add_argument("--shared-inputs", action="store_true",
                    help="pipelined pass: every slot reads the first batch's tokens (by default "
                         "each slot has its own seeded batch, so tokens come from HBM)")
    args = ap.parse_args(argv)
    if args.hw_queues:
        if not 1 <= args.hw_queues <= 32:
            print("--hw-queues must be 1..32", file=sys.stderr)
            return 2
        os.environ["GPU_MAX_HW_QUEUES"] = str(args.hw_queues)   # read when HIP starts
    if args.copy_probe_mib:
        return copy_probe(args.copy_probe_mib)
    if args.lds_probe:
        _ensure_built()
        print(json.dumps(lds_probe()), flush=True)
        return 0
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the selection path shards by image with no "
              "communication, and bench.py measures the one-GPU share (--gpus 1).",
              file=sys.stderr)
        return 2

    _ensure_built()
    import numpy as np
    import torch
    from paper_2609_13804_amd import workloads as W
    from paper_2609_13804_amd.runner import DeviceRun

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    torch.cuda.set_device(0)
    w = W.WORKLOADS[args.workload]
    lay = W.make_layout(w)
    b_stop = W.stop_bias(w)
    inp = W.make_inputs(w)
    run = DeviceRun(w, inp, lay, b_stop,
                    trace_steps=int(lay.grp_cap.max()) + 1 if args.trajectory is not None else 0)
    run.flags = 0      # the timed passes run the untraced kernels (a trace buffer is only
    del inp            # allocated for the traced variant of --trajectory)
    stream = torch.cuda.current_stream().cuda_stream
    hip = HipEvents()

    for _ in range(args.warmup):
        run.run()
    torch.cuda.synchronize()
    if any(run.device_errors()):
        raise RuntimeError(f"device error words {run.device_errors()}")

    K = args.steps
    names = ["step0", "proj0", "proj1", "projd", "gram0", "gram1", "rec0", "rec1", "seld",
             "gath0", "gath1", "step1"]
    evs = [{n: hip.create() for n in names} for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(K):
        e = evs[k]
        hip.record(e["step0"], stream)
        run.project(stream, events=[e["proj0"], e["proj1"]])
        hip.record(e["projd"], stream)
        run.select(stream, events=[e["gram0"], e["gram1"], e["rec0"], e["rec1"]])
        hip.record(e["seld"], stream)
        run.compact(stream, events=[e["gath0"], e["gath1"]])
        hip.record(e["step1"], stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    if any(run.device_errors()):
        raise RuntimeError(f"device error words {run.device_errors()}")

    def per_step_us(a, b):
        return np.array([1e3 * hip.ms(e[a], e[b]) for e in evs])

    spans = {"project": ("step0", "projd"), "select": ("projd", "seld"),
             "compact": ("seld", "step1"), "select_compact": ("projd", "step1"),
             "step": ("step0", "step1")}
    stage_t = {k: per_step_us(*v) for k, v in spans.items()}
    stages = {k: float(v.mean()) for k, v in stage_t.items()}
    stage_pct = {k: {"p10": float(np.percentile(v, 10)), "p50": float(np.median(v)),
                     "p90": float(np.percentile(v, 90))} for k, v in stage_t.items()}
    kern_spans = {"project_gemm": ("proj0", "proj1"), "gram_gemm": ("gram0", "gram1"),
                  "select_recurrence": ("rec0", "rec1"), "compact_gather": ("gath0", "gath1")}
    kernels = {k: float(per_step_us(*v).mean()) for k, v in kern_spans.items()}
    for e in evs:
        for ev in e.values():
            hip.destroy(ev)

    s = run.sizes
    sizes = np.diff(lay.grp_off)
    kept_g = run.grp_cnt.cpu().numpy()[:s.G]
    kept_b = run.kept_cnt.cpu().numpy()
    steps_g = _episode_steps(run.caps_host, sizes, kept_g, w.g)
    eb = 2 if w.dtype == "bf16" else 4
    L = np.diff(lay.text_off)

    mfma_peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_MATRIX_TFLOPS
    proj_flop = 2.0 * (s.T_vis + 2) * w.d * 3 * w.h * 1e-12
    text_flop = 2.0 * s.T_txt * w.d_text * w.h * 1e-12
    gram_flop = sum(2.0 * (2 * (n + 1) + 3) * (n + 2) * w.h for n in sizes) * 1e-12
    work = {
        # the projection launch also computes the text projection's tiles
        "project_gemm": ("mfma", proj_flop + text_flop, mfma_peak, "TFLOP/s"),
        "gram_gemm": ("mfma", gram_flop, mfma_peak, "TFLOP/s"),
        # round t reads n + 1 columns against a history of 1 + g (t - 1) entries
        "select_recurrence": ("alu", sum(2.0 * (n + 1) * (st + w.g * st * (st - 1) / 2)
                                         for n, st in zip(sizes, steps_g)) * 1e-12,
                              PEAK_F32_VALU_TFLOPS, "TFLOP/s"),
        "compact_gather": ("hbm", float(((kept_b + L) * w.d * eb * 2).sum() + kept_b.sum() * 4) * 1e-9,
                           PEAK_HBM_GBS, "GB/s"),
    }
    # The dominant kernel is the one that takes the largest share of the GPU:
    # kernel time x the fraction of compute units it occupies.  The recurrence
    # runs one workgroup per episode (16 of 256 CUs on the 16-image batch), so
    # a long recurrence can still be a small share of the chip; throughput
    # (the pipelined `value`) is bound by the kernels that fill the chip.
    NCU = 256
    share = {"project_gemm": 1.0, "gram_gemm": 1.0, "compact_gather": 1.0,
             "select_recurrence": min(1.0, s.G / NCU)}
    gpu_time = {k: v * share[k] for k, v in kernels.items()}
    dom = max(gpu_time, key=gpu_time.get)

    def roof(k):
        bound, amount, peak, unit = work[k]
        achieved = amount / (kernels[k] * 1e-6)
        return {"bound": bound, "achieved": round(achieved, 3), "peak": peak, "unit": unit,
                "frac": round(achieved / peak, 4), "traffic": hbm_traffic(k, w.name), "kernel": k,
                "algorithmic": f"{amount:.6g} {'TFLOP' if unit == 'TFLOP/s' else 'GB'} per launch",
                "kernel_us": round(kernels[k], 2), "gpu_share_us": round(gpu_time[k], 2)}
    roofline = roof(dom)
    roofline["dominant_by"] = "kernel time x share of compute units (256 CUs)"

    elapsed = t1 - t0
    single = {"images_per_s": round(K * s.B / elapsed, 2), "ms_per_step": round(1e3 * elapsed / K, 4)}

    # Roofline fraction of each stage against the unit that bounds its main
    # kernel: the project stage against the matrix cores (both products), the
    # select stage against the matrix cores for its Gram products plus the
    # vector ALU for the recurrence (time-weighted peak), compaction against HBM.
    def frac(amount, peak, us):
        return round(amount / (us * 1e-6) / peak, 4)
    sel_amount = work["select_recurrence"][1]
    # The selector against a roofline that assumes a per-step scan of the
    # unselected keys from LDS plus one HBM read of the keys and the history
    # rows (the traffic model that the Gram rewrite used here replaces): the time
    # the scan's bytes would take at the LDS and HBM peaks, over the measured
    # select stage.
    eb_keys = eb
    lds_scan = sum(sum((max(n - w.g * (t - 1), 0) + 2) * w.h * eb_keys for t in range(1, st + 1))
                   for n, st in zip(sizes, steps_g))
    hbm_keys = sum(n * w.h * eb_keys + (k + 1) * 2 * w.h * eb_keys
                   for n, k in zip(sizes, kept_g))
    t_scan_roof = max(lds_scan / (PEAK_LDS_GBS * 1e9), hbm_keys / (PEAK_HBM_GBS * 1e9))
    stage_roofline = {
        "project": {"bound": "mfma", "frac": frac(proj_flop + text_flop, mfma_peak, stages["project"]),
                    "frac_gemm_kernel": frac(proj_flop + text_flop, mfma_peak,
                                             kernels["project_gemm"])},
        "select": {"bound": "mfma+alu",
                   "frac_gram": frac(gram_flop, mfma_peak, kernels["gram_gemm"]),
                   "frac_recurrence": frac(sel_amount, PEAK_F32_VALU_TFLOPS,
                                           kernels["select_recurrence"]),
                   "recurrence_us_per_step_longest_episode":
                       round(kernels["select_recurrence"] / max(1, max(steps_g)), 3),
                   "frac_keyscan_roofline": round(t_scan_roof / (stages["select"] * 1e-6), 4),
                   "keyscan_roofline_us": round(t_scan_roof * 1e6, 2)},
        "compact": {"bound": "hbm", "frac": frac(work["compact_gather"][1], PEAK_HBM_GBS,
                                                 stages["compact"]),
                    "frac_kernel": frac(work["compact_gather"][1], PEAK_HBM_GBS,
                                        kernels["compact_gather"]),
                    "kernel_us": round(kernels["compact_gather"], 2),
                    "algorithmic": f"{work['compact_gather'][1]:.6g} GB per launch"},
    }

    # Pipelined pass: projections on one stream in batch order, batch k's
    # select + compact on the stream of slot k mod S (runner.Pipeline), so one
    # batch's projection and Gram products run on the compute units that
    # earlier batches' recurrences (one workgroup per episode) leave free.
    # --schedule rr instead issues whole batches round-robin on S streams.
    S = max(1, args.streams)
    slot_inputs = None
    if S > 1:
        from paper_2609_13804_amd.runner import Pipeline
        n_slots = max(S, args.slots) if args.schedule.startswith("staggered") else S
        if not args.shared_inputs:
            # a stream of fresh batches: every slot its own seeded tokens (same
            # sizes), so no batch's tokens are still in the caches from the last
            slot_inputs = [W.make_inputs(w, batch_index=k) for k in range(1, n_slots)]
        if args.schedule.startswith("staggered"):
            pipe = Pipeline(run, n_slots, min(S, Pipeline.max_streams()),
                            split_gram=args.schedule == "staggered-gram", inputs=slot_inputs)
            runs = pipe.runs
            issue = lambda k: pipe.issue()
        else:
            runs = [run] + [run.sibling(None if slot_inputs is None else slot_inputs[k])
                            for k in range(S - 1)]
            streams = [torch.cuda.Stream() for _ in range(S)]     # default priority
            def issue(k):
                r, st = runs[k % S], streams[k % S].cuda_stream
                r.project(st)
                r.select(st)
                if r.out is not None:
                    r.compact(st)
        # Each slot's own result, one stream at a time, for the check below.
        slot_inputs = None
        refs = []
        for r in runs:
            r.run()
            torch.cuda.synchronize()
            refs.append((r.kept_idx.clone(), None if r.out is None else r.out.clone()))
        # Untimed warm-up of the overlapped streams: at least W batches, every
        # slot used, and at least PIPE_WARMUP_BATCHES in all.  In a fresh process
        # the first few tens of milliseconds of overlapped work have run up to
        # 40 % slower than the rest, which a 50-batch timed region would include.
        for k in range(max(args.warmup, len(runs), PIPE_WARMUP_BATCHES)):
            issue(k)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(K):
            issue(k)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        errs = [e for r in runs for e in r.device_errors()]
        if any(errs):
            raise RuntimeError(f"device error words {errs}")
        for r, (kept_ref, out_ref) in zip(runs, refs):
            if not (torch.equal(r.kept_idx, kept_ref) and
                    (r.out is None or torch.equal(r.out, out_ref))):
                raise RuntimeError("the overlapped streams disagree with one stream on a batch")
        del refs
        elapsed = t1 - t0
    value = K * s.B / elapsed

    # Second denominators: what plain library work reaches on this GPU.
    peaks = measured_peaks()
    mpeak = {"mfma": peaks["bf16_matmul_TFLOPs"] if w.dtype == "bf16" else None,
             "hbm": peaks["hbm_copy_GBs"]}
    if mpeak["mfma"]:
        stage_roofline["project"]["frac_measured_peak"] = frac(
            proj_flop + text_flop, mpeak["mfma"], stages["project"])
        stage_roofline["select"]["frac_gram_measured_peak"] = frac(
            gram_flop, mpeak["mfma"], kernels["gram_gemm"])
    stage_roofline["compact"]["frac_measured_peak"] = frac(
        work["compact_gather"][1], mpeak["hbm"], stages["compact"])
    stage_roofline["compact"]["frac_kernel_measured_peak"] = frac(
        work["compact_gather"][1], mpeak["hbm"], kernels["compact_gather"])
    t_scan_meas = max(lds_scan / (peaks["lds_read_GBs"] * 1e9), hbm_keys / (PEAK_HBM_GBS * 1e9))
    stage_roofline["select"]["frac_keyscan_roofline_measured_lds"] = round(
        t_scan_meas / (stages["select"] * 1e-6), 4)
    if mpeak.get(roofline["bound"]):
        roofline["measured_peak"] = mpeak[roofline["bound"]]
        roofline["frac_measured_peak"] = round(roofline["achieved"] / mpeak[roofline["bound"]], 4)
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(1e3 * elapsed / K, 4),
        "us_per_image": round(1e6 * elapsed / (K * s.B), 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "images": s.B, "groups": s.G, "streams": S,
                   "schedule": args.schedule if S > 1 else "single",
                   "slot_inputs": ("shared" if args.shared_inputs else "own seeded batch per slot")
                                  if S > 1 else None,
                   "slots": max(S, args.slots) if S > 1 and args.schedule != "rr" else S,
                   "tokens": int(s.T_vis), "d": w.d, "h": w.h, "text_tokens": int(s.T_txt),
                   "layout": w.layout, "b_stop": b_stop, "tokens_per_round": w.g,
                   "kept_mean_per_image": round(float(kept_b.mean()), 3),
                   "selection_steps": int(sum(steps_g)),
                   "longest_episode_steps": int(max(steps_g))},
        "single_stream": single,
        "stages_us": {k: round(v, 2) for k, v in stages.items()},
        "stages_us_pct": {k: {q: round(x, 2) for q, x in v.items()} for k, v in stage_pct.items()},
        "stage_roofline": stage_roofline,
        "measured_peaks": peaks,
        "kernels_us": {k: round(v, 2) for k, v in kernels.items()},
        "selection_steps_per_s": round(sum(steps_g) / (stages["select"] * 1e-6), 1),
        "roofline": roofline,
        # the longest single kernel, a latency chain on one CU per episode
        "roofline_select_recurrence": dict(
            roof("select_recurrence"), bound="latency",
            us_per_step_longest_episode=round(kernels["select_recurrence"] / max(1, max(steps_g)), 3),
            note="one workgroup per episode; its time is the longest episode's chain of "
                 "dependent steps, so the FMA-rate fraction says little"),
    }
    # the plain selection's kept lists, before an optional pass reuses the run
    plain_kept = run.kept_lists()
    if args.trajectory is not None:
        out["trajectory"] = trajectory_pass(run, args.trajectory, K, hip)
    if args.encoder:
        if w.dtype != "bf16" or w.d % 128:
            raise SystemExit("--encoder needs a bfloat16 workload with d a multiple of 128")
        out["encoder"] = encoder_pass(w, K, hip, stream, mfma_peak)
        if peaks.get("bf16_matmul_TFLOPs"):
            out["encoder"]["frac_measured_peak"] = round(
                out["encoder"]["achieved_tflops"] / peaks["bf16_matmul_TFLOPs"], 4)
    if args.denoise:
        if w.dtype != "bf16":
            raise SystemExit("--denoise needs a bfloat16 workload")
        out["gate_denoise"] = gate_denoise_pass(w, K, hip, stream, mfma_peak)
        if peaks.get("bf16_matmul_TFLOPs"):
            out["gate_denoise"]["frac_measured_peak"] = round(
                out["gate_denoise"]["achieved_tflops"] / peaks["bf16_matmul_TFLOPs"], 4)
    steady = args.steady if args.steady >= 0 else (max(1, N_CU // s.G) if s.G < 128 else 0)
    if steady > 0:
        out["select_steady"] = steady_pass(w, steady, b_stop, hip, stream, t_scan_roof,
                                           plain_kept, max(steps_g))
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, lay, b_stop, args.cpu_budget, gpu_kept=plain_kept)
        one = cpu_baseline(w, lay, b_stop, args.cpu_budget * 0.5, single_thread=True)
        out["cpu_baseline"]["single_core"] = {"value": one["value"], "unit": one["unit"],
                                              "sample": one["sample"]}
        out["cpu_baseline"]["host"] = host_info()
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
