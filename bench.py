"""Benchmark: decoded frames/s of batched FSA-based one-symbol-per-frame beam search
on one MI355X, with the dominant kernel's roofline fraction and the CPU oracle's rate.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload standard]
                    [--schedule auto|frame|stream]

A step is one tbs_decode of the whole batch (every frame of every stream: joiner,
expansion, merge, pruning, history, traceback) on inputs already resident in HBM.
`value` is frames over the median duration of K plain steps (HIP events between
consecutive steps on the decode stream; the mean wall time is reported beside it).
Per-kernel durations come
from K further steps during which the library records HIP events around each launch
on the decode stream (tbs_model_set_profiling).  Algorithmic work (joiner FLOP,
search bytes) is counted from the survivor trace of one untimed decode.  The default
(standard) run also measures the graph, throughput, large and large-bf16 configurations
the same way and reports them under `other_workloads` (secondary figures; `value` is the
standard one).  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import statistics
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decoded frames/sec (B×T) at beam 4; joiner MFMA util %; prune HBM GB/s"
# MI355X published peaks: fp32 matrix and fp32 vector are both 157.3 TFLOP/s
PEAK = {"fp32_mfma_tflops": 157.3, "fp32_vector_tflops": 157.3, "bf16_mfma_tflops": 2500.0,
        "hbm_gbps": 8000.0}
DEFAULT_STEPS = {"tiny": 50, "standard": 20, "graph": 20, "throughput": 10, "large": 10}
KERNEL_SRC = os.path.join(ROOT, "paper_2211_00484_amd", "csrc", "kernels.hip")
TRAFFIC_TABLE = os.path.join(ROOT, "profiles", "traffic.md")
COPY_BYTES = 256 << 20
CPU_SAMPLE_STREAMS = {"tiny": None, "standard": None, "graph": None, "throughput": 24,
                      "large": 12}


def algorithmic_work(trace, lengths, graph, V, C, Vpad_tiles, Ns, frames=None):
    """Joiner rows (contexts) and search traffic implied by a survivor trace.

    General graphs: the search reads each arc record (dest, label, score) and gathers
    one logit per arc.  Trivial graph: arcs are implicit (every label); the joiner
    keeps each row's best Ns labels per 16-column sub-tile, and the search reads those
    lists (value + label) and the blank logit instead."""
    graphs = list(graph) if isinstance(graph, (list, tuple)) else None
    g0 = graphs[0] if graphs else graph
    trivial = not graphs and g0.num_states == 1 and g0.num_arcs == V - 1
    degs = [np.diff(g.row_ptr).astype(np.int64) for g in (graphs or [g0])]
    rows = 0
    cands = 0
    arcs = 0
    survivors_in = 0
    survivors_out = 0
    for b in range(trace.shape[1]):
        L = int(lengths[b])
        deg = degs[b] if graphs else degs[0]
        for f in (range(L) if frames is None else range(frames[0], min(frames[1], L))):
            cur = trace[f, b]
            n = int((cur[:, 0] >= 0).sum())
            rows += len(np.unique(cur[:n, 0]))
            a = int(deg[cur[:n, 1]].sum())
            arcs += a
            cands += n + a
            survivors_in += n
            survivors_out += int((trace[f + 1, b, :, 0] >= 0).sum())
    flop = 2.0 * rows * C * V
    # search kernel bytes: arc record (dest, label, score) + gathered logit per arc,
    # a logit per blank, survivor record in (ctx, state, row, score) + row_ptr pair,
    # per-row softmax partials, survivor record out + history (parent|label, arc).
    if trivial:
        arc_bytes = rows * (Vpad_tiles * 4 * Ns * 8 + 4)
    else:
        arc_bytes = arcs * (12 + 4) + (cands - arcs) * 4
    search_bytes = (arc_bytes + survivors_in * (16 + 8) + rows * Vpad_tiles * 8
                    + survivors_out * (16 + 8) + rows * 4)
    return dict(rows=rows, flop=flop, candidates=cands, arcs=arcs, search_bytes=search_bytes,
                survivors=survivors_in)


def kernel_source_hash() -> str:
    import hashlib
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter table
    (FETCH_SIZE and WRITE_SIZE per dispatch, scaled by the copy-kernel factor), or
    None if the table is absent, lacks the entry, or predates the current kernels."""
    if not os.path.exists(TRAFFIC_TABLE):
        return None
    src_hash, ffetch, fwrite, rows = None, None, None, {}
    for line in open(TRAFFIC_TABLE):
        line = line.strip()
        if line.startswith("kernels.hip sha256[:16]:"):
            src_hash = line.rsplit(":", 1)[1].strip().strip("`")
        elif line.startswith("copy factor FETCH_SIZE:"):
            ffetch = float(line.split(":", 1)[1].split()[0])
        elif line.startswith("copy factor WRITE_SIZE:"):
            fwrite = float(line.split(":", 1)[1].split()[0])
        elif line.startswith("|") and not line.startswith("|---") and "workload" not in line:
            cells = [c.strip().strip("`") for c in line.strip("|").split("|")]
            if len(cells) >= 4:
                rows[(cells[0], cells[1])] = (float(cells[2]), float(cells[3]))
    if (src_hash != kernel_source_hash() or ffetch is None or fwrite is None
            or (workload, kernel) not in rows):
        return None
    fetch_kib, write_kib = rows[(workload, kernel)]
    return {"bytes_per_launch": (fetch_kib / ffetch + write_kib / fwrite) * 1024.0,
            "fetch_kib_per_dispatch": fetch_kib, "write_kib_per_dispatch": write_kib,
            "copy_factor_fetch": ffetch, "copy_factor_write": fwrite,
            "source": "profiles/traffic.md"}


def copy_calibration(steps: int):
    """A plain device-to-device copy of COPY_BYTES, for scaling the traffic counters."""
    import torch
    src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    print(json.dumps({"copy_bytes": COPY_BYTES, "read_kib": COPY_BYTES / 1024,
                      "write_kib": COPY_BYTES / 1024, "gbps": 2 * COPY_BYTES / dt / 1e9}),
          flush=True)


def cpu_baseline(w, inputs, model_np, graph_np, dtype, threads=None, min_seconds=10.0,
                 max_passes=100):
    """The oracle (as it stands) on a bounded sample of the same workload: the sample's
    streams are decoded repeatedly until about min_seconds of wall time have passed."""
    import oracle
    sample = CPU_SAMPLE_STREAMS[w.name]
    streams = list(range(inputs.B)) if sample is None else list(range(0, inputs.B, inputs.B // sample))[:sample]
    threads = min(threads or os.cpu_count() or 1, len(streams))
    frames = int(inputs.lengths[streams].sum())
    passes = 0
    t0 = time.perf_counter()
    while True:
        oracle.decode(model_np, graph_np, inputs.encoder_out, inputs.lengths, w.beam,
                      w.max_states, w.max_contexts, bf16=(dtype == "bf16"), nthreads=threads,
                      want_trace=False, want_arcs=False, streams=streams)
        passes += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds or passes >= max_passes:
            break
    return {"value": passes * frames / dt, "unit": "frames/s", "cores": threads, "kind": "oracle",
            "sample": f"{len(streams)} of {inputs.B} streams ({frames} frames) x {passes} passes, "
                      f"fp64 C++ oracle, {threads} threads, {dt:.1f} s wall"}


SCALED = {"B": 8192, "T_short": 4, "T_long": 8}


def scaled_microbench(dtype: str, steps: int):
    """Labelled scaled microbenchmark (not a workload figure): the Large model and
    1M-state graph with B = 8,192 streams of fixed length, so that one frame's search
    (expansion over the CSR graph, max-merge, beam / max-states / max-contexts
    pruning) and joiner GEMM each fill the GPU.  Per-frame kernel times are the
    difference between decodes of T_long and T_short frames, divided by the frame
    difference (frames T_short..T_long-1, after the survivor sets have filled);
    algorithmic bytes and FLOP come from the survivor trace of those frames."""
    import torch
    from paper_2211_00484_amd import synth, tbs
    w = synth.WORKLOADS["large"]
    B, T1, T2 = SCALED["B"], SCALED["T_short"], SCALED["T_long"]
    rng = np.random.default_rng(0)
    inputs = synth.make_inputs(rng, B, T2, w.C)
    model_np = synth.make_model(rng, w.V, w.C, w.sigma)
    graph_np = synth.make_graph(w.graph, w.V)
    model = tbs.Model.from_synth(model_np, dtype=dtype)
    model.set_schedule("frame")
    graph = tbs.Graph.from_synth(graph_np)
    enc = torch.from_numpy(inputs.encoder_out).cuda()
    tr = tbs.decode(model, graph, enc, inputs.lengths, beam=w.beam, max_states=w.max_states,
                    max_contexts=w.max_contexts, want_trace=True)
    torch.cuda.synchronize()
    nvt = (w.V + 63) // 64
    work = algorithmic_work(tr.trace.cpu().numpy(), inputs.lengths, graph_np, w.V, w.C, nvt,
                            w.max_states, frames=(T1, T2))
    del tr
    res = {}
    for T in (T1, T2):
        lens = np.full(B, T, dtype=np.int32)
        out = tbs.allocate_outputs(B, T, w.max_states)
        e = enc[:, :T].contiguous()
        tbs.decode_into(model, graph, e, lens, w.beam, w.max_states, w.max_contexts, out)
        torch.cuda.synchronize()
        model.set_profiling(True)
        for _ in range(steps):
            tbs.decode_into(model, graph, e, lens, w.beam, w.max_states, w.max_contexts, out)
        prof = model.read_profile()
        model.set_profiling(False)
        res[T] = {k: v[1] / steps for k, v in prof.items()}  # ms per decode
        del out, e
    nf = T2 - T1
    s_us = 1e3 * (res[T2]["search"] - res[T1]["search"]) / nf
    j_us = 1e3 * (res[T2]["joiner"] - res[T1]["joiner"]) / nf
    s_bytes = work["search_bytes"] / nf
    j_flop = work["flop"] / nf
    peak_j = PEAK["bf16_mfma_tflops"] if dtype == "bf16" else PEAK["fp32_mfma_tflops"]
    line = {
        "microbenchmark": "scaled search + joiner, one frame at B = 8,192 (not a workload figure)",
        "config": {"model": "large (V=5,000, C=512)", "graph": "powerlaw1m", "B": B,
                   "frames_timed": f"{T1}..{T2 - 1}", "beam": w.beam, "max_states": w.max_states,
                   "max_contexts": w.max_contexts, "joiner": dtype, "steps": steps},
        "search": {"us_per_frame": s_us, "algorithmic_bytes_per_frame": s_bytes,
                   "gbps": s_bytes / (s_us * 1e-6) / 1e9, "peak_gbps": PEAK["hbm_gbps"],
                   "frac": s_bytes / (s_us * 1e-6) / 1e9 / PEAK["hbm_gbps"],
                   "arcs_per_frame": work["arcs"] / nf, "survivors_per_frame": work["survivors"] / nf},
        "joiner": {"us_per_frame": j_us, "algorithmic_flop_per_frame": j_flop,
                   "tflops": j_flop / (j_us * 1e-6) / 1e12, "peak_tflops": peak_j,
                   "frac": j_flop / (j_us * 1e-6) / 1e12 / peak_j,
                   "rows_per_frame": work["rows"] / nf},
    }
    print(json.dumps(line), flush=True)


def decode_roofline(prof, K, work, dtype):
    """Per-kernel timing (tbs_model_read_profile over K steps) -> (kernels, roofline,
    schedule, joiner TFLOP/s, search GB/s) for the dominant decode kernel."""
    peak_j = PEAK["bf16_mfma_tflops"] if dtype == "bf16" else PEAK["fp32_mfma_tflops"]
    kernels = {}
    for name, (n, ms) in prof.items():
        if n == 0:
            continue
        kernels[name] = {"launches_per_step": n / K, "avg_us": 1e3 * ms / max(n, 1),
                         "ms_per_step": ms / K}
    sk = "stream_group" if "stream_group" in kernels else "stream"
    if sk in kernels:
        # one persistent kernel runs joiner and search for every frame: its joiner FLOP
        # and search bytes are both divided by the whole kernel's duration
        schedule = sk
        st_avg_s = kernels[sk]["avg_us"] * 1e-6
        launches = max(kernels[sk]["launches_per_step"], 1)
        flop_per_launch = work["flop"] / launches
        bytes_per_launch = work["search_bytes"] / launches
        j_tflops = flop_per_launch / st_avg_s / 1e12
        s_gbps = bytes_per_launch / st_avg_s / 1e9
        kernels[sk].update({"algorithmic_flop_per_launch": flop_per_launch,
                                  "tflops": j_tflops, "peak_tflops": peak_j,
                                  "frac": j_tflops / peak_j,
                                  "algorithmic_search_bytes_per_launch": bytes_per_launch,
                                  "search_gbps": s_gbps})
        # the grouped kernel's joiner runs on 4x4x1 fp32 MFMA blocks and the single-
        # workgroup kernel's bf16 joiner on 4x4x4 bf16 blocks (bound "mfma"); the single-
        # workgroup fp32 joiner on VALU FMAs (bound "alu", against the fp32 vector peak)
        mfma = sk == "stream_group" or dtype == "bf16"
        roofline = {"kernel": "k_" + sk, "bound": "mfma" if mfma else "alu",
                    "achieved": j_tflops, "peak": peak_j, "unit": "TFLOP/s",
                    "frac": j_tflops / peak_j}
    else:
        schedule = "frame"
        j_avg_s = kernels["joiner"]["avg_us"] * 1e-6
        s_avg_s = kernels["search"]["avg_us"] * 1e-6
        j_launches = kernels["joiner"]["launches_per_step"]
        flop_per_launch = work["flop"] / max(j_launches, 1)
        bytes_per_launch = work["search_bytes"] / max(kernels["search"]["launches_per_step"], 1)
        j_tflops = flop_per_launch / j_avg_s / 1e12
        s_gbps = bytes_per_launch / s_avg_s / 1e9
        kernels["joiner"].update({"algorithmic_flop_per_launch": flop_per_launch,
                                  "tflops": j_tflops, "peak_tflops": peak_j,
                                  "frac": j_tflops / peak_j})
        kernels["search"].update({"algorithmic_bytes_per_launch": bytes_per_launch,
                                  "gbps": s_gbps, "peak_gbps": PEAK["hbm_gbps"],
                                  "frac": s_gbps / PEAK["hbm_gbps"]})
        if kernels["joiner"]["ms_per_step"] >= kernels["search"]["ms_per_step"]:
            roofline = {"kernel": "k_joiner", "bound": "mfma", "achieved": j_tflops,
                        "peak": peak_j, "unit": "TFLOP/s", "frac": j_tflops / peak_j}
        else:
            roofline = {"kernel": "k_search", "bound": "hbm", "achieved": s_gbps,
                        "peak": PEAK["hbm_gbps"], "unit": "GB/s",
                        "frac": s_gbps / PEAK["hbm_gbps"]}
    return kernels, roofline, schedule, j_tflops, s_gbps, peak_j


def measure_decode(w, inputs, model, graph, enc, dtype, K, W, work):
    """W untimed decodes, then K timed ones (the median of the per-step HIP-event
    intervals on the decode stream), then K more with per-kernel timing; the roofline
    of the dominant kernel."""
    import torch
    from paper_2211_00484_amd import tbs
    B, T = inputs.B, inputs.T
    frames = int(inputs.lengths.sum())
    out = tbs.allocate_outputs(B, T, w.max_states, status=True)
    for _ in range(W):
        tbs.decode_into(model, graph, enc, inputs.lengths, w.beam, w.max_states, w.max_contexts, out)
    torch.cuda.synchronize()

    # the timed steps: nothing but the decodes on the stream, with an event between
    # consecutive steps (a marker, no host synchronisation) for the per-step median
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record()
    for i in range(K):
        tbs.decode_into(model, graph, enc, inputs.lengths, w.beam, w.max_states, w.max_contexts, out)
        evs[i + 1].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    step_ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(K)]

    # the same steps again with HIP events around every kernel launch: per-kernel
    # durations for the roofline (the events add a little time between kernels)
    model.set_profiling(True)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for _ in range(K):
        tbs.decode_into(model, graph, enc, inputs.lengths, w.beam, w.max_states, w.max_contexts, out)
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    prof = model.read_profile()
    model.set_profiling(False)

    ms_step = statistics.median(step_ms)
    kernels, roofline, schedule, j_tflops, s_gbps, peak_j = decode_roofline(prof, K, work, dtype)
    tr = measured_traffic(w.name if dtype == w.dtype else f"{w.name}-{dtype}", roofline["kernel"])
    roofline["traffic"] = None if tr is None else tr["bytes_per_launch"]
    if tr is not None:
        roofline["traffic_detail"] = tr
    return {"value": frames / (ms_step * 1e-3), "ms_step": ms_step,
            "ms_step_mean_wall": (t1 - t0) * 1e3 / K, "ms_step_events": (t3 - t2) * 1e3 / K,
            "kernels": kernels, "roofline": roofline, "schedule": schedule,
            "j_tflops": j_tflops, "s_gbps": s_gbps, "peak_j": peak_j}


def other_workload(name, dtype=None):
    """A secondary configuration of the default run, measured as the main one (no CPU
    baseline): frames/s, per-frame latency, per-kernel times and the roofline."""
    import torch
    from paper_2211_00484_amd import synth, tbs
    w, inputs, model_np, graph_np = synth.make_workload(name, seed=0)
    dtype = dtype or w.dtype
    model = tbs.Model.from_synth(model_np, dtype=dtype)
    graph = tbs.Graph.from_synth(graph_np)
    enc = torch.from_numpy(inputs.encoder_out).cuda()
    tr_out = tbs.decode(model, graph, enc, inputs.lengths, beam=w.beam, max_states=w.max_states,
                        max_contexts=w.max_contexts, want_trace=True)
    torch.cuda.synchronize()
    work = algorithmic_work(tr_out.trace.cpu().numpy(), inputs.lengths, graph_np, w.V, w.C,
                            (w.V + 63) // 64, w.max_states)
    del tr_out
    K = DEFAULT_STEPS[w.name]
    m = measure_decode(w, inputs, model, graph, enc, dtype, K, 2, work)
    res = {"description": w.description, "joiner": dtype, "schedule": m["schedule"],
           "frames": int(inputs.lengths.sum()), "steps": K, "value": m["value"],
           "unit": "frames/s", "ms_per_step": m["ms_step"],
           "per_frame_latency_us": 1e3 * m["ms_step"] / max(int(inputs.lengths.max()), 1),
           "roofline": m["roofline"],
           "kernels": {k: round(v["avg_us"], 3) for k, v in m["kernels"].items()}}
    model.close()
    graph.close()
    return res


def chunked_bench(args, w, inputs, model_np, graph_np, model, graph, enc, dtype, K, W):
    """One step: a decode state for the batch, its frames in chunks of N (every stream
    advances by up to N frames per chunk), then finish."""
    import torch
    from paper_2211_00484_amd import tbs
    N = args.chunk
    B, T = inputs.B, inputs.T
    lens = inputs.lengths
    frames = int(lens.sum())
    chunks = []
    for c0 in range(0, T, N):
        piece = np.clip(lens - c0, 0, N).astype(np.int32)
        if piece.max() == 0:
            break
        chunks.append((enc[:, c0:c0 + int(piece.max())].contiguous(), piece))
    tr_out = tbs.decode(model, graph, enc, lens, beam=w.beam, max_states=w.max_states,
                        max_contexts=w.max_contexts, want_trace=True)
    torch.cuda.synchronize()
    work = algorithmic_work(tr_out.trace.cpu().numpy(), lens, graph_np, w.V, w.C,
                            (w.V + 63) // 64, w.max_states)
    del tr_out

    def step():
        st = tbs.DecodeState(model, graph, B, T, beam=w.beam, max_states=w.max_states,
                             max_contexts=w.max_contexts)
        for x, piece in chunks:
            st.chunk(x, piece)
        out = st.finish()
        st.close()
        return out

    for _ in range(W):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    model.set_profiling(True)
    for _ in range(K):
        step()
    torch.cuda.synchronize()
    prof = model.read_profile()
    model.set_profiling(False)
    kernels, roofline, schedule, j_tflops, s_gbps, peak_j = decode_roofline(prof, K, work, dtype)
    roofline["traffic"] = None  # counters are taken for the one-shot decode
    line = {
        "metric": METRIC + " (streaming: chunked decode)", "value": frames * K / (t1 - t0),
        "unit": "frames/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": (t1 - t0) * 1e3 / K, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32" if dtype == "fp32" else "bf16 joiner operands",
        "data": "synthetic",
        "config": {"workload": f"{w.name}+chunk{N}", "description": w.description, "B": B,
                   "T_max": T, "frames": frames, "chunk_frames": N, "chunks": len(chunks),
                   "per_stream_graphs": "2 alternating" if args.alt_graphs else None,
                   "schedule": schedule},
        "roofline": roofline,
        "kernels": kernels,
        "per_chunk_ms": (t1 - t0) * 1e3 / K / max(len(chunks), 1),
    }
    print(json.dumps(line), flush=True)


def transducer_bench(args):
    """One step: tbs_transducer_forward over a batch of random log-probabilities."""
    import torch
    from paper_2211_00484_amd import tbs
    B, T, U = (int(x) for x in args.tr_shape.split(","))
    kind = args.transducer
    rng = np.random.default_rng(0)
    blank_np = np.log(rng.uniform(0.01, 1.0, size=(B, T, U + 1))).astype(np.float32)
    label_np = np.log(rng.uniform(0.01, 1.0, size=(B, T, U))).astype(np.float32)
    lens = np.stack([np.full(B, T), np.full(B, min(U, T) if kind != "standard" else U)],
                    axis=1).astype(np.int32)
    blank, label = torch.from_numpy(blank_np).cuda(), torch.from_numpy(label_np).cuda()
    lens_d = torch.from_numpy(lens).cuda()
    K = args.steps or 50
    W = args.warmup
    for _ in range(W):
        tbs.transducer_forward(kind, blank, label, lens_d)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        tbs.transducer_forward(kind, blank, label, lens_d)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    # the kernel is the call's only launch: events on the launch stream bracket it
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(K)]
    for a, b in ev:
        a.record()
        tbs.transducer_forward(kind, blank, label, lens_d)
        b.record()
    torch.cuda.synchronize()
    avg_s = float(np.mean([a.elapsed_time(b) for a, b in ev])) * 1e-3
    cells = B * T * (U + 1)
    nbytes = 4 * B * T * (2 * U + 1)  # each log-probability read once
    gbps = nbytes / avg_s / 1e9
    line = {
        "metric": f"transducer forward recursion ({kind}, eq. {dict(standard=1, modified=2, constrained=3)[kind]}) grid cells/s",
        "value": cells * K / (t1 - t0), "unit": "cells/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": (t1 - t0) * 1e3 / K, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32 inputs, f64 scores", "data": "synthetic",
        "config": {"workload": f"transducer-{kind}", "B": B, "T": T, "U": U,
                   "inputs": "log U(0.01, 1) per cell"},
        "roofline": {"kernel": "k_transducer", "bound": "hbm", "achieved": gbps,
                     "peak": PEAK["hbm_gbps"], "unit": "GB/s", "frac": gbps / PEAK["hbm_gbps"],
                     "traffic": None},
        "kernel_avg_us": avg_s * 1e6,
    }
    if not args.no_cpu_baseline:
        import oracle
        n = 0
        t2 = time.perf_counter()
        while time.perf_counter() - t2 < 3.0:
            oracle.transducer_forward(kind, blank_np, label_np, lens[:, 0], lens[:, 1])
            n += 1
        dt = time.perf_counter() - t2
        line["cpu_baseline"] = {"value": cells * n / dt, "unit": "cells/s", "cores": 1,
                                "kind": "oracle", "sample": f"the whole batch, {n} passes"}
    print(json.dumps(line), flush=True)


def hyps_bench(args, w, inputs, model_np, model, graph, enc, dtype, K, W):
    """One step: tbs_hyp_search over the whole batch (beam_size hypotheses, max-symbols 1),
    with the FSA-based search of the same workload timed beside it."""
    import torch
    from paper_2211_00484_amd import tbs
    N, merge = args.beam_size, args.merge
    B, T = inputs.B, inputs.T
    frames = int(inputs.lengths.sum())
    run = lambda **kw: tbs.hyp_search(model, enc, inputs.lengths, beam_size=N, merge=merge, **kw)
    # algorithmic work from the hypotheses' back-pointers of one untimed run: the joiner
    # rows are the distinct contexts of each stream's hypotheses on each frame
    tr = run(want_trace=True).trace.cpu().numpy()
    V = w.V
    rows = 0
    for b in range(B):
        ctx = [0]
        for f in range(int(inputs.lengths[b])):
            rows += len(set(ctx))
            nxt = []
            for k in range(N):
                par, lab = tr[f + 1, b, k]
                if par < 0:
                    break
                c = ctx[par]
                nxt.append(c if lab == 0 else (c % V) * V + int(lab))
            ctx = nxt
    flop = 2.0 * w.C * V * rows
    for _ in range(W):
        run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        run()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    model.set_profiling(True)
    for _ in range(K):
        run()
    torch.cuda.synchronize()
    prof = model.read_profile()
    model.set_profiling(False)
    kernels = {n: {"launches_per_step": c / K, "avg_us": 1e3 * ms / max(c, 1),
                   "ms_per_step": ms / K} for n, (c, ms) in prof.items() if c}
    peak_j = PEAK["bf16_mfma_tflops"] if dtype == "bf16" else PEAK["fp32_mfma_tflops"]
    j = kernels["joiner"]
    j_tflops = flop / j["launches_per_step"] / (j["avg_us"] * 1e-6) / 1e12
    # the step kernel reads each joiner row's logits and statistics once per selection
    # round at most; algorithmic bytes: each row's logits and statistics once
    st_bytes = rows * (w.V * 4 + ((w.V + 63) // 64) * 8)
    sk = kernels["hyp_step"]
    st_gbps = st_bytes / sk["launches_per_step"] / (sk["avg_us"] * 1e-6) / 1e9
    if j["ms_per_step"] >= sk["ms_per_step"]:
        roofline = {"kernel": "k_joiner", "bound": "mfma", "achieved": j_tflops, "peak": peak_j,
                    "unit": "TFLOP/s", "frac": j_tflops / peak_j}
    else:
        roofline = {"kernel": "k_hyp_step", "bound": "hbm", "achieved": st_gbps,
                    "peak": PEAK["hbm_gbps"], "unit": "GB/s", "frac": st_gbps / PEAK["hbm_gbps"]}
    roofline["traffic"] = None
    # the FSA-based search on the same inputs (the paper's comparison, Table 5)
    out = tbs.allocate_outputs(B, T, w.max_states, status=True)
    for _ in range(W):
        tbs.decode_into(model, graph, enc, inputs.lengths, w.beam, w.max_states, w.max_contexts, out)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for _ in range(K):
        tbs.decode_into(model, graph, enc, inputs.lengths, w.beam, w.max_states, w.max_contexts, out)
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    value = frames * K / (t1 - t0)
    fsa = frames * K / (t3 - t2)
    line = {
        "metric": METRIC + " (full-sequence beam search, the comparison search of Table 5)",
        "value": value, "unit": "frames/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": (t1 - t0) * 1e3 / K, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32" if dtype == "fp32" else "bf16 joiner operands",
        "data": "synthetic",
        "config": {"workload": f"{w.name}+hyps{N}-{merge}", "description": w.description,
                   "B": B, "T_max": T, "frames": frames, "beam_size": N, "merge": merge,
                   "joiner": dtype},
        "roofline": roofline,
        "kernels": kernels,
        "joiner_rows_per_step": rows,
        "fsa_search_frames_per_s": fsa,
        "fsa_speedup_over_hyps": fsa / value,
    }
    if not args.no_cpu_baseline:
        import oracle
        t4 = time.perf_counter()
        sample = list(range(min(B, 8)))
        oracle.hyp_search(model_np, inputs.encoder_out, inputs.lengths, N, merge == "logadd",
                          bf16=(dtype == "bf16"), nthreads=args.cpu_threads or os.cpu_count(),
                          streams=sample)
        dt = time.perf_counter() - t4
        nf = int(inputs.lengths[sample].sum())
        line["cpu_baseline"] = {"value": nf / dt, "unit": "frames/s",
                                "cores": min(len(sample), args.cpu_threads or os.cpu_count()),
                                "kind": "oracle",
                                "sample": f"{len(sample)} of {B} streams ({nf} frames)"}
    print(json.dumps(line), flush=True)


def logadd_cpu_baseline(w, inputs, model_np, graph_np, dtype, n, threads=None,
                        min_seconds=10.0, max_seconds=30.0):
    """The oracle's lattice + n-best search on whole streams, timed on the host."""
    import oracle
    threads = threads or os.cpu_count() or 1
    rng = np.random.default_rng(1)
    t0 = time.perf_counter()
    frames = 0
    done = 0
    order = list(range(inputs.B))
    while time.perf_counter() - t0 < min_seconds and done < inputs.B:
        streams = order[done:done + threads]
        lat = oracle.lattice(model_np, graph_np, inputs.encoder_out, inputs.lengths, w.beam,
                             w.max_states, w.max_contexts, bf16=(dtype == "bf16"),
                             nthreads=threads, streams=streams)
        for k, b in enumerate(streams):
            L = int(inputs.lengths[b])
            lat.nbest(k, rng.uniform(size=(n, L + 1)))
            frames += L
        done += len(streams)
        if time.perf_counter() - t0 > max_seconds:
            break
    dt = time.perf_counter() - t0
    return {"value": frames / dt, "unit": "frames/s", "cores": threads, "kind": "oracle",
            "sample": f"{done} of {inputs.B} streams ({frames} frames): lattice search on "
                      f"{threads} threads, then the n-best search ({n} paths) per stream on "
                      "one thread"}


def logadd_bench(args, w, inputs, model_np, graph_np, model, graph, enc, dtype, K, W, work):
    """One step: tbs_lattice_create (the search, then the lattice) + tbs_lattice_nbest with
    N paths + destroy, on the whole batch."""
    import torch
    from paper_2211_00484_amd import tbs
    n = args.logadd
    B, T = inputs.B, inputs.T
    frames = int(inputs.lengths.sum())
    u = torch.from_numpy(np.random.default_rng(1).uniform(size=(B, n, T + 1))).cuda()

    def step(times=None):
        t0 = time.perf_counter()
        lat = tbs.Lattice(model, graph, enc, inputs.lengths, beam=w.beam,
                          max_states=w.max_states, max_contexts=w.max_contexts)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        out = lat.nbest(n, u)
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        arcs = lat.num_arcs()
        lat.close()
        if times is not None:
            times.append((t1 - t0, t2 - t1, arcs, float(out.num_unique.float().mean())))
        return out

    for _ in range(W):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    # the same steps again with the decode kernels timed by HIP events in their dispatch
    # packets: the search kernel remains the step's dominant kernel
    phases = []
    model.set_profiling(True)
    for _ in range(K):
        step(phases)
    prof = model.read_profile()
    model.set_profiling(False)
    kernels, roofline, schedule, j_tflops, s_gbps, peak_j = decode_roofline(prof, K, work, dtype)
    tr = measured_traffic(w.name if dtype == w.dtype else f"{w.name}-{dtype}", roofline["kernel"])
    roofline["traffic"] = None if tr is None else tr["bytes_per_launch"]
    ms_step = (t1 - t0) * 1e3 / K
    line = {
        "metric": METRIC + " (LogAdd: lattice + n-best label-sequence search)",
        "value": frames * K / (t1 - t0), "unit": "frames/s", "n_gpus": 1, "steps": K,
        "warmup": W, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 search and arc weights, f64 lattice scores" if dtype == "fp32"
                 else "bf16 joiner operands, f32 search and arc weights, f64 lattice scores",
        "data": "synthetic",
        "config": {"workload": f"{w.name}+logadd{n}", "description": w.description, "B": B,
                   "T_max": T, "frames": frames, "num_paths": n, "joiner": dtype,
                   "beam": "inf" if math.isinf(w.beam) else w.beam,
                   "max_states": w.max_states, "max_contexts": w.max_contexts},
        "roofline": roofline,
        "kernels": kernels,
        "phases_ms": {"search_and_lattice": 1e3 * float(np.mean([p[0] for p in phases])),
                      "nbest": 1e3 * float(np.mean([p[1] for p in phases]))},
        "lattice_arcs": phases[0][2],
        "distinct_sequences_per_stream": float(np.mean([p[3] for p in phases])),
        "work_per_step": work,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = logadd_cpu_baseline(w, inputs, model_np, graph_np, dtype, n,
                                                   threads=args.cpu_threads)
    print(json.dumps(line), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="standard",
                    choices=["tiny", "standard", "graph", "throughput", "large"])
    ap.add_argument("--schedule", default="auto", choices=["auto", "frame", "stream", "stream1"],
                    help="frame loop: per-frame joiner + search kernels, or one persistent "
                         "workgroup per stream (auto picks per shape)")
    ap.add_argument("--joiner-dtype", choices=["fp32", "bf16"], default=None,
                    help="override the workload's joiner dtype (e.g. Large in bf16)")
    ap.add_argument("--logadd", type=int, default=0, metavar="N",
                    help="time the LogAdd path instead: lattice of the search plus the n-best "
                         "label-sequence search with N sampled paths per stream")
    ap.add_argument("--search", choices=["fsa", "hyps"], default="fsa",
                    help="fsa: the FSA-based search (default); hyps: the full-sequence beam "
                         "search of Table 5 (trivial graph only), timed beside the FSA search")
    ap.add_argument("--beam-size", type=int, default=4, help="hypotheses for --search hyps")
    ap.add_argument("--merge", choices=["max", "logadd"], default="logadd",
                    help="merge of equal sequences for --search hyps")
    ap.add_argument("--transducer", choices=["standard", "modified", "constrained"],
                    default=None,
                    help="time the transducer forward recursion (eq. 1, 2 or 3) instead, on "
                         "random log-probabilities of B utterances of T frames and U labels")
    ap.add_argument("--tr-shape", default="32,250,80", metavar="B,T,U",
                    help="shape for --transducer (default: a training batch of 10 s "
                         "utterances at 25 frames/s with 80 labels)")
    ap.add_argument("--chunk", type=int, default=0, metavar="N",
                    help="streaming decode: every step decodes the batch in chunks of N "
                         "frames (tbs_state_create / tbs_decode_chunk / tbs_state_finish)")
    ap.add_argument("--alt-graphs", action="store_true",
                    help="one graph per stream: the workload's graph and a second graph of "
                         "the same kind (seed 2) alternate over the batch (tbs_decode_graphs)")
    ap.add_argument("--no-graph-capture", action="store_true",
                    help="frame schedule: launch every frame's kernels from the host instead "
                         "of replaying the captured frame loop")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--other-workloads", action=argparse.BooleanOptionalAction, default=True,
                    help="with the default (standard) workload, also measure the graph, "
                         "throughput, large and large-bf16 configurations the same way and "
                         "report them as secondary figures in the same line")
    ap.add_argument("--cpu-threads", type=int, default=None,
                    help="threads for the oracle baseline (default: all host threads)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain copy of 256 MiB (traffic-counter calibration)")
    ap.add_argument("--scaled-microbench", action="store_true",
                    help="only run the labelled scaled search + joiner microbenchmark "
                         "(Large model and graph, B = 8,192)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU (got --gpus {args.gpus}): streams are "
              "independent, so more GPUs would each decode their own share of the batch; "
              "multi-GPU runs are not part of this build.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2211_00484_amd import synth, tbs

    torch.cuda.set_device(0)
    if args.copy_calibration:
        copy_calibration(args.steps or 5)
        return
    if args.scaled_microbench:
        scaled_microbench(args.joiner_dtype or "fp32", args.steps or 3)
        return
    if args.transducer:
        transducer_bench(args)
        return
    w, inputs, model_np, graph_np = synth.make_workload(args.workload, seed=0)
    K = args.steps if args.steps is not None else DEFAULT_STEPS[w.name]
    W = args.warmup
    dtype = args.joiner_dtype or w.dtype
    model = tbs.Model.from_synth(model_np, dtype=dtype)
    model.set_schedule(args.schedule)
    model.set_graph_capture(not args.no_graph_capture)
    graph = tbs.Graph.from_synth(graph_np)
    enc = torch.from_numpy(inputs.encoder_out).cuda()
    B, T = inputs.B, inputs.T
    frames = int(inputs.lengths.sum())
    if args.alt_graphs:
        if w.graph == "trivial":
            sys.exit("--alt-graphs needs a workload with a general graph (graph, large)")
        g2_np = synth.power_law_graph(1_000_000, 5_000_000, w.V, seed=2) \
            if w.graph == "powerlaw1m" else synth.uniform_random_graph(5000, 100_000, w.V, seed=2)
        g2 = tbs.Graph.from_synth(g2_np)
        graph = [graph if b % 2 == 0 else g2 for b in range(B)]
        graph_np = [graph_np if b % 2 == 0 else g2_np for b in range(B)]
    if args.chunk:
        chunked_bench(args, w, inputs, model_np, graph_np, model, graph, enc, dtype, K, W)
        return

    # untimed decode with the survivor trace: algorithmic work of one step
    tr_out = tbs.decode(model, graph, enc, inputs.lengths, beam=w.beam, max_states=w.max_states,
                        max_contexts=w.max_contexts, want_trace=True)
    torch.cuda.synchronize()
    nvt = (w.V + 63) // 64
    work = algorithmic_work(tr_out.trace.cpu().numpy(), inputs.lengths, graph_np, w.V, w.C, nvt,
                            w.max_states)
    g_desc = graph_np[0] if isinstance(graph_np, list) else graph_np
    del tr_out

    if args.search == "hyps":
        hyps_bench(args, w, inputs, model_np, model, graph, enc, dtype, K, W)
        return
    if args.logadd:
        logadd_bench(args, w, inputs, model_np, graph_np, model, graph, enc, dtype, K, W, work)
        return

    m = measure_decode(w, inputs, model, graph, enc, dtype, K, W, work)
    value, ms_step, kernels, roofline, schedule = (m["value"], m["ms_step"], m["kernels"],
                                                   m["roofline"], m["schedule"])
    j_tflops, s_gbps, peak_j = m["j_tflops"], m["s_gbps"], m["peak_j"]
    ms_step_mean_wall, ms_step_events = m["ms_step_mean_wall"], m["ms_step_events"]

    line = {
        "metric": METRIC, "value": value, "unit": "frames/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32" if dtype == "fp32" else "bf16 joiner operands, f32 accumulate/scores",
        "data": "synthetic",
        "config": {"workload": w.name, "description": w.description, "B": B, "T_max": T,
                   "frames": frames, "C": w.C, "V": w.V, "graph": w.graph,
                   "graph_states": g_desc.num_states, "graph_arcs": g_desc.num_arcs,
                   "per_stream_graphs": "2 alternating" if args.alt_graphs else None,
                   "beam": "inf" if math.isinf(w.beam) else w.beam,
                   "max_states": w.max_states, "max_contexts": w.max_contexts,
                   "joiner": dtype, "schedule": schedule,
                   "frame_loop_graph": dict(zip(("captures", "replays"), model.graph_stats()))},
        "roofline": roofline,
        "kernels": kernels,
        "joiner_mfma_util_pct": 100.0 * j_tflops / peak_j,
        "search_hbm_gbps": s_gbps,
        "ms_per_step_mean_wall": ms_step_mean_wall,
        "ms_per_step_with_kernel_timing_events": ms_step_events,
        "per_frame_latency_us": 1e3 * ms_step / max(int(inputs.lengths.max()), 1),
        "work_per_step": work,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, inputs, model_np, graph_np, dtype,
                                            threads=args.cpu_threads)
    if (args.other_workloads and w.name == "standard" and dtype == w.dtype
            and args.schedule == "auto" and not args.alt_graphs):
        # the other configurations, measured the same way (secondary figures)
        line["other_workloads"] = {}
        for name, odt in (("graph", None), ("throughput", None), ("large", None),
                          ("large", "bf16")):
            key = name if odt is None else f"{name}-{odt}"
            line["other_workloads"][key] = other_workload(name, odt)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    try:
        main()
    finally:
        # release the library's handles while the HIP runtime is fully up
        if "paper_2211_00484_amd.tbs" in sys.modules:
            sys.modules["paper_2211_00484_amd.tbs"].close_all()
