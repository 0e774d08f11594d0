"""Benchmark of the Forgetting Attention hot path on one MI355X.

One step = the whole training-side path over one batch of the long-context
workload (B=2, H=16, L=16384, d=128, bf16): gate prefix -> forward (O, LSE) ->
backward (dQ, dK, dV, d(log f)).  Throughput counts the causal FLOPs of the
algorithm: 4d per causal (i, j) pair in the forward (QK^T and PV) and 10d in the
backward (QK^T recompute, dV, dP, dQ, dK), i.e. 14d per pair, the convention of
the paper's FLOP table (attention costs 2 n_layer d_model L per token and
direction of each product).  The decode step (B=64, H=16, T=32768, d=128) is
measured in the same run and reported in HBM GB/s.

Prints ONE JSON line.  Inputs are seeded synthetic tensors already resident in
HBM when the timed region starts.
"""
from __future__ import annotations

import argparse
import contextlib
import csv
import glob
import hashlib
import json
import os
import re
import sys
import time

import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import paper_2503_02130_amd as fox  # noqa: E402
from paper_2503_02130_amd import inputs  # noqa: E402

MFMA_BF16_PEAK_TFLOPS = 2516.6   # MI355X dense bf16 (256 CU x 2.4 GHz x 4096 FLOP/clk)
HBM_PEAK_GBS = 8000.0            # MI355X HBM3E

CSRC = os.path.join(ROOT, "paper_2503_02130_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")
TRAFFIC_FILE = os.path.join(PROFILES, "hbm_traffic_bench_workloads.txt")
# kernel -> the sources its machine code is built from (the traffic measured for
# a kernel is reported only while these are unchanged)
KERNEL_SOURCES = {
    "bwd_dkdv_bf16_kernel": ("attn_bwd.hip", "fox_device.h"),
    "bwd_dq_bf16_kernel": ("attn_bwd.hip", "fox_device.h"),
    "bwd_dq_stored_kernel": ("attn_bwd.hip", "fox_device.h"),
    "fwd_bf16_kernel": ("attn_fwd.hip", "fox_device.h"),
    "decode_split_kernel": ("attn_decode.hip", "fox_device.h"),
    "pro_prologue_kernel": ("pro_fusions.hip", "fox_device.h"),
    "pro_prologue_bwd_kernel": ("pro_fusions.hip", "fox_device.h"),
    "out_gate_kernel": ("pro_fusions.hip", "fox_device.h"),
    "out_gate_bwd_kernel": ("pro_fusions.hip", "fox_device.h"),
    "gate_proj_fwd_kernel": ("gate_proj.hip", "fox_device.h"),
    "gate_proj_bwd_kernel": ("gate_proj.hip", "fox_device.h"),
    "gate_proj_reduce_kernel": ("gate_proj.hip", "fox_device.h"),
}


def sources_hash(kernel: str) -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def causal_pairs(B: int, H: int, L: int) -> int:
    return B * H * L * (L + 1) // 2


def fwd_flops(B, H, L, d) -> float:
    return 4.0 * d * causal_pairs(B, H, L)


def bwd_flops(B, H, L, d) -> float:
    return 10.0 * d * causal_pairs(B, H, L)


def fwd_grid_threads(B, H, L) -> int:
    """Threads the bf16 forward launches: one 256-thread workgroup per 128 queries."""
    return B * H * ((L + 127) // 128) * 256


def decode_bytes(B, H, T, d, elem=2) -> float:
    return float(B * H * T * (2 * d * elem + 4))


def log(msg):
    print(msg, file=sys.stderr, flush=True)


class EventTimer:
    """Accumulates the duration of bracketed regions with HIP events on the
    current stream (the stream every library call is enqueued on)."""

    def __init__(self):
        self.pairs = []

    def __enter__(self):
        self.a = torch.cuda.Event(enable_timing=True)
        self.b = torch.cuda.Event(enable_timing=True)
        self.a.record()
        return self

    def __exit__(self, *exc):
        self.b.record()
        self.pairs.append((self.a, self.b))

    def maybe(self, on):
        return self if on else contextlib.nullcontext()

    def mean_ms(self):
        return sum(a.elapsed_time(b) for a, b in self.pairs) / max(1, len(self.pairs))

    def times_ms(self):
        return sorted(a.elapsed_time(b) for a, b in self.pairs)


def bench_train(w, steps, warmup):
    """One step = gate prefix -> forward -> backward keeping dS (the stages of
    fox_attn_bwd_stored, the last one also producing the gate-logit gradient), so
    that the dominant kernel, dK/dV with the dS store, can be bracketed by events
    on the call stream.  After it, the same step with the recompute backward (the
    stages of fox_attn_bwd, O(L) workspace) and with exact skipping."""
    dev = torch.device("cuda:0")
    x = inputs.workload_inputs(w, device=dev)
    s = fox.default_scale(w.d)
    B, H, L, d = w.B, w.H, w.L, w.d
    c = torch.empty((B, H, L), device=dev)
    o = torch.empty_like(x["q"])
    lse = torch.empty((B, H, L), device=dev)
    dq, dk, dv = torch.empty_like(x["q"]), torch.empty_like(x["k"]), torch.empty_like(x["v"])
    dlf, dlogit, delta, dcq, dck = (torch.empty((B, H, L), device=dev) for _ in range(5))
    store_bytes = fox.fox_attn_bwd_ds_store_bytes(x["q"].dtype, B, H, L, d)
    store = torch.empty(store_bytes, device=dev, dtype=torch.uint8)
    t_gate, t_fwd, t_dkdv, t_dq, t_bwd = (EventTimer() for _ in range(5))

    def step(timed):
        with t_gate.maybe(timed):
            fox.fox_gate_prefix(x["logit"], c=c)
        with t_fwd.maybe(timed):
            fox.fox_attn_fwd(x["q"], x["k"], x["v"], c, s, o=o, lse=lse)
        with t_bwd.maybe(timed):
            fox.fox_attn_bwd_delta(o, x["do"], delta=delta)
            with t_dkdv.maybe(timed):
                fox.fox_attn_bwd_dkdv_store(x["q"], x["k"], x["v"], c, lse, x["do"], delta, store,
                                            s, dk=dk, dv=dv, dc_k=dck)
            with t_dq.maybe(timed):
                fox.fox_attn_bwd_dq_stored(x["k"], store, s, dq=dq, dc_q=dcq)
            fox.fox_dlogit_from_dc(dcq, dck, x["logit"], d_logit=dlogit, d_log_f=dlf)

    for _ in range(warmup):
        step(False)
    torch.cuda.synchronize()
    log(f"[bench] {w.name}: warmup done")
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    t_step = EventTimer()  # each step on its own as well, for the median and minimum
    start.record()
    for _ in range(steps):
        with t_step:
            step(True)
    end.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / steps
    per_step = t_step.times_ms()
    ms = start.elapsed_time(end) / steps
    if not (torch.isfinite(o.float()).all() and torch.isfinite(dlf).all()):
        raise RuntimeError("non-finite outputs")
    stored = [t.clone() for t in (dq, dk, dv, dlf)]

    # The recompute backward: dK/dV bit for bit the same, dQ and d(log f) equal to
    # rounding (the two dQ passes sum the same bf16 dS in different orders).
    r_dkdv, r_dq, r_step = EventTimer(), EventTimer(), EventTimer()

    def step_recompute(timed):
        with r_step.maybe(timed):
            fox.fox_gate_prefix(x["logit"], c=c)
            fox.fox_attn_fwd(x["q"], x["k"], x["v"], c, s, o=o, lse=lse)
            fox.fox_attn_bwd_delta(o, x["do"], delta=delta)
            with r_dkdv.maybe(timed):
                fox.fox_attn_bwd_dkdv(x["q"], x["k"], x["v"], c, lse, x["do"], delta, s, dk=dk,
                                      dv=dv, dc_k=dck)
            with r_dq.maybe(timed):
                fox.fox_attn_bwd_dq(x["q"], x["k"], x["v"], c, lse, x["do"], delta, s, dq=dq,
                                    dc_q=dcq)
            fox.fox_dlogit_from_dc(dcq, dck, x["logit"], d_logit=dlogit, d_log_f=dlf)

    for _ in range(warmup):
        step_recompute(False)
    for _ in range(steps):
        step_recompute(True)
    torch.cuda.synchronize()
    if not (torch.equal(stored[1], dk) and torch.equal(stored[2], dv)):
        raise RuntimeError("dK/dV of the stored-dS backward differ from the recompute path")
    for a, b, name in ((stored[0], dq, "dQ"), (stored[3], dlf, "d(log f)")):
        e = float(torch.linalg.vector_norm((a - b).float()) / torch.linalg.vector_norm(b.float()))
        if e > 5e-3:
            raise RuntimeError(f"{name} of the two backward paths differ: rel-L2 {e:.3e}")

    # The step with exact gate-aware skipping (row-norm bounds computed inside
    # the timed step; backward keeping dS); its outputs must equal the training
    # step's bit for bit.
    ref = [t.clone() for t in (o, lse)] + stored
    qn = torch.empty((B, H), device=dev)
    kn = torch.empty((B, H), device=dev)
    ws = torch.empty(fox.fox_attn_bwd_stored_workspace_bytes(x["q"].dtype, B, H, L, d),
                     device=dev, dtype=torch.uint8)

    def step_skip():
        fox.fox_gate_prefix(x["logit"], c=c)
        fox.fox_row_norm_max(x["q"], out=qn)
        fox.fox_row_norm_max(x["k"], out=kn)
        fox.fox_attn_fwd_skip(x["q"], x["k"], x["v"], c, qn, kn, s, o=o, lse=lse)
        fox.fox_attn_bwd_skip_stored(x["q"], x["k"], x["v"], c, o, lse, x["do"], qn, kn, s, dq=dq,
                                     dk=dk, dv=dv, d_log_f=dlf, workspace=ws)

    for _ in range(warmup):
        step_skip()
    torch.cuda.synchronize()
    t_skip = EventTimer()
    for _ in range(steps):
        with t_skip:
            step_skip()
    torch.cuda.synchronize()
    if not all(torch.equal(a, b) for a, b in zip(ref, (o, lse, dq, dk, dv, dlf))):
        raise RuntimeError("the skipping step differs from the dense step")
    return {"ms": ms, "wall_ms": wall_ms, "step_median_ms": per_step[len(per_step) // 2],
            "step_min_ms": per_step[0], "gate_ms": t_gate.mean_ms(), "fwd_ms": t_fwd.mean_ms(),
            "bwd_ms": t_bwd.mean_ms(), "dkdv_ms": t_dkdv.mean_ms(), "dq_ms": t_dq.mean_ms(),
            "rc_ms": r_step.mean_ms(), "rc_dkdv_ms": r_dkdv.mean_ms(), "rc_dq_ms": r_dq.mean_ms(),
            "skip_ms": t_skip.mean_ms(), "store_bytes": store_bytes}


def _capture(fn):
    """fn's launches captured in a HIP graph (after one warm-up run on a side
    stream, as graph capture requires)."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def _graph_ms(g, reps, warmup):
    """Mean time of one replay: `reps` back-to-back replays bracketed by HIP events
    on the current stream (the stream replays run on), after `warmup` replays."""
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps


def bench_train_graph(w, steps, warmup):
    """The training step of a short-sequence workload (about 0.5 ms per step, so
    launches from Python would show between the kernels): the step keeping dS
    and the step recomputing P, each captured once in a HIP graph and replayed
    back to back; each stage is also captured alone for its own time.  Replays
    must reproduce the eager step bit for bit."""
    dev = torch.device("cuda:0")
    x = inputs.workload_inputs(w, device=dev)
    s = fox.default_scale(w.d)
    B, H, L, d = w.B, w.H, w.L, w.d
    c = torch.empty((B, H, L), device=dev)
    o = torch.empty_like(x["q"])
    lse = torch.empty((B, H, L), device=dev)
    dq, dk, dv = torch.empty_like(x["q"]), torch.empty_like(x["k"]), torch.empty_like(x["v"])
    dlf, dlogit, delta, dcq, dck = (torch.empty((B, H, L), device=dev) for _ in range(5))
    store = torch.empty(fox.fox_attn_bwd_ds_store_bytes(x["q"].dtype, B, H, L, d), device=dev,
                        dtype=torch.uint8)
    stage = {
        "gate_prefix": lambda: fox.fox_gate_prefix(x["logit"], c=c),
        "fwd": lambda: fox.fox_attn_fwd(x["q"], x["k"], x["v"], c, s, o=o, lse=lse),
        "delta": lambda: fox.fox_attn_bwd_delta(o, x["do"], delta=delta),
        "dkdv_store": lambda: fox.fox_attn_bwd_dkdv_store(x["q"], x["k"], x["v"], c, lse,
                                                          x["do"], delta, store, s, dk=dk, dv=dv,
                                                          dc_k=dck),
        "dq_stored": lambda: fox.fox_attn_bwd_dq_stored(x["k"], store, s, dq=dq, dc_q=dcq),
        "dkdv": lambda: fox.fox_attn_bwd_dkdv(x["q"], x["k"], x["v"], c, lse, x["do"], delta, s,
                                              dk=dk, dv=dv, dc_k=dck),
        "dq": lambda: fox.fox_attn_bwd_dq(x["q"], x["k"], x["v"], c, lse, x["do"], delta, s,
                                          dq=dq, dc_q=dcq),
        "scan": lambda: fox.fox_dlogit_from_dc(dcq, dck, x["logit"], d_logit=dlogit,
                                               d_log_f=dlf),
    }
    kept = ("gate_prefix", "fwd", "delta", "dkdv_store", "dq_stored", "scan")
    recomputed = ("gate_prefix", "fwd", "delta", "dkdv", "dq", "scan")
    outs = (c, o, lse, dq, dk, dv, dlf, dlogit)
    res = {}
    for name, order in (("stored", kept), ("recompute", recomputed)):
        def step(order=order):
            for n in order:
                stage[n]()
        step()
        torch.cuda.synchronize()
        ref = [t.clone() for t in outs]
        g = _capture(step)
        res[name + "_ms"] = _graph_ms(g, steps, warmup)
        if not all(torch.equal(a, b) for a, b in zip(outs, ref)):
            raise RuntimeError(f"{w.name}: graph replay of the {name} step differs from eager")
        if not (torch.isfinite(o.float()).all() and torch.isfinite(dlf).all()):
            raise RuntimeError("non-finite outputs")
        del g
    # each stage alone: ten launches per graph, so that the host's cost of one graph
    # launch does not show in the short kernels' times
    per_graph = 10
    for n, fn in stage.items():
        def many(fn=fn):
            for _ in range(per_graph):
                fn()
        g = _capture(many)
        res[n] = _graph_ms(g, max(2, steps // 2), warmup) / per_graph
        del g
    res["store_bytes"] = store.numel()
    return res


def train_graph_summary(w, r):
    """JSON object of a graph-timed training leg.  Both backwards are timed; the
    leg's step is the faster of the two (named in "backward"; at this short
    length the dS store saves less than it costs), the other one is reported
    beside it, with per-stage times and the MFMA roofline of the step's dK/dV
    kernel."""
    B, H, L, d = w.B, w.H, w.L, w.d
    fl_f, fl_b = fwd_flops(B, H, L, d), bwd_flops(B, H, L, d)
    fl_kv = 8.0 * d * causal_pairs(B, H, L)
    tf = {k: (fl_f + fl_b) / (r[k + "_ms"] * 1e-3) / 1e12 for k in ("stored", "recompute")}
    kv = {"stored": fl_kv / (r["dkdv_store"] * 1e-3) / 1e12,
          "recompute": fl_kv / (r["dkdv"] * 1e-3) / 1e12}
    fw = fl_f / (r["fwd"] * 1e-3) / 1e12
    main = "stored" if r["stored_ms"] <= r["recompute_ms"] else "recompute"
    other = "recompute" if main == "stored" else "stored"
    what = {"stored": "keeping dS (fox_attn_bwd_stored stages, %.2f GB workspace)"
                      % (r["store_bytes"] / 1e9),
            "recompute": "recomputing S and dP in the dQ pass (fox_attn_bwd stages, O(L) "
                         "workspace)"}
    kernel = {"stored": (f"bwd_dkdv_bf16_kernel<{d},false,false,true>", "fox_attn_bwd_dkdv_store"),
              "recompute": (f"bwd_dkdv_bf16_kernel<{d},false,false,false>", "fox_attn_bwd_dkdv")}
    return {
        "what": "training step (gate prefix -> forward -> backward -> d(logit)) at the 125M-model "
                "head shape; each step captured in a HIP graph and replayed back to back; each "
                "stage also captured alone, ten launches per graph, for its own time",
        "config": {"B": B, "H": H, "L": L, "d": d, "seed": w.seed, "flops_per_step": fl_f + fl_b},
        "ms_per_step": round(r[main + "_ms"], 4), "TFLOP/s": round(tf[main], 2),
        "frac_of_peak": round(tf[main] / MFMA_BF16_PEAK_TFLOPS, 4),
        "backward": what[main] + "; the faster of the two backwards at this shape",
        other: {"backward": what[other], "ms_per_step": round(r[other + "_ms"], 4),
                "TFLOP/s": round(tf[other], 2),
                "frac_of_peak": round(tf[other] / MFMA_BF16_PEAK_TFLOPS, 4),
                "dkdv_TFLOP/s": round(kv[other], 2)},
        "breakdown_ms": {n: round(r[n], 5) for n in ("gate_prefix", "fwd", "delta", "dkdv_store",
                                                     "dq_stored", "dkdv", "dq", "scan")},
        "roofline": {"bound": "mfma", "kernel": "%s (%s)" % kernel[main],
                     "achieved": round(kv[main], 2),
                     "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(kv[main] / MFMA_BF16_PEAK_TFLOPS, 4),
                     "traffic": measured_traffic(kernel[main][0]),
                     "algorithmic_flops_per_launch": fl_kv},
        "roofline_fwd": {"bound": "mfma", "kernel": f"fwd_bf16_kernel<{d}> (fox_attn_fwd)",
                         "achieved": round(fw, 2), "peak": MFMA_BF16_PEAK_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(fw / MFMA_BF16_PEAK_TFLOPS, 4)},
    }


def bench_prefill(w, steps, warmup):
    """Forward-only workload (the length-extrapolation prefill): gate prefix ->
    forward, timed per step with events on the call stream."""
    dev = torch.device("cuda:0")
    x = inputs.workload_inputs(w, device=dev)
    s = fox.default_scale(w.d)
    c = torch.empty((w.B, w.H, w.L), device=dev)
    o = torch.empty_like(x["q"])
    lse = torch.empty((w.B, w.H, w.L), device=dev)
    t_step, t_fwd = EventTimer(), EventTimer()

    def step(timed):
        with t_step.maybe(timed):
            fox.fox_gate_prefix(x["logit"], c=c)
            with t_fwd.maybe(timed):
                fox.fox_attn_fwd(x["q"], x["k"], x["v"], c, s, o=o, lse=lse)

    for _ in range(warmup):
        step(False)
    torch.cuda.synchronize()
    for _ in range(steps):
        step(True)
    torch.cuda.synchronize()
    if not (torch.isfinite(o.float()).all() and torch.isfinite(lse).all()):
        raise RuntimeError("non-finite prefill outputs")
    return {"ms": t_step.mean_ms(), "fwd_ms": t_fwd.mean_ms()}


def bench_pro(w, steps, warmup):
    """The FoX (Pro) layer's hot path at the training workload's shape: prologue
    (QK-norm, KV-shift), attention with the output norm and gate fused into the
    forward's epilogue, its backward (norm/gate backward fused with Delta; the
    attention backward keeping dS, as in the training step), and the prologue's
    backward.  Each part is timed on its own."""
    dev = torch.device("cuda:0")
    B, H, L, d = w.B, w.H, w.L, w.d
    x = inputs.pro_inputs(B, H, L, d, w.dtype, w.gate, w.seed + 1, device=dev)
    s = fox.default_scale(d)
    q, k, v = (torch.empty_like(x["q_raw"]) for _ in range(3))
    c = fox.fox_gate_prefix(x["logit"])
    o, y = torch.empty_like(q), torch.empty_like(q)
    lse = torch.empty((B, H, L), device=dev)
    pws = torch.empty(fox.fox_pro_prologue_bwd_workspace_bytes(q.dtype, B, H, L, d), device=dev,
                      dtype=torch.uint8)
    bws = torch.empty(fox.fox_attn_bwd_pro_stored_workspace_bytes(q.dtype, B, H, L, d),
                      device=dev, dtype=torch.uint8)
    pargs = (x["q_raw"], x["k_raw"], x["v_raw"], x["k_shift"], x["v_shift"], x["wq"], x["wk"])
    timers = {n: EventTimer() for n in ("prologue", "fwd_pro", "bwd_pro", "prologue_bwd",
                                         "out_gate")}
    grads = {}

    def step(timed):
        with timers["prologue"].maybe(timed):
            fox.fox_pro_prologue(*pargs, q=q, k=k, v=v)
        with timers["fwd_pro"].maybe(timed):
            fox.fox_attn_fwd_pro(q, k, v, c, x["g"], x["wo"], s, o=o, lse=lse, y=y)
        with timers["bwd_pro"].maybe(timed):
            grads["attn"] = fox.fox_attn_bwd_pro_stored(q, k, v, c, o, lse, x["g"], x["wo"],
                                                        x["dy"], s, workspace=bws)
        dq, dk, dv = grads["attn"][:3]
        with timers["prologue_bwd"].maybe(timed):
            grads["pro"] = fox.fox_pro_prologue_bwd(*pargs, dq, dk, dv, workspace=pws)
        with timers["out_gate"].maybe(timed):  # the standalone epilogue, for its bandwidth
            fox.fox_pro_output_gate(o, x["g"], x["wo"], y=y)

    for _ in range(warmup):
        step(False)
    torch.cuda.synchronize()
    for _ in range(steps):
        step(True)
    torch.cuda.synchronize()
    if not all(torch.isfinite(t.float()).all() for t in grads["attn"] + grads["pro"]):
        raise RuntimeError("non-finite Pro gradients")
    return {n: t.mean_ms() for n, t in timers.items()}


def bench_fixed(w, steps, warmup, t_min=2.0):
    """Fixed per-head gates (ALiBi form) at the training workload's shape, with
    the appendix initialisation for (T_min, T_max) = (2, L): time constants
    log-spaced from 2 to L steps over the heads.  The fwd+bwd step (backward
    keeping dS, as in the training step) dense and with exact skipping (bound
    kernels included); outputs must agree bit for bit."""
    dev = torch.device("cuda:0")
    x = inputs.workload_inputs(w, device=dev)
    B, H, L, d = w.B, w.H, w.L, w.d
    s = fox.default_scale(d)
    b = fox.fox_fixed_gate_init(H, t_min, float(L)).to(dev)
    ws = torch.empty(fox.fox_attn_bwd_fixed_gate_stored_workspace_bytes(x["q"].dtype, B, H, L, d),
                     device=dev, dtype=torch.uint8)
    out = {}

    def dense():
        o, lse = fox.fox_attn_fwd_fixed_gate(x["q"], x["k"], x["v"], b, s)
        g = fox.fox_attn_bwd_fixed_gate_stored(x["q"], x["k"], x["v"], b, o, lse, x["do"], s,
                                               workspace=ws)
        out["dense"] = (o, lse) + tuple(g)

    def skip():
        qn, kn = fox.fox_row_norm_max(x["q"]), fox.fox_row_norm_max(x["k"])
        o, lse = fox.fox_attn_fwd_fixed_gate_skip(x["q"], x["k"], x["v"], b, qn, kn, s)
        g = fox.fox_attn_bwd_fixed_gate_skip_stored(x["q"], x["k"], x["v"], b, o, lse, x["do"],
                                                    qn, kn, s, workspace=ws)
        out["skip"] = (o, lse) + tuple(g)

    res = {}
    for name, fn in (("dense", dense), ("skip", skip)):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        t = EventTimer()
        for _ in range(steps):
            with t:
                fn()
        torch.cuda.synchronize()
        res[name] = t.mean_ms()
    if not all(torch.equal(a, c) for a, c in zip(out["dense"], out["skip"])):
        raise RuntimeError("the fixed-gate skipping step differs from the dense step")
    return res


PROJ_SEED = 11  # seed of the gate projection's synthetic inputs


def projection_bytes(B, L, H, M):
    """Algorithmic HBM bytes of the gate projection with bf16 x: the logits read
    x and w_f, write the logits; the backward reads x, w_f and d_logit and writes
    dx, dw_f and db_f (the per-chunk partials are not counted)."""
    fwd = B * L * M * 2 + H * M * 4 + H * 4 + B * H * L * 4
    bwd = 2 * B * L * M * 2 + B * H * L * 4 + 2 * H * M * 4 + H * 4
    return fwd, bwd


def bench_projection(w, steps, warmup):
    """The forget-gate projection at the workload's model width M = H d: logits
    from x [B, L, M] bf16, then dx, dw_f and db_f; each direction captured in a HIP
    graph (ten launches) and replayed, for the kernels' own time."""
    dev = torch.device("cuda:0")
    B, H, L, M = w.B, w.H, w.L, w.H * w.d
    p = inputs.projection_inputs(B, L, H, M, "bf16", PROJ_SEED, device=dev)
    logit = torch.empty((B, H, L), device=dev)
    ws = torch.empty(fox.fox_gate_projection_bwd_workspace_bytes(torch.bfloat16, B, L, H, M),
                     device=dev, dtype=torch.uint8)
    dx = torch.empty_like(p["x"])
    dw, db = torch.empty((H, M), device=dev), torch.empty((H,), device=dev)
    # each direction lasts some tens of microseconds, so that launches from Python
    # would show in an event bracket: ten launches per HIP graph, replayed
    per_graph = 10

    def fwd():
        for _ in range(per_graph):
            fox.fox_gate_projection(p["x"], p["w_f"], p["b_f"], logit)

    def bwd():
        for _ in range(per_graph):
            fox.fox_gate_projection_bwd(p["x"], p["w_f"], p["d_logit"], workspace=ws, dx=dx,
                                        dw=dw, db=db)

    reps = max(2, steps // 2)
    gf, gb = _capture(fwd), _capture(bwd)
    res = {"B": B, "L": L, "H": H, "M": M, "fwd_ms": _graph_ms(gf, reps, warmup) / per_graph,
           "bwd_ms": _graph_ms(gb, reps, warmup) / per_graph}
    if not (torch.isfinite(logit).all() and torch.isfinite(dw).all()):
        raise RuntimeError("non-finite gate projection outputs")
    return res


def bench_decode(w, steps, warmup, cpu=False):
    dev = torch.device("cuda:0")
    y = inputs.workload_inputs(w, device=dev)
    T = w.L
    cc = torch.empty((w.B, w.H, T), device=dev)
    cc[..., : T - 1] = fox.fox_gate_prefix(y["cached_logit"])
    o = torch.empty_like(y["q"])
    lse = torch.empty((w.B, w.H), device=dev)
    ws = torch.empty(fox.fox_attn_decode_workspace_bytes(y["q"].dtype, w.B, w.H, T, w.d),
                     device=dev, dtype=torch.uint8)
    for _ in range(warmup):
        fox.fox_attn_decode(y["q"], y["k_cache"], y["v_cache"], cc, y["logit_new"], o=o, lse=lse,
                            workspace=ws)
    torch.cuda.synchronize()
    t = EventTimer()
    for _ in range(steps):
        with t:
            fox.fox_attn_decode(y["q"], y["k_cache"], y["v_cache"], cc, y["logit_new"], o=o,
                                lse=lse, workspace=ws)
    torch.cuda.synchronize()
    # exact gate-aware skipping: the key-norm bound is cache state (kept as keys
    # are appended), computed once here outside the timed region
    kn = fox.fox_row_norm_max(y["k_cache"])
    o2, lse2 = torch.empty_like(o), torch.empty_like(lse)
    for _ in range(warmup):
        fox.fox_attn_decode_skip(y["q"], y["k_cache"], y["v_cache"], cc, y["logit_new"], kn,
                                 o=o2, lse=lse2, workspace=ws)
    torch.cuda.synchronize()
    t2 = EventTimer()
    for _ in range(steps):
        with t2:
            fox.fox_attn_decode_skip(y["q"], y["k_cache"], y["v_cache"], cc, y["logit_new"], kn,
                                     o=o2, lse=lse2, workspace=ws)
    torch.cuda.synchronize()
    if not (torch.equal(o, o2) and torch.equal(lse, lse2)):
        raise RuntimeError("skipping decode differs from the dense decode")
    res = {"ms": t.mean_ms(), "skip_ms": t2.mean_ms()}
    if cpu:
        log("[bench] timing the fp64 oracle decode on the host")
        res["decode_cpu_baseline"] = cpu_baseline_decode(w, y)
    return res


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            return next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")),
                        "unknown")
    except OSError:
        return "unknown"


def _oracle_threads():
    threads = len(os.sched_getaffinity(0))
    torch.set_num_threads(threads)
    return torch.get_num_threads()


def cpu_baseline(w, n_heads=4):
    """The fp64 oracle, untouched, on a bounded sample: forward + backward of
    n_heads (batch, head) slices of the workload (n_heads / (B*H) of the step)."""
    import oracle
    cores = _oracle_threads()
    x = inputs.attn_inputs(1, n_heads, w.L, w.d, w.dtype, w.gate, w.seed, device="cpu")
    s = fox.default_scale(w.d)
    t0 = time.perf_counter()
    oracle.forward(x["q"], x["k"], x["v"], x["logit"], s)
    oracle.backward(x["q"], x["k"], x["v"], x["logit"], x["do"], s)
    dt = time.perf_counter() - t0
    flops = fwd_flops(1, n_heads, w.L, w.d) + bwd_flops(1, n_heads, w.L, w.d)
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": cores,
            "cpu_model": _cpu_model(), "kind": "oracle", "seconds": round(dt, 2),
            "sample": f"fp64 forward+backward of {n_heads} of {w.B * w.H} (batch, head) slices "
                      f"at L={w.L}, d={w.d}: {dt:.1f} s; value = those slices' causal FLOPs / time"}


def cpu_baseline_full(w):
    """The fp64 oracle on the whole workload (inputs drawn on the host with the
    workload's shapes, seed and distributions): forward, and backward for the
    training workloads, over every (batch, head) slice."""
    import oracle
    cores = _oracle_threads()
    x = inputs.workload_inputs(w, device="cpu")
    s = fox.default_scale(w.d)
    t0 = time.perf_counter()
    oracle.forward(x["q"], x["k"], x["v"], x["logit"], s)
    if w.kind == "fwdbwd":
        oracle.backward(x["q"], x["k"], x["v"], x["logit"], x["do"], s)
    dt = time.perf_counter() - t0
    flops = fwd_flops(w.B, w.H, w.L, w.d) + (bwd_flops(w.B, w.H, w.L, w.d)
                                             if w.kind == "fwdbwd" else 0.0)
    what = "forward+backward" if w.kind == "fwdbwd" else "forward"
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "seconds": round(dt, 3),
            "sample": f"full: fp64 {what} of all {w.B * w.H} (batch, head) slices at L={w.L}, "
                      f"d={w.d}: {dt:.2f} s"}


def cpu_baseline_rows(w, n_rows=512):
    """The fp64 oracle forward on n_rows query rows of one head of each gate group
    (the oracle computes a row block against all keys, masked, so the whole
    problem in blocks of n_rows costs L / n_rows blocks per head): the time is
    extrapolated to every row of every head, and labelled so."""
    import oracle
    cores = _oracle_threads()
    x = inputs.workload_inputs(w, device="cpu")
    s = fox.default_scale(w.d)
    heads = (0, w.H - 1)
    r0 = w.L // 2
    rows = list(range(r0, r0 + n_rows))
    t0 = time.perf_counter()
    for h in heads:
        sl = {k: v[:1, h:h + 1] for k, v in x.items()}
        oracle.forward(sl["q"], sl["k"], sl["v"], sl["logit"], s, rows=rows)
    dt = time.perf_counter() - t0
    full = dt / len(heads) * (w.L / n_rows) * w.B * w.H
    return {"value": fwd_flops(w.B, w.H, w.L, w.d) / full / 1e12, "unit": "TFLOP/s",
            "cores": cores, "kind": "oracle", "seconds": round(full, 1),
            "sample": f"extrapolated: fp64 forward of {n_rows} query rows of heads {heads} "
                      f"(one per gate group) at L={w.L} took {dt:.2f} s; scaled by "
                      f"(L / {n_rows}) row blocks x {w.B * w.H} heads to {full:.0f} s for the "
                      "whole forward"}


def cpu_baseline_decode(w, y):
    """The fp64 oracle decode over every (batch, head) slice of the decode
    workload's cache `y` (on the GPU): each batch row is copied to the host
    outside the timed region, then the oracle's step is timed."""
    import oracle
    cores = _oracle_threads()
    s = fox.default_scale(w.d)
    dt = 0.0
    for b in range(w.B):
        sl = {k: v[b:b + 1].cpu() for k, v in y.items()}
        t0 = time.perf_counter()
        oracle.decode(sl["q"], sl["k_cache"], sl["v_cache"], sl["cached_logit"], sl["logit_new"],
                      s)
        dt += time.perf_counter() - t0
        del sl
    byt = decode_bytes(w.B, w.H, w.L, w.d)
    return {"value": byt / dt / 1e9, "unit": "GB/s", "cores": cores, "kind": "oracle",
            "seconds": round(dt, 2),
            "sample": f"full: fp64 decode of all {w.B * w.H} (batch, head) slices at T={w.L}, "
                      f"d={w.d}: {dt:.1f} s (host copies of the cache not timed); value = the "
                      "step's algorithmic cache bytes / time"}


def calibration_copy(mib: int):
    """A plain device copy of `mib` MiB (reads and writes mib MiB): the reference
    that scales the FETCH_SIZE / WRITE_SIZE counters to bytes."""
    n = mib * 2**20 // 4
    src = torch.rand(n, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    log(f"[bench] calibration copy of {mib} MiB done")


def _counter_rows(d):
    rows = []
    for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            rows += list(csv.DictReader(f))
    if not rows:
        raise SystemExit(f"no counter_collection.csv under {d}")
    return rows


def _kernel_family(name):
    """fox::<family><...> (demangled or Itanium-mangled), or "copy" for the
    runtime's device-to-device copy kernel; None for anything else."""
    m = re.search(r"fox::(\w+)[<(]", name)
    if m:
        return m.group(1)
    m = re.match(r"_ZN3fox(\d+)", name)
    if m:
        n = int(m.group(1))
        return name[m.end():m.end() + n]
    return "copy" if "copyBuffer" in name else None


def _kernel_key(name):
    """The kernel family with its template arguments, e.g.
    bwd_dkdv_bf16_kernel<128,false,false> (dense and skipping instantiations of
    one family differ in traffic), or "copy"; None for anything else."""
    fam = _kernel_family(name)
    if fam in (None, "copy"):
        return fam
    m = re.search(r"fox::\w+<([^>]*)>", name)
    if m:
        return f"{fam}<{m.group(1).replace(' ', '')}>"
    # Itanium-mangled: _ZN3fox<n><family>I<args>E...; the argument kinds used here
    m = re.match(r"_ZN3fox\d+\w+?I((?:DF16b|f|Li\d+E|Lb[01]E)+)E", name)
    if not m:
        return fam
    toks = re.findall(r"DF16b|f|Li\d+E|Lb[01]E", m.group(1))
    out = []
    for t in toks:
        if t == "DF16b":
            out.append("__bf16")
        elif t == "f":
            out.append("float")
        elif t.startswith("Li"):
            out.append(t[2:-1])
        else:
            out.append("true" if t[2] == "1" else "false")
    return f"{fam}<{','.join(out)}>"


def _per_kernel_kib(rows, counter):
    """Counter value (KiB) per dispatch, per (kernel, launch grid in threads); the
    copy kernels are keyed ("copy", 0)."""
    per = {}
    for r in rows:
        if r["Counter_Name"] != counter:
            continue
        key = _kernel_key(r["Kernel_Name"])
        if key is None:
            continue
        k = (key, 0 if key == "copy" else int(r["Grid_Size"]))
        per.setdefault(k, {}).setdefault(r["Dispatch_Id"], 0.0)
        per[k][r["Dispatch_Id"]] += float(r["Counter_Value"])
    return per


def pmc_summary(fetch_dir, write_dir, copy_mib, command):
    """Text summary of two rocprofv3 --pmc passes (FETCH_SIZE, WRITE_SIZE) of this
    benchmark run with --calibrate-copy-mib: per-launch HBM bytes of each kernel,
    scaled by what the counters read for the plain copy of known size."""
    fetch = _per_kernel_kib(_counter_rows(fetch_dir), "FETCH_SIZE")
    write = _per_kernel_kib(_counter_rows(write_dir), "WRITE_SIZE")
    # the calibration copy is by far the largest device-to-device copy of the run
    cf = max(fetch[("copy", 0)].values())
    cw = max(write[("copy", 0)].values())
    f_fac = copy_mib * 1024.0 / cf
    w_fac = copy_mib * 1024.0 / cw
    lines = ["# HBM traffic per launch from rocprofv3 FETCH_SIZE / WRITE_SIZE",
             f"# command (one pass per counter): {command}",
             f"# calibration: plain copy of {copy_mib} MiB read {cf:.0f} KiB and wrote {cw:.0f} KiB;",
             f"#   scale factors fetch {f_fac:.4f}, write {w_fac:.4f}",
             "# kernel  grid_threads  dispatches  fetch_KiB  write_KiB  traffic_bytes_per_launch  "
             "sources_sha256"]
    for k, grid in sorted(set(fetch) & set(write)):
        fam = k.split("<")[0]
        if fam not in KERNEL_SOURCES:
            continue
        f_, w_ = fetch[(k, grid)], write[(k, grid)]
        fk = sum(f_.values()) / len(f_)
        wk = sum(w_.values()) / len(w_)
        tb = (fk * f_fac + wk * w_fac) * 1024.0
        lines.append(f"{k} {grid} {len(f_)} {fk:.1f} {wk:.1f} {tb:.0f} {sources_hash(fam)}")
    return "\n".join(lines) + "\n"


SQ_PASS_A = ("SQ_INSTS_MFMA", "SQ_INSTS_VALU", "SQ_INSTS_LDS", "SQ_INSTS_SALU",
             "SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_WAVE_CYCLES", "SQ_INSTS_VALU_TRANS_F32")
SQ_PASS_B = ("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_VALU_MFMA_COEXEC_CYCLES", "SQ_BUSY_CYCLES",
             "SQ_LDS_BANK_CONFLICT", "SQ_WAIT_INST_ANY", "SQ_WAIT_ANY", "SQ_ACTIVE_INST_VALU",
             "SQ_ACTIVE_INST_LDS")
# kernels whose measured traffic the JSON line reports
KV_STORE_KERNEL = "bwd_dkdv_bf16_kernel<128,false,false,true>"
KV_KERNEL = "bwd_dkdv_bf16_kernel<128,false,false,false>"
DQ_STORED_KERNEL = "bwd_dq_stored_kernel<128,false>"
DECODE_KERNEL = "decode_split_kernel<__bf16,128,false,false>"
PROJ_FWD_KERNEL = "gate_proj_fwd_kernel<true,1>"
PROJ_BWD_KERNEL = "gate_proj_bwd_kernel<true,1>"
PROJ_REDUCE_KERNEL = "gate_proj_reduce_kernel"
ROOFLINE_KERNELS = (KV_STORE_KERNEL, KV_KERNEL, DQ_STORED_KERNEL, DECODE_KERNEL, PROJ_FWD_KERNEL,
                    PROJ_BWD_KERNEL, PROJ_REDUCE_KERNEL)

SQ_KERNELS = tuple(k for dd in (128, 64) for k in (
    f"fwd_bf16_kernel<{dd},false,false,false>", f"bwd_dkdv_bf16_kernel<{dd},false,false,false>",
    f"bwd_dkdv_bf16_kernel<{dd},false,false,true>", f"bwd_dq_bf16_kernel<{dd},false,false>",
    f"bwd_dq_stored_kernel<{dd},false>"))


def sq_summary(dirs, command, ms):
    """Text summary of rocprofv3 --pmc passes (SQ_PASS_A, SQ_PASS_B) over this
    benchmark: per dense attention kernel and launch grid (the workloads launch
    different grids), instruction mix, MFMA work and issue counters.  `ms` maps
    (kernel, grid) -> median duration (ms) from a kernel trace of the same
    command; MFMA utilisation = executed MFMA FLOPs / (duration x peak)."""
    per = {}
    for d in dirs:
        for r in _counter_rows(d):
            k = _kernel_key(r["Kernel_Name"])
            if k not in SQ_KERNELS:
                continue
            c = per.setdefault((k, int(r["Grid_Size"])), {}).setdefault(r["Counter_Name"], {})
            c[r["Dispatch_Id"]] = c.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
    lines = ["# SQ counters of the dense attention kernels (rocprofv3 --pmc, two passes)",
             f"# command (one pass per counter set): {command}",
             "#   pass A: " + " ".join(SQ_PASS_A), "#   pass B: " + " ".join(SQ_PASS_B),
             "# values: mean per dispatch; MOPS_BF16 counts 512-FLOP MFMA operations; one section",
             "# per kernel and launch grid (threads), i.e. per workload"]
    for k in SQ_KERNELS:
        for (kk, grid) in sorted(g for g in per if g[0] == k):
            v = {n: sum(x.values()) / len(x) for n, x in per[(kk, grid)].items()}
            lines.append(f"\n## {k}, grid {grid} threads")
            for n in SQ_PASS_A + SQ_PASS_B:
                if n in v:
                    lines.append(f"{n:32s} {v[n]:.6g}")
            mf = v.get("SQ_INSTS_MFMA", 0.0)
            if mf:
                lines.append(f"{'non-MFMA VALU per MFMA':32s} {(v['SQ_INSTS_VALU'] - mf) / mf:.3f}")
                lines.append(f"{'LDS instructions per MFMA':32s} {v['SQ_INSTS_LDS'] / mf:.3f}")
            if v.get("SQ_VALU_MFMA_BUSY_CYCLES"):
                lines.append(f"{'MFMA/VALU co-issue share':32s} "
                             f"{v['SQ_VALU_MFMA_COEXEC_CYCLES'] / v['SQ_VALU_MFMA_BUSY_CYCLES']:.3f}")
            if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in v and (k, grid) in ms:
                fl = v["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512.0
                t = ms[(k, grid)]
                lines.append(f"{'executed MFMA FLOPs':32s} {fl:.4g}")
                lines.append(f"{'trace duration ms (median)':32s} {t:.4f}")
                lines.append(f"{'MFMA utilisation of 2516.6 TF':32s} "
                             f"{fl / (t * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS:.4f}")
    return "\n".join(lines) + "\n"


def trace_summary(db, command):
    """Markdown summary of a rocprofv3 --kernel-trace results database of this
    benchmark: per library kernel and launch grid (each workload launches its own
    grid), calls, mean / min / max duration and LDS bytes."""
    import sqlite3
    con = sqlite3.connect(db)
    rows = con.execute("select name, grid_x, grid_y, grid_z, workgroup_x, workgroup_y, "
                       "workgroup_z, duration, lds_size from kernels")
    groups = {}
    for name, gx, gy, gz, wx, wy, wz, dur, lds in rows:
        key = _kernel_key(name)
        if key in (None, "copy"):
            continue
        # the grid is given in work-items per dimension
        wgs = (gx // max(wx, 1)) * (gy // max(wy, 1)) * (gz // max(wz, 1))
        g = groups.setdefault((key, wgs, wx * wy * wz), {"d": [], "lds": lds})
        g["d"].append(dur / 1e3)
    lines = ["# Kernel trace of bench.py: every library kernel, per launch grid",
             "", f"Command: `{command}`", "",
             "Durations in microseconds from the trace (one line per kernel and grid; the "
             "workloads differ in grid size).", "",
             "| kernel | workgroups | threads | calls | mean us | min us | max us | LDS bytes |",
             "|---|---:|---:|---:|---:|---:|---:|---:|"]
    for (key, wgs, wx), g in sorted(groups.items(), key=lambda kv: -sum(kv[1]["d"])):
        d = g["d"]
        lines.append(f"| {key} | {wgs} | {wx} | {len(d)} | {sum(d) / len(d):.1f} | {min(d):.1f} | "
                     f"{max(d):.1f} | {g['lds']} |")
    return "\n".join(lines) + "\n"


def measured_traffic(kernel: str, grid: int = None):
    """Bytes per launch recorded for `kernel` (family<template arguments>) at
    launch grid `grid` (threads; may be omitted when the kernel ran with one grid
    only), or None when there is no record, the grid is ambiguous, or the family's
    sources changed since the counters were taken."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    found = []
    for line in open(TRAFFIC_FILE):
        f = line.split()
        if line.startswith("#") or len(f) != 7 or f[0] != kernel:
            continue
        if grid is None or int(f[1]) == grid:
            found.append(f)
    if len(found) != 1:
        return None
    f = found[0]
    return float(f[5]) if f[6] == sources_hash(kernel.split("<")[0]) else None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="fwdbwd_bf16_b2_h16_l16384_d128")
    ap.add_argument("--decode-workload", default="decode_bf16_b64_h16_t32768_d128")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-pro", action="store_true", help="skip the FoX (Pro) layer timings")
    ap.add_argument("--no-fixed", action="store_true", help="skip the fixed-gate timings")
    ap.add_argument("--no-projection", action="store_true",
                    help="skip the forget-gate projection timings")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-workloads", action="store_true",
                    help="skip the d = 64 training shape and the 65536-length prefill legs")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="run a plain device copy of this size first (counter calibration)")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two rocprofv3 --pmc passes of this benchmark and exit")
    ap.add_argument("--pmc-command", default="", help="the profiled command, for the summary")
    ap.add_argument("--trace-summary", metavar="RESULTS_DB",
                    help="summarise a rocprofv3 --kernel-trace results.db of this benchmark and exit")
    ap.add_argument("--sq-summary", nargs="+", metavar="DIR",
                    help="summarise rocprofv3 --pmc SQ passes of this benchmark and exit; the "
                         "last argument is a kernel-trace results.db for the durations")
    args = ap.parse_args()
    if args.trace_summary:
        print(trace_summary(args.trace_summary, args.pmc_command), end="")
        return
    if args.sq_summary:
        import sqlite3
        *dirs, db = args.sq_summary
        con = sqlite3.connect(db)
        durs = {}
        for name, gx, dur in con.execute("select name, grid_x, duration from kernels"):
            k = _kernel_key(name)
            if k in SQ_KERNELS:
                durs.setdefault((k, int(gx)), []).append(float(dur) / 1e6)  # ns -> ms
        ms = {key: sorted(v)[len(v) // 2] for key, v in durs.items()}
        print(sq_summary(dirs, args.pmc_command, ms), end="")
        return
    if args.pmc_summary:
        print(pmc_summary(*args.pmc_summary, args.calibrate_copy_mib or 1024, args.pmc_command),
              end="")
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(Forgetting Attention shards over (batch, head) with no communication).",
              file=sys.stderr)
        sys.exit(2)
    if not os.path.exists(fox.LIB_PATH):
        from paper_2503_02130_amd import build
        build.build()
    fox.load()

    if args.calibrate_copy_mib:
        calibration_copy(args.calibrate_copy_mib)
    w = inputs.WORKLOADS[args.workload]
    r = bench_train(w, args.steps, args.warmup)
    B, H, L, d = w.B, w.H, w.L, w.d
    fl_f, fl_b = fwd_flops(B, H, L, d), bwd_flops(B, H, L, d)
    tflops = (fl_f + fl_b) / (r["ms"] * 1e-3) / 1e12
    fwd_tf = fl_f / (r["fwd_ms"] * 1e-3) / 1e12
    bwd_tf = fl_b / (r["bwd_ms"] * 1e-3) / 1e12
    # dK/dV kernel: its 4 GEMMs (S recomputed, dV, dP, dK) are 8d FLOPs per causal pair
    fl_kv = 8.0 * d * causal_pairs(B, H, L)
    kv_tf = fl_kv / (r["dkdv_ms"] * 1e-3) / 1e12
    # compulsory HBM bytes of one dK/dV launch: read q, k, v, dO (bf16), c, LSE,
    # delta (fp32); write dK, dV (bf16), dc_k (fp32) and the stored dS
    kv_bytes = B * H * L * (6 * d * 2 + 4 * 4) + r["store_bytes"]
    kv_traffic = measured_traffic(KV_STORE_KERNEL)
    # dQ from the stored dS: read dS and k, write dQ (bf16) and dc_q (fp32)
    dq_bytes = r["store_bytes"] + B * H * L * (2 * d * 2 + 4)
    dq_gbs = dq_bytes / (r["dq_ms"] * 1e-3) / 1e9
    rc_tf = (fl_f + fl_b) / (r["rc_ms"] * 1e-3) / 1e12
    out = {
        "metric": "Forgetting-attn fwd+bwd TFLOP/s bf16 L=16k d=128 (% MFMA peak); decode GB/s",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["ms"], 4),
        "step_ms_median": round(r["step_median_ms"], 4),
        "step_ms_min": round(r["step_min_ms"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": B, "H": H, "L": L, "d": d,
                   "gate_logits": "per-head mean U[0,6], std 1", "causal": True,
                   "flops_per_step": fl_f + fl_b, "parallelism": "none (1 GPU)",
                   "seed": w.seed},
        "frac_of_peak": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
        "backward": "fox_attn_bwd_stored stages: dK/dV also store bf16 dS (%.2f GB workspace), "
                    "the dQ pass reads it instead of recomputing S and dP" % (r["store_bytes"] / 1e9),
        "breakdown_ms": {"gate_prefix": round(r["gate_ms"], 4), "fwd": round(r["fwd_ms"], 4),
                         "bwd": round(r["bwd_ms"], 4), "bwd_dkdv_store": round(r["dkdv_ms"], 4),
                         "bwd_dq_stored": round(r["dq_ms"], 4),
                         "wall_per_step": round(r["wall_ms"], 4)},
        "roofline": {"bound": "mfma",
                     "kernel": "bwd_dkdv_bf16_kernel<128,false,false,true> (fox_attn_bwd_dkdv_store)",
                     "achieved": round(kv_tf, 2), "peak": MFMA_BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(kv_tf / MFMA_BF16_PEAK_TFLOPS, 4),
                     "traffic": kv_traffic, "algorithmic_flops_per_launch": fl_kv,
                     "compulsory_bytes_per_launch": kv_bytes},
        "roofline_dq_stored": {"bound": "hbm", "kernel": "bwd_dq_stored_kernel<128,false> "
                               "(fox_attn_bwd_dq_stored)", "achieved": round(dq_gbs, 1),
                               "peak": HBM_PEAK_GBS, "unit": "GB/s",
                               "frac": round(dq_gbs / HBM_PEAK_GBS, 4),
                               "traffic": measured_traffic(DQ_STORED_KERNEL),
                               "compulsory_bytes_per_launch": dq_bytes},
        "recompute": {"what": "the same step with fox_attn_bwd's stages (the dQ pass recomputes "
                              "S and dP; O(L) workspace)",
                      "ms_per_step": round(r["rc_ms"], 4), "TFLOP/s": round(rc_tf, 2),
                      "frac_of_peak": round(rc_tf / MFMA_BF16_PEAK_TFLOPS, 4),
                      "bwd_dkdv_ms": round(r["rc_dkdv_ms"], 4),
                      "bwd_dq_ms": round(r["rc_dq_ms"], 4),
                      "dkdv_traffic": measured_traffic(KV_KERNEL)},
        "skip": {"what": "the same step through fox_attn_fwd_skip / fox_attn_bwd_skip_stored "
                         "(exact gate-aware tile skipping, bound kernels included); outputs "
                         "bitwise equal to the dense step",
                 "ms_per_step": round(r["skip_ms"], 4),
                 "speedup_vs_dense": round(r["ms"] / r["skip_ms"], 3),
                 "dense_equivalent_TFLOP/s": round((fl_f + fl_b) / (r["skip_ms"] * 1e-3) / 1e12,
                                                   2)},
        "roofline_fwd": {"bound": "mfma", "kernel": "fwd_bf16_kernel<128> (fox_attn_fwd)",
                         "achieved": round(fwd_tf, 2), "peak": MFMA_BF16_PEAK_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(fwd_tf / MFMA_BF16_PEAK_TFLOPS, 4),
                         "traffic": measured_traffic(f"fwd_bf16_kernel<{d},false,false,false>",
                                                     fwd_grid_threads(B, H, L))},
        "roofline_bwd": {"bound": "mfma",
                         "kernels": "fox_attn_bwd_stored stages (delta, dkdv_store, dq_stored, scan)",
                         "achieved": round(bwd_tf, 2), "peak": MFMA_BF16_PEAK_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(bwd_tf / MFMA_BF16_PEAK_TFLOPS, 4)},
    }
    log(f"[bench] train step {r['ms']:.3f} ms -> {tflops:.1f} TFLOP/s; recompute backward "
        f"{r['rc_ms']:.3f} ms; with skipping {r['skip_ms']:.3f} ms")
    if not args.no_fixed:
        rf = bench_fixed(w, args.steps, args.warmup)
        out["fixed_gate"] = {
            "what": "fixed per-head gates f = sigmoid(b_h) (ALiBi form), appendix initialisation "
                    "with (T_min, T_max) = (2, L); fwd+bwd step (backward keeping dS) dense and "
                    "with exact skipping (bound kernels included), outputs bitwise equal",
            "dense_ms": round(rf["dense"], 4), "skip_ms": round(rf["skip"], 4),
            "speedup": round(rf["dense"] / rf["skip"], 3),
            "dense_TFLOP/s": round((fl_f + fl_b) / (rf["dense"] * 1e-3) / 1e12, 2)}
        log(f"[bench] fixed gates: step {rf['dense']:.3f} ms, with skipping {rf['skip']:.3f} ms")
    if not args.no_pro:
        rp = bench_pro(w, args.steps, args.warmup)
        rows = B * H * L
        e = 2  # bf16
        # compulsory bytes per row: prologue reads q~, k~, v~ and two shift logits,
        # writes q, k, v; its backward reads q~, k~, v~, dq, dk, dv and the shift
        # logits, writes dq~, dk~, dv~ and two logit gradients; the standalone
        # output gate reads o, g and writes y
        pb = {"prologue": rows * (6 * d * e + 8), "prologue_bwd": rows * (9 * d * e + 16),
              "out_gate": rows * 3 * d * e}
        kern = {"prologue": "pro_prologue_kernel<__bf16,128>",
                "prologue_bwd": "pro_prologue_bwd_kernel<__bf16,128>",
                "out_gate": "out_gate_kernel<__bf16,128>"}
        hbm = {n: {"ms": round(rp[n], 4), "GB/s": round(b / (rp[n] * 1e-3) / 1e9, 1),
                   "frac_of_hbm_peak": round(b / (rp[n] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                   "compulsory_bytes": b, "kernel": kern[n],
                   "traffic": measured_traffic(kern[n])} for n, b in pb.items()}
        pro_ms = rp["prologue"] + rp["fwd_pro"] + rp["bwd_pro"] + rp["prologue_bwd"]
        # practical ceiling for kernels that read and write HBM: a plain device copy
        # of about the prologue's traffic (half read, half written)
        src = torch.empty(pb["prologue"] // 2 // 4, device="cuda:0", dtype=torch.float32)
        dst = torch.empty_like(src)
        tc = EventTimer()
        for i in range(6):
            with tc.maybe(i > 0):
                dst.copy_(src)
        torch.cuda.synchronize()
        copy_gbs = 2 * src.numel() * 4 / (tc.mean_ms() * 1e-3) / 1e9
        del src, dst
        out["pro"] = {
            "what": "FoX (Pro) layer hot path at the same shape: prologue (QK-norm, KV-shift) -> "
                    "attention with the output RMSNorm and sigmoid gate in the forward epilogue "
                    "-> its backward (norm/gate backward fused with Delta, attention backward "
                    "keeping dS: fox_attn_bwd_pro_stored) -> prologue backward",
            "ms_per_step": round(pro_ms, 4),
            "overhead_vs_plain_step": round(pro_ms / (r["fwd_ms"] + r["bwd_ms"]) - 1.0, 4),
            "fwd_pro_ms": round(rp["fwd_pro"], 4), "bwd_pro_ms": round(rp["bwd_pro"], 4),
            "hbm_kernels": hbm,
            "device_copy_GB/s": round(copy_gbs, 1)}
        log(f"[bench] Pro layer {pro_ms:.3f} ms (fwd_pro {rp['fwd_pro']:.3f}, bwd_pro "
            f"{rp['bwd_pro']:.3f}, prologue {rp['prologue']:.3f}, prologue_bwd "
            f"{rp['prologue_bwd']:.3f}, out_gate {rp['out_gate']:.3f})")
    if not args.no_decode:
        wd = inputs.WORKLOADS[args.decode_workload]
        rd = bench_decode(wd, max(args.steps, 10), args.warmup, cpu=not args.no_cpu_baseline)
        byt = decode_bytes(wd.B, wd.H, wd.L, wd.d)
        gbs = byt / (rd["ms"] * 1e-3) / 1e9
        out["decode"] = {"metric": "decode HBM GB/s", "value": round(gbs, 1), "unit": "GB/s",
                         "ms_per_step": round(rd["ms"], 4),
                         "config": {"workload": wd.name, "B": wd.B, "H": wd.H, "T": wd.L,
                                    "d": wd.d, "bytes_per_step": byt, "seed": wd.seed},
                         "roofline": {"bound": "hbm", "kernel": "fox_attn_decode (split + combine)",
                                      "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                                      "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                                      "traffic": measured_traffic(DECODE_KERNEL)},
                         "skip": {"what": "fox_attn_decode_skip: exact gate-aware skipping of key "
                                          "splits, outputs bitwise equal to the dense decode",
                                  "ms_per_step": round(rd["skip_ms"], 4),
                                  "speedup_vs_dense": round(rd["ms"] / rd["skip_ms"], 2),
                                  "dense_equivalent_GB/s": round(byt / (rd["skip_ms"] * 1e-3)
                                                                 / 1e9, 1)}}
        log(f"[bench] decode {rd['ms']:.3f} ms -> {gbs:.0f} GB/s; with skipping "
            f"{rd['skip_ms']:.3f} ms")
    if not args.no_projection:
        rj = bench_projection(w, max(args.steps, 20), args.warmup)
        fb, bb = projection_bytes(rj["B"], rj["L"], rj["H"], rj["M"])
        legs = {}
        tb, tr = measured_traffic(PROJ_BWD_KERNEL), measured_traffic(PROJ_REDUCE_KERNEL)
        for leg, ms, byt, traffic, what in (
                ("fwd", rj["fwd_ms"], fb, measured_traffic(PROJ_FWD_KERNEL), "gate_proj_fwd_kernel"),
                ("bwd", rj["bwd_ms"], bb, None if tb is None or tr is None else tb + tr,
                 "gate_proj_bwd_kernel + gate_proj_reduce_kernel")):
            gbs = byt / (ms * 1e-3) / 1e9
            legs[leg] = {"ms": round(ms, 5), "bytes": byt,
                         "roofline": {"bound": "hbm", "kernel": what, "achieved": round(gbs, 1),
                                      "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                      "frac": round(gbs / HBM_PEAK_GBS, 4),
                                      "traffic": traffic}}
        out["gate_projection"] = {
            "what": "forget-gate logits w_f^T x_t + b_f per head and their backward (dx, dw_f, "
                    "db_f), x bf16 [B, L, H*d]",
            "config": {"B": rj["B"], "L": rj["L"], "H": rj["H"], "M": rj["M"], "seed": PROJ_SEED},
            **legs}
        log(f"[bench] gate projection fwd {rj['fwd_ms'] * 1e3:.1f} us, bwd "
            f"{rj['bwd_ms'] * 1e3:.1f} us")
    if not args.no_other_workloads:
        out["workloads"] = {}
        w2 = inputs.WORKLOADS["fwdbwd_bf16_b8_h12_l2048_d64"]
        r2 = bench_train_graph(w2, args.steps, args.warmup)
        out["workloads"][w2.name] = train_graph_summary(w2, r2)
        log(f"[bench] {w2.name}: step {r2['stored_ms']:.4f} ms (keeping dS), "
            f"{r2['recompute_ms']:.4f} ms (recomputing)")
        w4 = inputs.WORKLOADS["fwd_bf16_b1_h16_l65536_d128"]
        r4 = bench_prefill(w4, max(3, args.steps // 4), 1)
        fl4 = fwd_flops(w4.B, w4.H, w4.L, w4.d)
        tf4 = fl4 / (r4["fwd_ms"] * 1e-3) / 1e12
        out["workloads"][w4.name] = {
            "what": "length-extrapolation prefill: gate prefix -> forward (O, LSE); heads 0-7 "
                    "logits N(6, 1), heads 8-15 N(0, variance 2)",
            "config": {"B": w4.B, "H": w4.H, "L": w4.L, "d": w4.d, "seed": w4.seed,
                       "flops_per_step": fl4},
            "ms_per_step": round(r4["ms"], 4),
            "TFLOP/s": round(fl4 / (r4["ms"] * 1e-3) / 1e12, 2),
            "frac_of_peak": round(fl4 / (r4["ms"] * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
            "roofline": {"bound": "mfma", "kernel": "fwd_bf16_kernel<128> (fox_attn_fwd)",
                         "achieved": round(tf4, 2), "peak": MFMA_BF16_PEAK_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(tf4 / MFMA_BF16_PEAK_TFLOPS, 4),
                         "traffic": measured_traffic(f"fwd_bf16_kernel<{w4.d},false,false,false>",
                                                     fwd_grid_threads(w4.B, w4.H, w4.L)),
                         "algorithmic_flops_per_launch": fl4}}
        log(f"[bench] {w4.name}: forward {r4['fwd_ms']:.3f} ms -> {tf4:.1f} TFLOP/s")
    if not args.no_cpu_baseline:
        log("[bench] timing the fp64 oracle on the host")
        out["cpu_baseline"] = cpu_baseline(w)
        if not args.no_other_workloads:
            w1 = inputs.WORKLOADS["fwd_f32_b1_h2_l256_d64"]
            out["workloads"][w1.name] = {"what": "fp32 forward (parity workload; oracle time "
                                                 "only)",
                                         "cpu_baseline": cpu_baseline_full(w1)}
            out["workloads"][w2.name]["cpu_baseline"] = cpu_baseline_full(w2)
            out["workloads"][w4.name]["cpu_baseline"] = cpu_baseline_rows(w4)
            log("[bench] oracle times of the other workloads done")
        if not args.no_decode and "decode_cpu_baseline" in rd:
            out["decode"]["cpu_baseline"] = rd["decode_cpu_baseline"]
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
