"""Benchmark: jagged HSTU attention forward + backward on one MI355X.

One step = the whole hot path over one batch: the forward call (scheduler,
attention, LayerNorm x U) and the backward call (scheduler, LayerNorm
backward, dQ, dK/dV with table gradients, table finalize), on synthetic
inputs already resident in HBM.

Headline: valid-token TFLOP/s = 12 d H P / t_step, with P = sum_b
L_b (L_b + 1) / 2 causal pairs per head (forward 4 d H P for QK^T and AV,
backward 8 d H P for dA, dV, dQ, dK; recompute, bias, SiLU and LayerNorm
work are not credited; padding does not exist), on the largest workload
that fits one GPU: the Zipf batch (1024 sequences, lengths 1..8192, H = 4,
d = 64, position bias).  Prints one JSON line, which also carries a
"configs" object with every workload timed the same way (the fp32
forward-only parity batch by its forward time), each beside its roofline
ceiling.

With the layer workload (--workload 4) the line also carries a "layer"
object: the whole HSTU layer around the attention (f1/f2 GEMMs, SiLU split
and their backward) timed the same way.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 5]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0          # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3           # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0              # MI355X HBM3E
RIDGE = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)   # flop per byte

KERNEL_SOURCES = ["device.h", "internal.h", "sched_impl.h", "sched.hip", "attn_bf16.hip",
                  "attn_f32.hip", "norm.hip", "api.cpp"]


def _code_only(text: str) -> str:
    """C/C++ source without comments and with whitespace collapsed, so that a
    change to comments or layout does not mark measurements as stale."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":                       # string or char literal, kept whole
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_sha() -> str:
    """Hash of the kernel and launch sources' code (comments and layout
    ignored) and their compiler flags: profiles taken from other code are
    reported as stale."""
    from paper_2605_13433_amd import build as _build
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2605_13433_amd", "csrc", f), encoding="utf-8") as fh:
            h.update(_code_only(fh.read()).encode())
        h.update(repr(_build.FILE_FLAGS.get(f, [])).encode())
    h.update(repr(_build.CFLAGS).encode())
    return h.hexdigest()[:16]


def kernel_work(name, w, elem_bytes):
    """(algorithmic bytes, algorithmic flops) of one launch of `name`.

    Bytes count each tensor element read or written once at its storage
    width, per (token, head, dim) element E = T*H*d:
      attn_fwd   reads q, k, v; writes o                    4 E elements
      ln_fwd     reads o, u; writes y  (+ mean, rstd)       3 E (+ 2 T fp32)
      ln_bwd     reads dy, u, o; writes du, dO (+ stats)    5 E (+ 2 T fp32)
      attn_bwd      reads q, k, v, dO; writes dq, dk, dv    7 E   (one launch)
      attn_bwd_dkv  reads q, k, v, dO; writes dk, dv        6 E   (or two
      attn_bwd_dq   reads q, k, v, dO; writes dq            5 E    launches)
    Flops are the credited contractions: fwd QK^T + AV = 4 d H P; backward
    dA, dQ, dV, dK = 8 d H P, of which dA, dV, dK (6 d H P) are the dK/dV
    kernel's and dQ (2 d H P) the dQ kernel's when the backward runs as two
    launches (the dQ kernel's recomputed scores and dA are not credited).
    """
    E = w.T * w.H * w.d
    P = w.pairs
    tok = 8 * w.T
    table = {
        "attn_fwd": (4 * E * elem_bytes, 4 * w.d * w.H * P),
        "ln_fwd": (3 * E * elem_bytes + tok, 0),
        "ln_bwd": (5 * E * elem_bytes + tok, 0),
        "attn_bwd": (7 * E * elem_bytes, 8 * w.d * w.H * P),
        "attn_bwd_dkv": (6 * E * elem_bytes, 6 * w.d * w.H * P),
        "attn_bwd_dq": (5 * E * elem_bytes, 2 * w.d * w.H * P),
    }
    return table.get(name, (0, 0))


def load_traffic(kernel: str, workload: str, sha: str):
    """HBM bytes per launch from the committed rocprofv3 --pmc summary, if it
    was taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_counters.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_sha") != sha:
        return None
    try:
        fetch = float(vals["fetch_kib_per_dispatch"])
        write = float(vals["write_kib_per_dispatch"])
        scale_f = float(vals.get("fetch_scale", 1.0))
        scale_w = float(vals.get("write_scale", 1.0))
    except (KeyError, ValueError):
        return None
    return (fetch * scale_f + write * scale_w) * 1024.0


def load_clock(kernel: str, workload: str, sha: str):
    """Average shader clock (MHz) during the kernel's dispatches, from the
    committed counter summary (GRBM_GUI_ACTIVE cycles over the dispatch
    duration), if taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_counters.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_sha") != sha:
        return None
    try:
        return float(vals["clock_mhz"])
    except (KeyError, ValueError):
        return None


def read_kernel_profile(lib):
    """Per-kernel averages from the library's event profiler (same stream)."""
    import ctypes
    nmax = 32
    names = (ctypes.c_char_p * nmax)()
    tot = (ctypes.c_double * nmax)()
    cnt = (ctypes.c_int * nmax)()
    lib.hstu_profile_read.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_char_p),
                                      ctypes.POINTER(ctypes.c_double),
                                      ctypes.POINTER(ctypes.c_int)]
    rows = lib.hstu_profile_read(nmax, names, tot, cnt)
    return {names[i].decode(): {"avg_us": 1e3 * tot[i] / cnt[i], "launches": cnt[i]}
            for i in range(max(rows, 0))}


def layer_bench(lib, w, steps, warmup, stream):
    """The full HSTU layer (f1 GEMM, SiLU split, attention + LN*U, f2 GEMM,
    and the backward through all of them) on the same batch: step time,
    credited flops (six GEMMs + the attention's 12 d H P) and per-kernel
    times, GEMMs with their TFLOP/s against the bf16 MFMA peak."""
    import torch
    from paper_2605_13433_amd import hstu
    e = w.extra
    dev = lambda t: None if t is None else t.contiguous().cuda()
    x, w1, w2, off, dout = (dev(t) for t in (e["x"], e["w1"], e["w2"], w.seq_offsets,
                                             e["dout"]))
    pos, tw, ts = dev(w.pos_w), dev(w.time_w), dev(w.timestamps)
    plan = hstu.LayerPlan(x, off, w.N, w.H, w.d, pos, tw, ts, w.num_buckets)

    def step():
        plan.forward(x, w1, w2, off, stream)
        plan.backward(x, w1, w2, off, dout, stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(steps):
        step()
    b.record(stream)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    lib.hstu_profile_enable(1)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    lib.hstu_profile_enable(0)
    kernels = read_kernel_profile(lib)
    T, D, C = w.T, x.shape[1], w.H * w.d
    big, small = 2.0 * T * D * 4 * C, 2.0 * T * C * D
    gemm_flops = {"gemm_f1": big, "gemm_f2": small, "gemm_dy": small,
                  "gemm_dw2": small, "gemm_dx": big, "gemm_dw1": big}
    for n, r in kernels.items():
        if n in gemm_flops:
            r["TFLOP_s"] = round(gemm_flops[n] / (r["avg_us"] * 1e-6) / 1e12, 1)
            r["frac_of_bf16_peak"] = round(r["TFLOP_s"] / PEAK_BF16_TFLOPS, 4)
        r["avg_us"] = round(r["avg_us"], 2)
    attn = 12.0 * w.d * w.H * w.pairs
    g = sum(gemm_flops.values())
    return {
        "ms_per_step": round(ms, 5),
        "credited_flops": g + attn,
        "gemm_flops": g,
        "attention_flops": attn,
        "TFLOP_s": round((g + attn) / (ms * 1e-3) / 1e12, 2),
        "pct_of_bf16_peak": round(100.0 * (g + attn) / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 3),
        "d_model": int(D),
        "kernels": kernels,
    }


def embedding_bench(stream, steps, warmup, dtype_name="f32"):
    """The jagged multi-table embedding lookup on the sequence-feature batch
    (8 tables of 128 .. 4 M rows, 32 sequences of 1 .. 4160 tokens, D = 128,
    token-major output): forward and backward times with HIP events on the
    launch stream, and the forward's HBM roofline (algorithmic bytes: the id,
    the table row read and the output row written per id)."""
    import torch
    from paper_2605_13433_amd import emb_inputs
    from paper_2605_13433_amd import embedding as emb
    dtype = torch.float32 if dtype_name == "f32" else torch.bfloat16
    b = emb_inputs.sequence_batch(dtype=dtype)
    W = b.weights.cuda()
    ids = b.ids.cuda()
    ro, io = b.row_offsets.cuda(), b.id_offsets.cuda()
    dout = emb_inputs.token_layout(b.dout, b.F).cuda()
    p = emb.plan(W, ro, io, b.total_rows, b.n, "token")
    out = torch.empty(p.out_shape, dtype=W.dtype, device="cuda")
    grad = torch.zeros(b.total_rows, b.D, dtype=torch.float32, device="cuda")
    uniq = torch.empty(b.n, dtype=torch.int64, device="cuda")
    cnt = torch.empty(1, dtype=torch.int32, device="cuda")

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        z = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(steps):
            fn()
        z.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(z) / steps * 1e3

    fwd_us = timed(lambda: emb.lookup(p, W, ids, out, stream))
    pf = emb.plan(W, ro, io, b.total_rows, b.n, "flat", with_bwd=False)
    out_flat = torch.empty(pf.out_shape, dtype=W.dtype, device="cuda")
    fwd_flat_us = timed(lambda: emb.lookup(pf, W, ids, out_flat, stream))
    del out_flat
    bwd_us = timed(lambda: emb.lookup_backward(p, ids, dout, grad, uniq, cnt, stream))
    U = int(cnt.item())
    es = W.element_size()
    fwd_bytes = b.n * (8 + 2 * b.D * es)
    bwd_bytes = b.n * (8 + b.D * es) + U * (b.D * 4 + 8)
    fwd_gbs = fwd_bytes / (fwd_us * 1e-6) / 1e9
    padded = b.F * len(b.lengths) * emb_inputs.EMB_MAX_LEN
    return {
        "workload": b.name,
        "tables": b.F, "rows": [int(r) for r in b.rows], "D": b.D, "dtype": dtype_name,
        "num_ids": b.n, "padded_ids": padded, "distinct_rows": U,
        "fwd_us": round(fwd_us, 2), "bwd_us": round(bwd_us, 2),
        "fwd_flat_layout_us": round(fwd_flat_us, 2),
        "fwd_GB_s": round(fwd_gbs, 1),
        "bwd_GB_s": round(bwd_bytes / (bwd_us * 1e-6) / 1e9, 1),
        "roofline": {"bound": "hbm", "kernel": "emb_fwd", "achieved": round(fwd_gbs, 1),
                     "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(fwd_gbs / PEAK_HBM_GBS, 4),
                     "algorithmic_bytes": fwd_bytes},
    }


def rab_bench(stream, steps, warmup, idx=3):
    """The standalone RAB operator on workload `idx` (position table, time
    buckets and the functional time encoding): the jagged bias tensor the
    fused attention never materialises, its size, and forward / backward
    times with HIP events on the launch stream (HBM roofline on the bytes
    of that tensor: written by the forward, read by the backward)."""
    import torch
    from paper_2605_13433_amd import hstu, inputs
    w = inputs.workload(idx)
    L = w.lengths.astype(np.int64)
    S = int((L * L).sum())
    fn = torch.tensor([[0.3, 0.5]] * w.H, dtype=torch.float32)
    dev = lambda t: None if t is None else t.contiguous().cuda()
    plan = hstu.RabPlan(dev(w.seq_offsets), w.N, w.H, w.T, S, dev(w.pos_w), dev(w.time_w),
                        dev(fn), dev(w.timestamps), w.num_buckets)
    g = torch.randn(w.H, S, device="cuda", dtype=torch.float32)

    def timed(fn_):
        for _ in range(warmup):
            fn_()
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        z = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(steps):
            fn_()
        z.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(z) / steps * 1e3

    fwd_us = timed(lambda: plan.forward(stream))
    bwd_us = timed(lambda: plan.backward(g, stream))
    nbytes = 4 * w.H * S
    gbs = nbytes / (fwd_us * 1e-6) / 1e9
    return {
        "workload": w.name, "H": w.H, "square_elements_per_head": S,
        "materialized_bytes": nbytes,
        "fwd_us": round(fwd_us, 2), "bwd_us": round(bwd_us, 2),
        "fwd_GB_s": round(gbs, 1),
        "bwd_GB_s": round(nbytes / (bwd_us * 1e-6) / 1e9, 1),
        "roofline": {"bound": "hbm", "kernel": "rab_fwd", "achieved": round(gbs, 1),
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                     "algorithmic_bytes": nbytes},
    }


def cpu_baseline(w, target_s=20.0):
    """The oracle, as it stands, on a bounded sample of the same workload:
    whole sequences in a seeded random order until the estimated
    forward+backward time reaches `target_s`."""
    from oracle import oracle
    from paper_2605_13433_amd import inputs
    oracle.build(force=False)
    rng = np.random.default_rng(12345)
    order = rng.permutation(w.B)
    # calibrate on a small slice, then size the sample
    pairs = w.lengths * (w.lengths + 1) // 2
    probe, acc = [], 0
    for b in order:
        probe.append(int(b))
        acc += pairs[b]
        if acc >= 2e6:
            break
    sub = inputs.subset(w, sorted(probe))
    oracle.fwd_workload(sub)                 # first run: thread pool and pages warm up
    oracle.bwd_workload(sub)
    t0 = time.perf_counter()
    oracle.fwd_workload(sub)
    oracle.bwd_workload(sub)
    rate = max(acc, 1) / max(time.perf_counter() - t0, 1e-6)   # pairs per second
    budget = rate * target_s
    seqs, acc = [], 0
    for b in order:
        if acc + pairs[b] > budget and seqs:
            continue
        seqs.append(int(b))
        acc += pairs[b]
    sub = inputs.subset(w, sorted(seqs))
    # when the whole batch is far below the budget, repeat it
    reps = max(1, int(budget // max(acc, 1)))
    t0 = time.perf_counter()
    for _ in range(reps):
        oracle.fwd_workload(sub)
        oracle.bwd_workload(sub)
    dt = time.perf_counter() - t0
    flops = 12.0 * w.d * w.H * sub.pairs * reps
    return {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": oracle.num_threads(),
        "kind": "oracle",
        "sample": (f"{len(seqs)} of {w.B} sequences ({sub.T} tokens, {sub.pairs} "
                   f"causal pairs/head, {100.0 * sub.pairs / w.pairs:.1f}% of the "
                   f"batch's pairs) x {reps} repetition(s), f64 forward + backward, "
                   f"{dt:.1f} s"),
    }


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def ceiling_frac(w):
    """Roofline ceiling of a workload as a fraction of bf16 MFMA peak: its
    credited flops (12 d H P) over the minimum HBM bytes of forward and
    backward in bf16 (36 bytes per (token, head, dim) element: forward reads
    q, k, v, u and writes y, o; LayerNorm backward reads dy, u, o and writes
    du, dO; attention backward reads q, k, v, dO and writes dq, dk, dv),
    times 8 TB/s, capped at 1."""
    ai = 12.0 * w.d * w.H * w.pairs / (36.0 * w.T * w.H * w.d)
    return min(1.0, ai * PEAK_HBM_GBS * 1e9 / (PEAK_BF16_TFLOPS * 1e12))


class AttnRun:
    """One workload resident on the GPU with its plan; step() enqueues one
    forward + backward (forward only for forward-only workloads)."""

    def __init__(self, w, stream):
        from paper_2605_13433_amd import hstu
        dev = lambda t: None if t is None else t.contiguous().cuda()
        self.w = w
        self.stream = stream
        self.q, self.k, self.v, self.u, self.off = (
            dev(x) for x in (w.q, w.k, w.v, w.u, w.seq_offsets))
        self.dy = dev(w.dy)
        pos, tw, ts = dev(w.pos_w), dev(w.time_w), dev(w.timestamps)
        self.bwd = w.dy is not None
        self.plan = hstu.Plan(self.q, self.off, w.N, pos, tw, ts, w.num_buckets,
                              backward=self.bwd)

    def step(self):
        self.plan.forward(self.q, self.k, self.v, self.u, self.off, self.stream)
        if self.bwd:
            self.plan.backward(self.q, self.k, self.v, self.u, self.off, self.dy, self.stream)

    def time(self, steps, warmup):
        """(ms per step, wall seconds of the timed region): HIP events on the
        launch stream around exactly `steps` steps after `warmup` untimed ones."""
        import torch
        for _ in range(warmup):
            self.step()
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        ev0.record(self.stream)
        for _ in range(steps):
            self.step()
        ev1.record(self.stream)
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / steps, time.perf_counter() - t0

    def kernel_times(self, lib, steps):
        """Per-kernel averages from the library's event profiler."""
        import torch
        lib.hstu_profile_enable(1)
        for _ in range(steps):
            self.step()
        torch.cuda.synchronize()
        lib.hstu_profile_enable(0)
        return read_kernel_profile(lib)


def config_summary(w, ms, kernels):
    """One entry of the per-workload report."""
    flops = (12.0 if w.dy is not None else 4.0) * w.d * w.H * w.pairs
    tf = flops / (ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if w.dtype_name == "bf16" else PEAK_FP32_TFLOPS
    out = {
        "workload": w.name,
        "dtype": w.dtype_name,
        "pass": "fwd+bwd" if w.dy is not None else "fwd",
        "total_tokens": w.T,
        "causal_pairs_per_head": w.pairs,
        "max_seq_len": int(w.lengths.max()),
        "ms_per_step": round(ms, 5),
        "TFLOP_s": round(tf, 3),
        "pct_of_peak": round(100.0 * tf / peak, 3),
        "peak_TFLOP_s": peak,
        "kernels_us": {n: round(r["avg_us"], 2) for n, r in kernels.items()},
    }
    if w.dy is not None and w.dtype_name == "bf16":
        c = ceiling_frac(w)
        out["roofline_ceiling_pct"] = round(100.0 * c, 2)
        out["pct_of_ceiling"] = round(100.0 * tf / PEAK_BF16_TFLOPS / c, 2)
    return out


# ------------------------------------------------------------ counter summaries
# rocprofv3 passes over one bench.py command (see counters_commands()): a
# kernel trace for durations, two passes of SQ_ / GRBM_ counters, FETCH_SIZE
# and WRITE_SIZE; and the same two HBM counters over a 256 MiB device copy
# (bench.py --copy-probe-mib 256) to calibrate them.
SQ_PASS_A = ["SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES", "SQ_ACTIVE_INST_VALU",
             "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_ACTIVE_INST_LDS", "SQ_WAIT_INST_ANY",
             "SQ_ACTIVE_INST_ANY", "SQ_INSTS_VALU", "GRBM_GUI_ACTIVE"]
SQ_PASS_B = ["SQ_INSTS_MFMA", "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT",
             "SQ_INSTS_VALU_TRANS_F32", "SQ_WAIT_INST_LDS", "SQ_THREAD_CYCLES_VALU",
             "SQ_VALU_MFMA_COEXEC_CYCLES", "SQ_LDS_IDX_ACTIVE"]
SHORT_KERNEL = {"attn_fwd_kernel": "attn_fwd", "attn_bwd_kernel": "attn_bwd",
                "attn_bwd_dkv_kernel": "attn_bwd_dkv", "attn_bwd_dq_kernel": "attn_bwd_dq",
                "ln_fwd_kernel": "ln_fwd", "ln_bwd_kernel": "ln_bwd",
                "schedule_kernel": "schedule", "finalize_tables_kernel": "finalize_tables"}


def counters_commands(workload: int):
    run = (f"python3 bench.py --workload {workload} --steps 5 --warmup 2 --no-cpu-baseline "
           f"--cold-steps 0 --no-configs")
    return {
        "trace": f"rocprofv3 --kernel-trace --stats --output-format csv -d <dir> -o trace -- {run}",
        "sq_a": f"rocprofv3 --pmc {' '.join(SQ_PASS_A)} --output-format csv -d <dir> -o sqa -- {run}",
        "sq_b": f"rocprofv3 --pmc {' '.join(SQ_PASS_B)} --output-format csv -d <dir> -o sqb -- {run}",
        "fetch": f"rocprofv3 --pmc FETCH_SIZE --output-format csv -d <dir> -o fetch -- {run}",
        "write": f"rocprofv3 --pmc WRITE_SIZE --output-format csv -d <dir> -o write -- {run}",
        "calibration": ("rocprofv3 --pmc FETCH_SIZE (then WRITE_SIZE) --output-format csv "
                        "-d <dir> -o cal_fetch (cal_write) -- python3 bench.py --copy-probe-mib 256"),
    }


def _kernel_key(name: str):
    import re
    m = re.search(r"(\w+_kernel|__amd_rocclr_copyBuffer)(<[^>]*>)?", name)
    if not m:
        return None
    base = m.group(1)
    return base, (m.group(2) or "")


def _read_counters(path):
    """{(kernel, template): {counter: [per-dispatch values]}} from a rocprofv3
    counter_collection.csv (one row per dispatch and counter)."""
    import csv
    import collections
    out = collections.defaultdict(lambda: collections.defaultdict(list))
    with open(path) as fh:
        for row in csv.DictReader(fh):
            key = _kernel_key(row["Kernel_Name"])
            if key:
                out[key][row["Counter_Name"]].append(float(row["Counter_Value"]))
    return out


def summarize_counters(d, workload, num_cu=256):
    """Per-kernel counter summaries of one workload from the rocprofv3 output
    directory `d`; returns {short kernel name: text}."""
    import csv
    import glob
    w_name = inputs_name(workload)
    # the kernel-source hash of the code that ran: from the bench JSON line
    # the profiled runs printed
    sha = None
    for f in sorted(glob.glob(os.path.join(d, "*.log"))):
        with open(f) as fh:
            for line in fh:
                if line.startswith("{") and "kernel_source_sha" in line:
                    sha = json.loads(line)["kernel_source_sha"]
    if sha is None:
        raise SystemExit(f"no bench.py JSON line with kernel_source_sha under {d}")
    durs = {}
    for f in glob.glob(os.path.join(d, "*trace_kernel_stats.csv")):
        with open(f) as fh:
            for row in csv.DictReader(fh):
                key = _kernel_key(row["Name"])
                if key:
                    durs[key] = (float(row["AverageNs"]) / 1e3, int(row["Calls"]))
    cnt = {}
    for f in glob.glob(os.path.join(d, "*counter_collection.csv")):
        for key, c in _read_counters(f).items():
            cnt.setdefault(key, {}).update(c)
    cal = {}
    for tag, name in (("cal_fetch", "FETCH_SIZE"), ("cal_write", "WRITE_SIZE")):
        for f in glob.glob(os.path.join(d, f"{tag}*counter_collection.csv")):
            for key, c in _read_counters(f).items():
                if key[0] == "__amd_rocclr_copyBuffer" and name in c:
                    cal[name] = max(c[name])
    copy_kib = 256 * 1024.0
    fscale = copy_kib / cal["FETCH_SIZE"] if cal.get("FETCH_SIZE") else None
    wscale = copy_kib / cal["WRITE_SIZE"] if cal.get("WRITE_SIZE") else None
    # GPU geometry from the profiler's agent table: GRBM_GUI_ACTIVE is summed
    # over the XCDs (accelerator dies), each with its own clock counter
    num_xcc, num_cu = 8, num_cu
    for f in glob.glob(os.path.join(d, "*agent_info.csv")):
        with open(f) as fh:
            for row in csv.DictReader(fh):
                if row.get("Agent_Type") == "GPU" or row.get("Num_Xcc", "0") not in ("0", ""):
                    if int(row.get("Cu_Count") or 0) > 0:
                        num_xcc = int(row["Num_Xcc"])
                        num_cu = int(row["Cu_Count"])
    cmds = counters_commands(workload)
    out = {}
    for key, c in cnt.items():
        short = SHORT_KERNEL.get(key[0])
        if not short or key not in durs:
            continue
        avg = {n: sum(v) / len(v) for n, v in c.items()}
        us, calls = durs[key]
        lines = [f"# rocprofv3 counters: {key[0]}{key[1]}, workload {w_name}",
                 "# commands (each a run of its own; <dir> = the output directory):"]
        lines += [f"#   {k}: {v}" for k, v in cmds.items()]
        lines += ["# values: mean over the kernel's dispatches in the run.  GRBM_GUI_ACTIVE"
                  f" sums the {num_xcc} XCDs' busy cycles: clock = GRBM_GUI_ACTIVE / {num_xcc}"
                  " / duration;",
                  f"# SIMD-cycles = GRBM_GUI_ACTIVE / {num_xcc} x {num_cu} CUs x 4 SIMDs;"
                  " SQ_VALU_MFMA_BUSY_CYCLES counts SIMD-cycles (32 per 32x32x16 MFMA);",
                  "# SQ_ACTIVE_INST_VALU and SQ_ACTIVE_INST_LDS count quad-cycles (x4);"
                  " SQ_LDS_IDX_ACTIVE counts CU-cycles.",
                  f"source_sha: {sha}",
                  f"dispatches_traced: {calls}",
                  f"trace_avg_us: {us:.2f}"]
        for n in SQ_PASS_A + SQ_PASS_B + ["FETCH_SIZE", "WRITE_SIZE"]:
            if n in avg:
                lines.append(f"{n}: {avg[n]:.1f}")
        g = avg.get("GRBM_GUI_ACTIVE")
        if g:
            cyc = g / num_xcc                     # busy cycles of one XCD
            simd = cyc * num_cu * 4
            lines.append(f"clock_mhz: {cyc / us:.0f}")
            if "SQ_VALU_MFMA_BUSY_CYCLES" in avg:
                lines.append(f"mfma_busy_frac: {avg['SQ_VALU_MFMA_BUSY_CYCLES'] / simd:.4f}")
            if "SQ_INSTS_MFMA" in avg:
                # v_mfma_f32_32x32x16_bf16: 8 passes of 4 cycles on one SIMD
                lines.append(f"mfma_insts_x32_frac: {avg['SQ_INSTS_MFMA'] * 32 / simd:.4f}")
            if "SQ_ACTIVE_INST_VALU" in avg:
                lines.append(f"valu_busy_frac: {4 * avg['SQ_ACTIVE_INST_VALU'] / simd:.4f}")
            if "SQ_ACTIVE_INST_LDS" in avg:
                lines.append(f"lds_inst_busy_frac: {4 * avg['SQ_ACTIVE_INST_LDS'] / simd:.4f}")
            if "SQ_LDS_IDX_ACTIVE" in avg:
                lines.append(f"lds_idx_active_frac: "
                             f"{avg['SQ_LDS_IDX_ACTIVE'] / (cyc * num_cu):.4f}")
        if "SQ_INSTS_MFMA" in avg and avg["SQ_INSTS_MFMA"] > 0:
            m = avg["SQ_INSTS_MFMA"]
            for n, lab in (("SQ_INSTS_VALU", "valu"), ("SQ_INSTS_VALU_TRANS_F32", "trans"),
                           ("SQ_INSTS_LDS", "lds")):
                if n in avg:
                    lines.append(f"{lab}_insts_per_mfma: {avg[n] / m:.3f}")
        if "SQ_LDS_BANK_CONFLICT" in avg and avg.get("SQ_LDS_IDX_ACTIVE"):
            lines.append(f"lds_bank_conflict_per_idx_active: "
                         f"{avg['SQ_LDS_BANK_CONFLICT'] / avg['SQ_LDS_IDX_ACTIVE']:.4f}")
        if "FETCH_SIZE" in avg and fscale:
            lines += [f"fetch_kib_per_dispatch: {avg['FETCH_SIZE']:.1f}",
                      f"fetch_scale: {fscale:.4f}"]
        if "WRITE_SIZE" in avg and wscale:
            lines += [f"write_kib_per_dispatch: {avg['WRITE_SIZE']:.1f}",
                      f"write_scale: {wscale:.4f}"]
        if "FETCH_SIZE" in avg and "WRITE_SIZE" in avg and fscale and wscale:
            hbm = (avg["FETCH_SIZE"] * fscale + avg["WRITE_SIZE"] * wscale) * 1024.0
            lines += [f"hbm_bytes_per_dispatch: {hbm:.0f}",
                      f"hbm_GB_s: {hbm / (us * 1e-6) / 1e9:.1f}"]
        out[short] = "\n".join(lines) + "\n"
    return out


def inputs_name(workload: int) -> str:
    from paper_2605_13433_amd import inputs
    return inputs.WORKLOADS[workload]["name"]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=5)
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-workload report of the other workloads")
    ap.add_argument("--config-steps", type=int, default=20,
                    help="timed steps of each other workload in the per-workload report")
    ap.add_argument("--cold-steps", type=int, default=10,
                    help="extra steps, each after a 1 GiB cache flush")
    ap.add_argument("--no-embedding", action="store_true",
                    help="skip the embedding-lookup measurement")
    ap.add_argument("--embedding-only", action="store_true",
                    help="only time the embedding lookup (prints its JSON object)")
    ap.add_argument("--rab-only", action="store_true",
                    help="only time the standalone RAB operator (workloads 2-4)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run 5 device copies of this many MiB (counter calibration)")
    ap.add_argument("--summarize-counters", metavar="DIR", default=None,
                    help="only write profiles/<kernel>_<workload>_counters.txt from the "
                         "rocprofv3 output in DIR (see counters_commands)")
    args = ap.parse_args()

    if args.summarize_counters:
        for short, text in summarize_counters(args.summarize_counters, args.workload).items():
            path = os.path.join(ROOT, "profiles",
                                f"{short}_{inputs_name(args.workload)}_counters.txt")
            with open(path, "w") as fh:
                fh.write(text)
            print(path)
        return

    if args.copy_probe_mib:
        import torch
        src = torch.ones(args.copy_probe_mib << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": src.numel() * 4}))
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the jagged attention runs on a single "
              "MI355X here (sequences are independent, so a multi-GPU run would shard "
              "them with no forward exchange and one table all-reduce in the "
              "backward). Use --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2605_13433_amd import hstu, inputs

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    lib = hstu.load_library()
    stream = torch.cuda.current_stream()

    if args.embedding_only:
        for dt in ("f32", "bf16"):
            print(json.dumps(embedding_bench(stream, args.steps, args.warmup, dt)), flush=True)
        return
    if args.rab_only:
        for idx in (2, 3, 4):
            print(json.dumps(rab_bench(stream, args.steps, args.warmup, idx)), flush=True)
        return

    w = inputs.workload(args.workload, args.seed)
    if w.dy is None:
        print(f"workload {args.workload} is forward-only; pick a fwd+bwd workload",
              file=sys.stderr)
        sys.exit(2)
    print(f"[bench] workload {args.workload} {w.name}: T={w.T} pairs/head={w.pairs}",
          file=sys.stderr, flush=True)
    run = AttnRun(w, stream)

    # ---- timed region: exactly K steps
    ms_per_step, wall_s = run.time(args.steps, args.warmup)
    flops_step = 12.0 * w.d * w.H * w.pairs
    value = flops_step / (ms_per_step * 1e-3) / 1e12
    print(f"[bench] timed {args.steps} steps: {ms_per_step:.4f} ms/step", file=sys.stderr,
          flush=True)

    # ---- per-kernel durations: HIP events around every launch, same stream
    kernels = run.kernel_times(lib, args.steps)

    # ---- cold cache: flush L2 + MALL (1 GiB of writes) before each step
    cold_ms = None
    if args.cold_steps > 0:
        flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        times = []
        for _ in range(args.cold_steps):
            flush.fill_(1.0)
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            run.step()
            b.record(stream)
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b))
        cold_ms = float(np.median(times))
        del flush

    # ---- roofline of the dominant kernel
    elem_bytes = 2 if w.dtype == torch.bfloat16 else 4
    sha = kernel_source_sha()
    per_kernel_total = {n: r["avg_us"] * r["launches"] for n, r in kernels.items()}
    dominant = max(per_kernel_total, key=per_kernel_total.get)
    nbytes, nflops = kernel_work(dominant, w, elem_bytes)
    avg_s = kernels[dominant]["avg_us"] * 1e-6
    if nflops and nbytes and nflops / nbytes > RIDGE:
        roof = {"bound": "mfma", "achieved": nflops / avg_s / 1e12,
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": nbytes / avg_s / 1e9,
                "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["kernel"] = dominant
    traffic = load_traffic(dominant, w.name, sha)
    roof["traffic"] = traffic
    roof["algorithmic_bytes"] = nbytes
    roof["algorithmic_flops"] = nflops
    clock = load_clock(dominant, w.name, sha)
    roof["clock_mhz"] = clock

    for n, r in kernels.items():
        b, f = kernel_work(n, w, elem_bytes)
        s = r["avg_us"] * 1e-6
        r["GB_s"] = round(b / s / 1e9, 1) if b else None
        r["TFLOP_s"] = round(f / s / 1e12, 2) if f else None
        r["avg_us"] = round(r["avg_us"], 2)

    w.dtype_name = "bf16" if w.dtype == torch.bfloat16 else "f32"
    out = {
        "metric": "jagged HSTU attn fwd+bwd valid-token TFLOP/s + % of bf16 MFMA peak, 1 GPU",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype_name,
        "data": "synthetic (seeded long-tailed jagged lengths, N(0,1) q/k/v/u/dy, "
                "N(0,0.1) bias tables, Poisson-gap timestamps)",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "d": w.d, "max_len": w.N,
                   "total_tokens": w.T, "causal_pairs_per_head": w.pairs,
                   "max_seq_len": int(w.lengths.max()), "rab": {
                       "pos": w.pos_w is not None, "time": w.time_w is not None,
                       "num_buckets": w.num_buckets if w.time_w is not None else 0},
                   "seed": args.workload if args.seed is None else args.seed,
                   "parallelism": "single GPU"},
        "pct_of_bf16_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 3),
        "roofline_ceiling_pct": round(100.0 * ceiling_frac(w), 2),
        "wall_s_timed_region": round(wall_s, 4),
        "cold_ms_per_step": None if cold_ms is None else round(cold_ms, 5),
        "cold_value": None if cold_ms is None else round(flops_step / (cold_ms * 1e-3) / 1e12, 3),
        "kernels": kernels,
        "roofline": roof,
        "kernel_source_sha": sha,
        "gpu": torch.cuda.get_device_name(0),
    }
    if "x" in w.extra:
        out["layer"] = layer_bench(lib, w, args.steps, args.warmup, stream)
    del run
    torch.cuda.empty_cache()

    # ---- every workload, timed the same way, beside its roofline ceiling
    if not args.no_configs:
        configs = {}
        for idx in sorted(inputs.WORKLOADS):
            if idx == args.workload and args.seed is None:
                configs[str(idx)] = config_summary(w, ms_per_step, kernels)
                continue
            wc = inputs.workload(idx)
            wc.dtype_name = "bf16" if wc.dtype == torch.bfloat16 else "f32"
            rc = AttnRun(wc, stream)
            ms, _ = rc.time(args.config_steps, min(args.warmup, 5))
            kt = rc.kernel_times(lib, args.config_steps)
            configs[str(idx)] = config_summary(wc, ms, kt)
            print(f"[bench] workload {idx} {wc.name}: {ms:.4f} ms/step", file=sys.stderr,
                  flush=True)
            del rc
            torch.cuda.empty_cache()
        out["configs"] = configs

    if not args.no_embedding:
        out["embedding"] = embedding_bench(stream, args.config_steps, min(args.warmup, 5))
        torch.cuda.empty_cache()
        out["rab_standalone"] = rab_bench(stream, args.config_steps, min(args.warmup, 5))
        torch.cuda.empty_cache()

    if not args.no_cpu_baseline:
        cb = cpu_baseline(w)
        cb["cpu_model"] = cpu_model()
        out["cpu_baseline"] = cb
    print(json.dumps(out))


if __name__ == "__main__":
    main()
