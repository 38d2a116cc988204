"""Helpers shared by the GPU tests: run the HIP path on a Workload, compare
against the oracle at the stated tolerance, print what names the case."""
from __future__ import annotations

import numpy as np
import torch

from paper_2605_13433_amd import hstu

TOL = {torch.bfloat16: 2e-2, torch.float32: 1e-5}


def say(msg):
    print(msg, flush=True)


def to_dev(t):
    return None if t is None else t.contiguous().cuda()


def run_gpu(w, bwd=True):
    """Forward (and backward) of workload `w` through the C ABI; CPU f64 results."""
    q, k, v, u = (to_dev(x) for x in (w.q, w.k, w.v, w.u))
    off = to_dev(w.seq_offsets)
    pos, tw, ts = to_dev(w.pos_w), to_dev(w.time_w), to_dev(w.timestamps)
    plan = hstu.Plan(q, off, w.N, pos, tw, ts, w.num_buckets, backward=bwd)
    f = plan.forward(q, k, v, u, off)
    out = dict(o=f.o, y=f.y, mean=f.ln_mean, rstd=f.ln_rstd)
    if bwd:
        g = plan.backward(q, k, v, u, off, to_dev(w.dy))
        out.update(dq=g.dq, dk=g.dk, dv=g.dv, du=g.du, d_pos=g.d_pos_w, d_time=g.d_time_w)
    torch.cuda.synchronize()
    return {n: (None if t is None else t.detach().to("cpu", torch.float64).numpy())
            for n, t in out.items()}


def rel_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), "non-finite values in GPU output"
    if ref.size == 0:
        return 0.0
    scale = np.abs(ref).max()
    err = np.abs(got - ref).max()
    return float(err / scale) if scale > 0 else float(err)


def check(name, got, ref, tol):
    e = rel_err(got, ref)
    say(f"    {name:7s} max|gpu-ref|/max|ref| = {e:.3e} (tol {tol:g})")
    assert e <= tol, f"{name}: {e:.3e} > {tol:g}"
    return e


def rows_of(w, seqs):
    off = w.seq_offsets.numpy()
    return np.concatenate([np.arange(off[b], off[b + 1]) for b in seqs]).astype(np.int64)
