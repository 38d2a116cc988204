"""Seeded synthetic workloads for jagged HSTU attention.

This module only draws random numbers and packs them; it holds none of the
attention arithmetic, so both the HIP path and the CPU oracle may consume what
it produces.

The paper measures its jagged fusion operators on KuaiRand-27K / Amazon-all
training runs (Sec. 4.1.1, Appendix A).  Those datasets are not used here;
instead each workload below draws sequence lengths from a long-tailed
distribution of the same character (most users short, a few very long), with
head geometry taken from the paper's model settings (8 heads x 128 for the
large/long variants, Appendix A "Parameter Settings").

Recipe (fixed, so every run of a given workload sees identical bits):
  * rng = numpy.random.default_rng(seed); draws happen in this order:
    lengths, timestamp gaps, q, k, v, u, pos_w, time_w, dy (and, for the
    layer workload, x, w1, w2).
  * lengths: "uniform" = integers uniform on [lo, hi]; "powerlaw" = pmf
    proportional to L**-alpha restricted to the integers of [lo, hi];
    "mix" = Bernoulli(p_long) per sequence, then uniform on the short or
    long range.
  * timestamps (int64): per sequence ts_0 = 0 and gaps 1 + floor(Exp(mean)),
    a Poisson-process clock, strictly increasing.
  * q, k, v, u, dy ~ N(0, 1) in float32, rounded once to the compute dtype
    (bf16 by round-to-nearest-even, or kept as float32).
  * pos_w [H, 2N-1] and time_w [H, num_buckets] ~ N(0, 0.1) in float32.
  * layer workload: x ~ N(0, 1); w1, w2 ~ N(0, 1/fan_in).
  * device workload (sizes whose inputs are too large to draw and move from
    the host): lengths and timestamps as above, then pos_w and time_w on the
    host; q, k, v, u, dy ~ N(0, 1) in float32 drawn on the GPU, in that
    order, by torch's Philox generator seeded with `seed`, rounded once to
    the compute dtype.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np
import torch

NUM_TIME_BUCKETS = 128
TIME_GAP_MEAN_S = 600.0
RAB_STD = 0.1

# The five workloads: sizes, length distributions, rab composition.
WORKLOADS = {
    1: dict(name="tiny_fp32_fwd_B4_H2_d32_N64", B=4, H=2, d=32, N=64,
            dtype="f32", lengths=("uniform", 1, 64), pos=True, time=False,
            bwd=False),
    2: dict(name="powerlaw1.2_B128_L16-512_H4_d64", B=128, H=4, d=64, N=512,
            dtype="bf16", lengths=("powerlaw", 1.2, 16, 512), pos=True,
            time=True, bwd=True),
    3: dict(name="longtail_B64_L32-2048_H8_d128", B=64, H=8, d=128, N=2048,
            dtype="bf16", lengths=("mix", 0.2, (32, 256), (256, 2048)),
            pos=True, time=True, bwd=True),
    4: dict(name="hstu_layer_B32_L64-4096_H4_d128_D512", B=32, H=4, d=128,
            N=4096, dtype="bf16", lengths=("powerlaw", 1.1, 64, 4096),
            pos=True, time=True, bwd=True, layer=True, D_model=512),
    5: dict(name="zipf1.05_B1024_L1-8192_H4_d64", B=1024, H=4, d=64, N=8192,
            dtype="bf16", lengths=("powerlaw", 1.05, 1, 8192), pos=True,
            time=False, bwd=True),
}


@dataclass
class Workload:
    """One batch of jagged inputs; tensors live on the CPU (q, k, v, u and dy
    on the GPU for a device workload)."""
    B: int
    H: int
    d: int
    N: int
    dtype: torch.dtype
    lengths: np.ndarray          # int64 [B]
    seq_offsets: torch.Tensor    # int64 [B+1]
    q: torch.Tensor              # [T, H, d]
    k: torch.Tensor
    v: torch.Tensor
    u: torch.Tensor
    dy: Optional[torch.Tensor]   # [T, H*d] or None
    pos_w: Optional[torch.Tensor]    # float32 [H, 2N-1]
    time_w: Optional[torch.Tensor]   # float32 [H, NB]
    timestamps: Optional[torch.Tensor]  # int64 [T]
    num_buckets: int = NUM_TIME_BUCKETS
    name: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def T(self) -> int:
        return int(self.seq_offsets[-1])

    @property
    def pairs(self) -> int:
        """Causal (i, j<=i) pairs per head, summed over sequences."""
        L = self.lengths.astype(np.int64)
        return int((L * (L + 1) // 2).sum())


def _draw_lengths(rng, B, spec):
    kind = spec[0]
    if kind == "uniform":
        lo, hi = spec[1], spec[2]
        return rng.integers(lo, hi + 1, size=B).astype(np.int64)
    if kind == "powerlaw":
        alpha, lo, hi = spec[1], spec[2], spec[3]
        support = np.arange(lo, hi + 1, dtype=np.float64)
        p = support ** (-alpha)
        p /= p.sum()
        return rng.choice(np.arange(lo, hi + 1), size=B, p=p).astype(np.int64)
    if kind == "mix":
        p_long, (slo, shi), (llo, lhi) = spec[1], spec[2], spec[3]
        is_long = rng.random(B) < p_long
        short = rng.integers(slo, shi + 1, size=B)
        long_ = rng.integers(llo, lhi + 1, size=B)
        return np.where(is_long, long_, short).astype(np.int64)
    raise ValueError(f"unknown length distribution {kind!r}")


def _normal(rng, shape, std=1.0):
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return x


def _to_dtype(x: np.ndarray, dtype: torch.dtype) -> torch.Tensor:
    t = torch.from_numpy(x)
    return t.to(dtype) if dtype != torch.float32 else t


def timestamps_for(rng, lengths: np.ndarray) -> np.ndarray:
    """Per-sequence Poisson-process clocks: ts_0 = 0, gaps 1 + floor(Exp)."""
    T = int(lengths.sum())
    gaps = 1 + np.floor(rng.exponential(TIME_GAP_MEAN_S, size=T)).astype(np.int64)
    ts = np.empty(T, dtype=np.int64)
    off = 0
    for L in lengths:
        L = int(L)
        if L:
            g = gaps[off:off + L].copy()
            g[0] = 0
            ts[off:off + L] = np.cumsum(g)
        off += L
    return ts


def make_workload(lengths, H, d, N, dtype=torch.bfloat16, pos=True, time=True,
                  bwd=True, seed=0, num_buckets=NUM_TIME_BUCKETS,
                  rab_std=RAB_STD, name="custom", layer_dim=None) -> Workload:
    """Inputs for explicit sequence lengths (the length draw is skipped)."""
    rng = np.random.default_rng(seed)
    lengths = np.asarray(lengths, dtype=np.int64)
    return _fill(rng, lengths, H, d, N, dtype, pos, time, bwd, num_buckets,
                 rab_std, name, layer_dim)


def _fill(rng, lengths, H, d, N, dtype, pos, time, bwd, num_buckets, rab_std,
          name, layer_dim):
    B = len(lengths)
    offsets = np.zeros(B + 1, dtype=np.int64)
    np.cumsum(lengths, out=offsets[1:])
    T = int(offsets[-1])
    ts = timestamps_for(rng, lengths)
    q = _to_dtype(_normal(rng, (T, H, d)), dtype)
    k = _to_dtype(_normal(rng, (T, H, d)), dtype)
    v = _to_dtype(_normal(rng, (T, H, d)), dtype)
    u = _to_dtype(_normal(rng, (T, H, d)), dtype)
    pos_w = torch.from_numpy(_normal(rng, (H, 2 * N - 1), rab_std)) if pos else None
    time_w = (torch.from_numpy(_normal(rng, (H, num_buckets), rab_std))
              if time else None)
    dy = _to_dtype(_normal(rng, (T, H * d)), dtype) if bwd else None
    extra = {}
    if layer_dim is not None:
        D = layer_dim
        extra["x"] = _to_dtype(_normal(rng, (T, D)), dtype)
        extra["w1"] = _to_dtype(_normal(rng, (D, 4 * H * d), 1.0 / np.sqrt(D)), dtype)
        extra["w2"] = _to_dtype(_normal(rng, (H * d, D), 1.0 / np.sqrt(H * d)), dtype)
        extra["dout"] = _to_dtype(_normal(rng, (T, D)), dtype) if bwd else None
    return Workload(B=B, H=H, d=d, N=N, dtype=dtype, lengths=lengths,
                    seq_offsets=torch.from_numpy(offsets), q=q, k=k, v=v, u=u,
                    dy=dy, pos_w=pos_w, time_w=time_w,
                    timestamps=torch.from_numpy(ts) if time else None,
                    num_buckets=num_buckets, name=name, extra=extra)


def workload(index: int, seed: Optional[int] = None) -> Workload:
    """Workload `index` (1..5) drawn with `seed` (default: the index)."""
    spec = WORKLOADS[index]
    seed = index if seed is None else seed
    rng = np.random.default_rng(seed)
    lengths = _draw_lengths(rng, spec["B"], spec["lengths"])
    dtype = torch.float32 if spec["dtype"] == "f32" else torch.bfloat16
    return _fill(rng, lengths, spec["H"], spec["d"], spec["N"], dtype,
                 spec["pos"], spec["time"], spec["bwd"], NUM_TIME_BUCKETS,
                 RAB_STD, spec["name"],
                 spec.get("D_model") if spec.get("layer") else None)


def device_workload(lengths, H, d, N, dtype=torch.bfloat16, seed=0,
                    num_buckets=NUM_TIME_BUCKETS, rab_std=RAB_STD, device="cuda",
                    name="device") -> Workload:
    """Inputs for explicit lengths with q, k, v, u and dy drawn on `device`
    (both biases; seq_offsets, timestamps and tables stay on the host)."""
    rng = np.random.default_rng(seed)
    lengths = np.asarray(lengths, dtype=np.int64)
    offsets = np.zeros(len(lengths) + 1, dtype=np.int64)
    np.cumsum(lengths, out=offsets[1:])
    T = int(offsets[-1])
    ts = timestamps_for(rng, lengths)
    pos_w = torch.from_numpy(_normal(rng, (H, 2 * N - 1), rab_std))
    time_w = torch.from_numpy(_normal(rng, (H, num_buckets), rab_std))
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)

    def draw(shape):
        x = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
        return x.to(dtype) if dtype != torch.float32 else x

    q, k, v, u = (draw((T, H, d)) for _ in range(4))
    dy = draw((T, H * d))
    return Workload(B=len(lengths), H=H, d=d, N=N, dtype=dtype, lengths=lengths,
                    seq_offsets=torch.from_numpy(offsets), q=q, k=k, v=v, u=u,
                    dy=dy, pos_w=pos_w, time_w=time_w,
                    timestamps=torch.from_numpy(ts), num_buckets=num_buckets,
                    name=name)


def prefix(w: Workload, seq: int, n: int) -> Workload:
    """The first `n` rows of sequence `seq` as a one-sequence batch on the
    host (same N, tables and absolute timestamps)."""
    start = int(w.seq_offsets[seq])
    n = min(int(n), int(w.lengths[seq]))
    rows = torch.arange(start, start + n, dtype=torch.int64)
    pick = lambda t: None if t is None else t.index_select(0, rows.to(t.device)).cpu()
    return Workload(B=1, H=w.H, d=w.d, N=w.N, dtype=w.dtype,
                    lengths=np.array([n], dtype=np.int64),
                    seq_offsets=torch.tensor([0, n], dtype=torch.int64),
                    q=pick(w.q), k=pick(w.k), v=pick(w.v), u=pick(w.u),
                    dy=pick(w.dy), pos_w=w.pos_w, time_w=w.time_w,
                    timestamps=pick(w.timestamps), num_buckets=w.num_buckets,
                    name=w.name + "[prefix]")


def subset(w: Workload, seqs) -> Workload:
    """The sub-batch made of sequences `seqs` (same N, tables and bits), on
    the host whatever device `w`'s tensors live on."""
    seqs = np.asarray(seqs, dtype=np.int64)
    off = w.seq_offsets.numpy()
    rows = np.concatenate([np.arange(off[b], off[b + 1]) for b in seqs]) \
        if len(seqs) else np.zeros(0, dtype=np.int64)
    rows_t = torch.from_numpy(rows)
    lengths = w.lengths[seqs]
    offsets = np.zeros(len(seqs) + 1, dtype=np.int64)
    np.cumsum(lengths, out=offsets[1:])
    pick = lambda t: None if t is None else t.index_select(0, rows_t.to(t.device)).cpu()
    extra = {}
    if "x" in w.extra:   # layer inputs: token rows follow, weights are shared
        extra = dict(x=pick(w.extra["x"]), w1=w.extra["w1"], w2=w.extra["w2"],
                     dout=pick(w.extra.get("dout")))
    return Workload(B=len(seqs), H=w.H, d=w.d, N=w.N, dtype=w.dtype,
                    lengths=lengths, seq_offsets=torch.from_numpy(offsets),
                    q=pick(w.q), k=pick(w.k), v=pick(w.v), u=pick(w.u),
                    dy=pick(w.dy), pos_w=w.pos_w, time_w=w.time_w,
                    timestamps=pick(w.timestamps), num_buckets=w.num_buckets,
                    name=w.name + "[subset]", extra=extra)
