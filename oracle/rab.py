"""CPU oracle of the standalone relative attention bias (RAB) operator and
its backward (paper Sec. 4.1.1, the RAB half of "Jagged Fusion Operators for
Attention and RAB", and Appendix A for the time encodings).

TEST INFRASTRUCTURE ONLY: only tests, the smoke check and the benchmark's
CPU-baseline leg may import this module.  The HIP library never does, and
this module imports nothing from it.

The paper's fused operator takes relative time and position biases over
jagged sequences; this is the same bias produced on its own, as the jagged
tensor that an unfused attention would add to its scores (the memory the
fusion saves), with its backward into the bias parameters.  For sequence b
(rows off[b] .. off[b+1]-1, L = L_b), head h and local positions i, j < L:

    rab[h, sq[b] + i L + j] = pos_w[h, j - i + N - 1]          (if given)
                            + time_w[h, bucket(ts_i - ts_j)]    (table encoding)
                            + a_h (1 + |ts_i - ts_j|) ** -beta_h  (functional encoding)

with sq[b] = sum of L_b'^2 over b' < b: one L x L square per sequence, no
padding.  The bucket rule is the fused operator's (four log buckets per
octave, clamped to nb-1).  The functional time encoding is the library's
reading of the paper's "functional time encodings" of FuXi (Appendix A
names them without a formula): a per-head power-law decay of the bias with
the time gap, amplitude a_h and exponent beta_h as learnable parameters
(time_fn [H][2]).

Backward, given d_rab in the same layout: d_pos_w[h, x] and d_time_w[h, k]
sum d_rab over the entries with that offset / bucket; d_time_fn[h] =
(sum d_rab g, -sum d_rab a_h g ln(1 + |dt|)) with g = (1 + |dt|) ** -beta_h.
Every sum runs over all L x L entries of every sequence.  float64.
"""
from __future__ import annotations

import numpy as np


def _np(x, dtype):
    if x is None:
        return None
    if hasattr(x, "detach"):
        import torch
        x = x.detach().cpu()
        if x.is_floating_point():
            x = x.to(torch.float64)
        x = x.numpy()
    return np.ascontiguousarray(x, dtype=dtype)


def time_bucket(delta, nb):
    """The integer bucket rule on int64 arrays: |x| < 4 -> |x|; else with
    e = floor(log2 |x|) (by repeated halving), 4(e-1) + ((|x| >> (e-2)) & 3),
    clamped to nb - 1."""
    x = np.abs(np.asarray(delta, dtype=np.int64)).astype(np.uint64)
    e = np.zeros(x.shape, dtype=np.int64)
    while True:
        more = (x >> (e + 1).astype(np.uint64)) != 0
        if not more.any():
            break
        e += more
    m = ((x >> np.maximum(e - 2, 0).astype(np.uint64)) & np.uint64(3)).astype(np.int64)
    b = np.where(x < 4, x.astype(np.int64), 4 * (e - 1) + m)
    return np.minimum(b, nb - 1)


def square_offsets(seq_offsets):
    off = _np(seq_offsets, np.int64)
    L = np.diff(off)
    sq = np.zeros(len(L) + 1, dtype=np.int64)
    np.cumsum(L * L, out=sq[1:])
    return sq


def _blocks(seq_offsets, timestamps):
    off = _np(seq_offsets, np.int64)
    ts = _np(timestamps, np.int64)
    for b in range(len(off) - 1):
        L = int(off[b + 1] - off[b])
        i = np.arange(L)[:, None]
        j = np.arange(L)[None, :]
        dt = None if ts is None else ts[off[b] + i] - ts[off[b] + j]
        yield b, L, i, j, dt


def rab_fwd(seq_offsets, N, H, pos_w=None, time_w=None, timestamps=None,
            num_buckets=128, time_fn=None):
    """rab [H, sum L^2] float64."""
    pos_w, time_w, time_fn = _np(pos_w, np.float64), _np(time_w, np.float64), \
        _np(time_fn, np.float64)
    sq = square_offsets(seq_offsets)
    out = np.zeros((H, int(sq[-1])), dtype=np.float64)
    for b, L, i, j, dt in _blocks(seq_offsets, timestamps):
        blk = np.zeros((H, L, L))
        if pos_w is not None:
            blk += pos_w[:, (j - i + N - 1)]
        if time_w is not None:
            blk += time_w[:, time_bucket(dt, num_buckets)]
        if time_fn is not None:
            g = (1.0 + np.abs(dt).astype(np.float64))[None] ** (-time_fn[:, 1][:, None, None])
            blk += time_fn[:, 0][:, None, None] * g
        out[:, sq[b]:sq[b + 1]] = blk.reshape(H, L * L)
    return out


def rab_bwd(d_rab, seq_offsets, N, H, has_pos=True, has_time=False, timestamps=None,
            num_buckets=128, time_fn=None):
    """Gradients (d_pos [H, 2N-1] or None, d_time [H, nb] or None,
    d_time_fn [H, 2] or None); the tables' values do not enter their
    gradients, time_fn's do."""
    G = _np(d_rab, np.float64)
    time_fn = _np(time_fn, np.float64)
    sq = square_offsets(seq_offsets)
    d_pos = np.zeros((H, 2 * N - 1)) if has_pos else None
    d_time = np.zeros((H, num_buckets)) if has_time else None
    d_fn = np.zeros((H, 2)) if time_fn is not None else None
    for b, L, i, j, dt in _blocks(seq_offsets, timestamps):
        blk = G[:, sq[b]:sq[b + 1]].reshape(H, L, L)
        if d_pos is not None:
            idx = np.broadcast_to(j - i + N - 1, (L, L)).reshape(-1)
            for h in range(H):
                np.add.at(d_pos[h], idx, blk[h].reshape(-1))
        if d_time is not None:
            idx = time_bucket(dt, num_buckets).reshape(-1)
            for h in range(H):
                np.add.at(d_time[h], idx, blk[h].reshape(-1))
        if d_fn is not None:
            lg = np.log1p(np.abs(dt).astype(np.float64))
            for h in range(H):
                a, beta = time_fn[h]
                g = np.exp(-beta * lg)
                d_fn[h, 0] += float((blk[h] * g).sum())
                d_fn[h, 1] += float((blk[h] * (-a * g * lg)).sum())
    return d_pos, d_time, d_fn
