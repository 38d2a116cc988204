"""CPU oracle of the jagged multi-table embedding lookup (paper Sec. 4.1.2,
"Jagged Embedding Lookup Acceleration").

TEST INFRASTRUCTURE ONLY: only tests, the smoke check and the benchmark's
CPU-baseline leg may import this module.  The HIP library never does, and
this module imports nothing from it.

The paper describes the operator by what it avoids (padding ids, zero
checks, per-sample multi-table access) rather than by formulas; what it
computes is the plain definition of a non-pooled multi-table lookup over
explicit jagged indices, written out here in float64:

  * tables t = 0 .. F-1 are row ranges [row_offsets[t], row_offsets[t+1])
    of one weight matrix W [sum rows, D];
  * the ids of table t are ids[id_offsets[t] : id_offsets[t+1]] (explicit
    offsets, not lengths: no padding entries exist);
  * forward: the embedding of id position r of table t is
    W[row_offsets[t] + ids[r]]; an id outside [0, rows_t) is a contract
    violation and reads as a zero row;
  * backward: dW[g] = sum of dout[r] over every position r whose global row
    row_offsets[t] + ids[r] equals g (positions with invalid ids add
    nothing); only rows that some valid id touches are part of the result,
    returned as the ascending list of those rows with their sums.

Output layouts: "flat" puts position r at row r ([n, D], table-major, as the
ids); "token" requires every table to hold the same number T of ids and puts
position j of table t at row j, columns t*D .. t*D+D-1 ([T, F*D]: the
concatenated per-token embedding a sequence model consumes).
"""
from __future__ import annotations

import numpy as np


def _np(x, dtype):
    if hasattr(x, "detach"):
        import torch
        x = x.detach().cpu()
        if x.is_floating_point():
            x = x.to(torch.float64)
        x = x.numpy()
    return np.ascontiguousarray(x, dtype=dtype)


def _place(F, T_or_n, D, layout):
    if layout == "flat":
        return np.zeros((T_or_n, D), dtype=np.float64)
    return np.zeros((T_or_n, F * D), dtype=np.float64)


def _rows_source(weights):
    """The weight matrix without a float64 copy of every row (only the rows
    a lookup touches are upcast; bf16 -> float32 is exact)."""
    if hasattr(weights, "detach"):
        import torch
        w = weights.detach().cpu()
        return (w.float() if w.dtype == torch.bfloat16 else w).numpy()
    return np.asarray(weights)


def embedding_fwd(weights, row_offsets, ids, id_offsets, layout="flat"):
    """Forward lookup; returns float64 [n, D] (flat) or [T, F*D] (token)."""
    W = _rows_source(weights)
    ro = _np(row_offsets, np.int64)
    ids = _np(ids, np.int64)
    io = _np(id_offsets, np.int64)
    F, D = len(ro) - 1, W.shape[1]
    n = int(io[F])
    if layout == "token":
        counts = np.diff(io)
        assert F == 0 or (counts == counts[0]).all(), "token layout needs equal counts"
        out = _place(F, int(counts[0]) if F else 0, D, layout)
    else:
        out = _place(F, n, D, layout)
    for t in range(F):
        base, rows = int(ro[t]), int(ro[t + 1] - ro[t])
        seg = ids[io[t]:io[t + 1]]
        ok = (seg >= 0) & (seg < rows)
        vals = np.zeros((len(seg), D), dtype=np.float64)
        vals[ok] = W[base + seg[ok]].astype(np.float64)
        if layout == "flat":
            out[io[t]:io[t + 1]] = vals
        else:
            out[:, t * D:(t + 1) * D] = vals
    return out


def flat_rows(dout, id_offsets, layout="flat"):
    """The output gradient as float64 [n, D] rows in id order."""
    g = _np(dout, np.float64)
    io = _np(id_offsets, np.int64)
    if layout == "flat":
        return g
    F = len(io) - 1
    D = g.shape[1] // F
    return np.concatenate([g[:, t * D:(t + 1) * D] for t in range(F)], axis=0)


def embedding_bwd(dout, row_offsets, ids, id_offsets, layout="flat"):
    """Backward: (rows, grads) with rows the ascending global rows touched by
    a valid id (int64 [U]) and grads their summed gradients (float64 [U, D])."""
    ro = _np(row_offsets, np.int64)
    ids = _np(ids, np.int64)
    io = _np(id_offsets, np.int64)
    G = flat_rows(dout, io, layout)
    F = len(ro) - 1
    keys, pos = [], []
    for t in range(F):
        base, rows = int(ro[t]), int(ro[t + 1] - ro[t])
        seg = ids[io[t]:io[t + 1]]
        ok = (seg >= 0) & (seg < rows)
        keys.append(base + seg[ok])
        pos.append(np.arange(io[t], io[t + 1], dtype=np.int64)[ok])
    keys = np.concatenate(keys) if keys else np.zeros(0, dtype=np.int64)
    pos = np.concatenate(pos) if pos else np.zeros(0, dtype=np.int64)
    rows_u, inverse = np.unique(keys, return_inverse=True)
    grads = np.zeros((len(rows_u), G.shape[1]), dtype=np.float64)
    np.add.at(grads, inverse, G[pos])
    return rows_u.astype(np.int64), grads
