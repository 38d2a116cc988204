"""Seeded synthetic inputs for the jagged multi-table embedding lookup.

Like `inputs.py`, this module only draws random numbers and packs them; it
holds none of the lookup's arithmetic, so both the HIP path and the CPU
oracle consume what it produces.

The paper measures its jagged embedding lookup (Sec. 4.1.2) on a batch of
about one million indices of which half are padding zeros, from a
multi-table sequence model on KuaiRand-27K.  That dataset is not used.  The
stand-in keeps the shape: F = 8 feature tables whose sizes span hot (128
rows) to cold (4 M rows), B = 32 sequences with lengths uniform on
[1, 4160] (so the padded batch F * B * 4160 = 1 064 960 indices is about
half padding), one id per token and table, ids drawn from a power law over
each table's rows (a few hot rows, a long cold tail).

Recipe (fixed, so every run of a given seed sees identical bits):
  * rng = numpy.random.default_rng(seed); draws in this order: lengths,
    then per table its ranks, then weights, then the output gradient.
  * ranks: pmf proportional to (r + 1) ** -alpha restricted to [0, rows);
    the id of rank r is (r * 2654435761) mod rows (rows a power of two, so
    hot ranks land on scattered rows, as in a hashed id space).
  * weights [sum rows, D] and dout ~ N(0, 1) in float32, rounded once to the
    compute dtype (bf16 by round-to-nearest-even, or kept as float32).
  * ids are grouped table-major (all ids of table 0, then table 1, ...),
    each table's ids in token order; id_offsets[t] is where table t starts.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np
import torch

EMB_ROWS = (1 << 22, 1 << 20, 1 << 18, 1 << 16, 1 << 14, 1 << 12, 1 << 10, 1 << 7)
EMB_DIM = 128
EMB_B = 32
EMB_MAX_LEN = 4160
EMB_ALPHA = 1.05
HASH_MUL = 2654435761


@dataclass
class EmbeddingBatch:
    """One multi-table lookup batch; tensors live on the CPU."""
    rows: np.ndarray            # int64 [F] rows per table
    row_offsets: torch.Tensor   # int64 [F+1] first row of each table in `weights`
    weights: torch.Tensor       # [sum rows, D]
    ids: torch.Tensor           # int64 [n], table-major
    id_offsets: torch.Tensor    # int64 [F+1]
    dout: Optional[torch.Tensor]  # [n, D] in the flat layout (row r <-> ids[r])
    lengths: np.ndarray         # int64 [B] tokens per sequence (token layout)
    D: int
    dtype: torch.dtype
    name: str = ""

    @property
    def F(self) -> int:
        return len(self.rows)

    @property
    def n(self) -> int:
        return int(self.id_offsets[-1])

    @property
    def total_rows(self) -> int:
        return int(self.row_offsets[-1])


def _to_dtype(x: np.ndarray, dtype: torch.dtype) -> torch.Tensor:
    t = torch.from_numpy(x)
    return t.to(dtype) if dtype != torch.float32 else t


def draw_ranks(rng, rows: int, count: int, alpha: float) -> np.ndarray:
    """`count` ranks from the power law (r + 1) ** -alpha on [0, rows)."""
    p = np.arange(1, rows + 1, dtype=np.float64) ** (-alpha)
    p /= p.sum()
    return rng.choice(rows, size=count, p=p).astype(np.int64)


def make_batch(rows: Sequence[int], counts: Sequence[int], D: int,
               dtype=torch.float32, seed: int = 0, alpha: float = EMB_ALPHA,
               lengths=None, with_dout: bool = True, ids=None,
               name: str = "custom") -> EmbeddingBatch:
    """A batch with `counts[t]` ids in table t (drawn unless `ids` is given)."""
    rng = np.random.default_rng(seed)
    rows = np.asarray(rows, dtype=np.int64)
    counts = np.asarray(counts, dtype=np.int64)
    F = len(rows)
    row_offsets = np.zeros(F + 1, dtype=np.int64)
    np.cumsum(rows, out=row_offsets[1:])
    id_offsets = np.zeros(F + 1, dtype=np.int64)
    np.cumsum(counts, out=id_offsets[1:])
    if ids is None:
        parts = []
        for t in range(F):
            r = draw_ranks(rng, int(rows[t]), int(counts[t]), alpha)
            parts.append((r * HASH_MUL) % rows[t])
        ids = np.concatenate(parts) if parts else np.zeros(0, dtype=np.int64)
    ids = np.asarray(ids, dtype=np.int64)
    assert len(ids) == id_offsets[-1]
    w = rng.standard_normal(size=(int(row_offsets[-1]), D), dtype=np.float32)
    dout = (rng.standard_normal(size=(len(ids), D), dtype=np.float32)
            if with_dout else None)
    return EmbeddingBatch(rows=rows, row_offsets=torch.from_numpy(row_offsets),
                          weights=_to_dtype(w, dtype), ids=torch.from_numpy(ids),
                          id_offsets=torch.from_numpy(id_offsets),
                          dout=None if dout is None else _to_dtype(dout, dtype),
                          lengths=np.asarray(lengths if lengths is not None else [],
                                             dtype=np.int64),
                          D=D, dtype=dtype, name=name)


def sequence_batch(seed: int = 6, rows: Sequence[int] = EMB_ROWS, D: int = EMB_DIM,
                   B: int = EMB_B, max_len: int = EMB_MAX_LEN, dtype=torch.float32,
                   alpha: float = EMB_ALPHA, with_dout: bool = True) -> EmbeddingBatch:
    """The sequence-feature workload: every token of every sequence has one
    id in each table, so each table holds T = sum of lengths ids."""
    rng = np.random.default_rng(seed)
    lengths = rng.integers(1, max_len + 1, size=B).astype(np.int64)
    T = int(lengths.sum())
    F = len(rows)
    ids = np.concatenate([(draw_ranks(rng, int(R), T, alpha) * HASH_MUL) % R
                          for R in rows])
    sub = int(rng.integers(0, 2 ** 31))      # weights/dout from their own stream
    name = f"emb_F{F}_B{B}_L1-{max_len}_D{D}_" + ("f32" if dtype == torch.float32 else "bf16")
    return make_batch(rows, [T] * F, D, dtype, seed=sub, alpha=alpha, lengths=lengths,
                      with_dout=with_dout, ids=ids, name=name)


def token_layout(x: torch.Tensor, F: int) -> torch.Tensor:
    """Flat [F*T, D] (table-major) -> token-major [T, F*D] (pure data movement)."""
    n, D = x.shape
    T = n // F
    return x.reshape(F, T, D).permute(1, 0, 2).reshape(T, F * D).contiguous()
