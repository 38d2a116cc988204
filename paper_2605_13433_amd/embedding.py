"""Python binding of the jagged embedding lookup C ABI
(include/hstu_embedding.h).

Argument marshalling only: the lookup and its backward run in the HIP
kernels of libhstu_jagged.so (the same library as the attention).  The
functions with the C names take device tensors and write into
caller-provided outputs; `lookup` / `lookup_backward` allocate outputs and
the workspace with torch and then call them.  Without the built library
every call raises: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import Optional

import torch

from . import hstu

HSTU_EMB_FLAT, HSTU_EMB_TOKEN = 0, 1
LAYOUTS = {"flat": HSTU_EMB_FLAT, "token": HSTU_EMB_TOKEN}


class EmbDesc(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int), ("num_tables", ctypes.c_int32),
                ("dim", ctypes.c_int32), ("row_offsets", ctypes.c_void_p),
                ("id_offsets", ctypes.c_void_p), ("total_rows", ctypes.c_int64),
                ("num_ids", ctypes.c_int64), ("layout", ctypes.c_int)]


_bound = False


def _lib():
    global _bound
    lib = hstu.load_library()
    if not _bound:
        P = ctypes.c_void_p
        D = ctypes.POINTER(EmbDesc)
        lib.hstu_jagged_embedding_fwd.argtypes = [D, P, P, P, P]
        lib.hstu_jagged_embedding_fwd.restype = ctypes.c_int
        lib.hstu_jagged_embedding_bwd_workspace_bytes.argtypes = [D]
        lib.hstu_jagged_embedding_bwd_workspace_bytes.restype = ctypes.c_size_t
        lib.hstu_jagged_embedding_bwd.argtypes = [D, P, P, P, P, P, P, ctypes.c_size_t, P]
        lib.hstu_jagged_embedding_bwd.restype = ctypes.c_int
        _bound = True
    return lib


def make_desc(dtype_code: int, row_offsets: torch.Tensor, id_offsets: torch.Tensor,
              dim: int, total_rows: int, num_ids: int, layout: str = "flat") -> EmbDesc:
    """Descriptor for device offset tensors (the host sizes are passed in so
    that no device memory is read here)."""
    return EmbDesc(int(dtype_code), int(row_offsets.numel() - 1), int(dim),
                   hstu._ptr(row_offsets), hstu._ptr(id_offsets), int(total_rows),
                   int(num_ids), LAYOUTS[layout])


def hstu_jagged_embedding_fwd(desc: EmbDesc, weights, ids, out, stream=None) -> None:
    hstu._check(_lib().hstu_jagged_embedding_fwd(
        ctypes.byref(desc), hstu._ptr(weights), hstu._ptr(ids), hstu._ptr(out),
        hstu._stream(stream)))


def hstu_jagged_embedding_bwd_workspace_bytes(desc: EmbDesc) -> int:
    n = _lib().hstu_jagged_embedding_bwd_workspace_bytes(ctypes.byref(desc))
    if n == 0:
        raise hstu.HstuError(-1, hstu.last_error())
    return n


def hstu_jagged_embedding_bwd(desc: EmbDesc, ids, dout, grad_weights, unique_rows,
                              num_unique, workspace, stream=None) -> None:
    hstu._check(_lib().hstu_jagged_embedding_bwd(
        ctypes.byref(desc), hstu._ptr(ids), hstu._ptr(dout), hstu._ptr(grad_weights),
        hstu._ptr(unique_rows), hstu._ptr(num_unique), hstu._ptr(workspace),
        workspace.numel() if workspace is not None else 0, hstu._stream(stream)))


@dataclass
class EmbPlan:
    """Descriptor and backward workspace of one batch shape.  The plan holds
    the offset tensors whose device addresses the descriptor carries, so they
    live as long as the plan."""
    desc: EmbDesc
    workspace: Optional[torch.Tensor]
    out_shape: tuple
    row_offsets: torch.Tensor
    id_offsets: torch.Tensor


def plan(weights: torch.Tensor, row_offsets: torch.Tensor, id_offsets: torch.Tensor,
         total_rows: int, num_ids: int, layout: str = "flat",
         with_bwd: bool = True) -> EmbPlan:
    F = row_offsets.numel() - 1
    D = weights.shape[1]
    desc = make_desc(hstu._dtype_code(weights), row_offsets, id_offsets, D, total_rows,
                     num_ids, layout)
    ws = None
    if with_bwd and num_ids > 0:
        nbytes = hstu_jagged_embedding_bwd_workspace_bytes(desc)
        ws = torch.empty(nbytes, dtype=torch.uint8, device=weights.device)
    shape = (num_ids, D) if layout == "flat" else ((num_ids // F if F else 0), F * D)
    return EmbPlan(desc, ws, shape, row_offsets, id_offsets)


def lookup(p: EmbPlan, weights, ids, out=None, stream=None) -> torch.Tensor:
    if out is None:
        out = torch.empty(p.out_shape, dtype=weights.dtype, device=weights.device)
    hstu_jagged_embedding_fwd(p.desc, weights, ids, out, stream)
    return out


def lookup_backward(p: EmbPlan, ids, dout, grad_weights, unique_rows=None,
                    num_unique=None, stream=None) -> None:
    hstu_jagged_embedding_bwd(p.desc, ids, dout, grad_weights, unique_rows, num_unique,
                              p.workspace, stream)
