"""Python binding of the jagged HSTU attention C ABI (include/hstu_jagged.h),
including the HSTU layer shell calls.

Argument marshalling only: every step of the computation runs in the HIP
kernels of libhstu_jagged.so.  PyTorch supplies device memory and the
current stream.  The functions with the C names take device tensors and
write into caller-provided outputs; `forward` / `backward` are conveniences
that allocate the outputs and the workspace with torch and then call them.

If the shared library has not been built, every call raises: there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libhstu_jagged.so")

HSTU_BF16, HSTU_F32 = 0, 1
# seq_offsets status word bits (include/hstu_jagged.h)
HSTU_SEQ_FIRST_NOT_ZERO = 0x1
HSTU_SEQ_DECREASING = 0x2
HSTU_SEQ_TOO_LONG = 0x4
HSTU_SEQ_LAST_NOT_T = 0x8
HSTU_SEQ_UNCHECKED = 0x40000000
ERRORS = {-1: "HSTU_EINVAL", -2: "HSTU_ENOTSUP", -3: "HSTU_EWORKSPACE", -4: "HSTU_EHIP"}


class HstuError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


class Rab(ctypes.Structure):
    _fields_ = [("pos_w", ctypes.c_void_p), ("time_w", ctypes.c_void_p),
                ("timestamps", ctypes.c_void_p), ("num_buckets", ctypes.c_int32),
                ("alpha", ctypes.c_float)]


class FwdOut(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int), ("total_tokens", ctypes.c_int64),
                ("y", ctypes.c_void_p), ("o", ctypes.c_void_p),
                ("ln_mean", ctypes.c_void_p), ("ln_rstd", ctypes.c_void_p),
                ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t)]


class BwdIO(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int), ("total_tokens", ctypes.c_int64),
                ("dy", ctypes.c_void_p), ("o", ctypes.c_void_p),
                ("ln_mean", ctypes.c_void_p), ("ln_rstd", ctypes.c_void_p),
                ("dq", ctypes.c_void_p), ("dk", ctypes.c_void_p),
                ("dv", ctypes.c_void_p), ("du", ctypes.c_void_p),
                ("d_pos_w", ctypes.c_void_p), ("d_time_w", ctypes.c_void_p),
                ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t),
                ("deterministic", ctypes.c_int32)]


class RabParams(ctypes.Structure):
    _fields_ = [("pos_w", ctypes.c_void_p), ("time_w", ctypes.c_void_p),
                ("time_fn", ctypes.c_void_p), ("timestamps", ctypes.c_void_p),
                ("num_buckets", ctypes.c_int32)]


class LayerFwdOut(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int), ("total_tokens", ctypes.c_int64),
                ("out", ctypes.c_void_p), ("h", ctypes.c_void_p), ("z", ctypes.c_void_p),
                ("y", ctypes.c_void_p), ("o", ctypes.c_void_p),
                ("ln_mean", ctypes.c_void_p), ("ln_rstd", ctypes.c_void_p),
                ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t)]


class LayerBwdIO(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int), ("total_tokens", ctypes.c_int64),
                ("dout", ctypes.c_void_p), ("h", ctypes.c_void_p), ("z", ctypes.c_void_p),
                ("y", ctypes.c_void_p), ("o", ctypes.c_void_p),
                ("ln_mean", ctypes.c_void_p), ("ln_rstd", ctypes.c_void_p),
                ("dx", ctypes.c_void_p), ("dw1", ctypes.c_void_p), ("dw2", ctypes.c_void_p),
                ("d_pos_w", ctypes.c_void_p), ("d_time_w", ctypes.c_void_p),
                ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Loads libhstu_jagged.so; raises if it is missing (no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run __graft_entry__.build() "
                          "(or python paper_2605_13433_amd/build.py) first")
    lib = ctypes.CDLL(path)
    P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.hstu_jagged_attn_fwd.argtypes = [P, P, P, P, P, i32, i32, i32, i32,
                                         ctypes.POINTER(Rab), ctypes.POINTER(FwdOut), P]
    lib.hstu_jagged_attn_fwd.restype = ctypes.c_int
    lib.hstu_jagged_attn_fwd_noalloc.argtypes = [P, P, P, P, P, i32, i32, i32, i32,
                                                 ctypes.POINTER(Rab), ctypes.POINTER(FwdOut), P]
    lib.hstu_jagged_attn_fwd_noalloc.restype = ctypes.c_int
    lib.hstu_jagged_attn_bwd.argtypes = [P, P, P, P, P, i32, i32, i32, i32,
                                         ctypes.POINTER(Rab), ctypes.POINTER(BwdIO), P]
    lib.hstu_jagged_attn_bwd.restype = ctypes.c_int
    lib.hstu_jagged_attn_workspace_bytes.argtypes = [i32, i32, i32, i32, i64, i32,
                                                     ctypes.c_int, ctypes.POINTER(Rab)]
    lib.hstu_jagged_attn_workspace_bytes.restype = ctypes.c_size_t
    lib.hstu_jagged_schedule.argtypes = [P, i32, i32, i64, P, P, P, P, ctypes.c_size_t, P]
    lib.hstu_jagged_schedule.restype = ctypes.c_int
    lib.hstu_layer_fwd.argtypes = [P, P, P, P, i32, i32, i32, i32, i32,
                                   ctypes.POINTER(Rab), ctypes.POINTER(LayerFwdOut), P]
    lib.hstu_layer_fwd.restype = ctypes.c_int
    lib.hstu_layer_bwd.argtypes = [P, P, P, P, i32, i32, i32, i32, i32,
                                   ctypes.POINTER(Rab), ctypes.POINTER(LayerBwdIO), P]
    lib.hstu_layer_bwd.restype = ctypes.c_int
    lib.hstu_layer_workspace_bytes.argtypes = [i32, i32, i32, i32, i32, i64, i32,
                                               ctypes.c_int, ctypes.POINTER(Rab)]
    lib.hstu_layer_workspace_bytes.restype = ctypes.c_size_t
    RP = ctypes.POINTER(RabParams)
    lib.hstu_jagged_rab_workspace_bytes.argtypes = [i32, i32, i32, RP]
    lib.hstu_jagged_rab_workspace_bytes.restype = ctypes.c_size_t
    lib.hstu_jagged_rab_fwd.argtypes = [P, i32, i32, i32, i64, i64, RP, P, P,
                                        ctypes.c_size_t, P]
    lib.hstu_jagged_rab_fwd.restype = ctypes.c_int
    lib.hstu_jagged_rab_bwd.argtypes = [P, i32, i32, i32, i64, i64, RP, P, P, P, P, P,
                                        ctypes.c_size_t, P]
    lib.hstu_jagged_rab_bwd.restype = ctypes.c_int
    lib.hstu_jagged_status.argtypes = [P, P, P]
    lib.hstu_jagged_status.restype = ctypes.c_int
    lib.hstu_last_error.argtypes = []
    lib.hstu_last_error.restype = ctypes.c_char_p
    lib.hstu_version.argtypes = []
    lib.hstu_version.restype = ctypes.c_char_p
    _lib = lib
    return lib


def last_error() -> str:
    return load_library().hstu_last_error().decode()


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to the HIP library must be contiguous")
    return t.data_ptr()


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return HSTU_BF16
    if t.dtype == torch.float32:
        return HSTU_F32
    raise ValueError(f"unsupported dtype {t.dtype}")


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def make_rab(pos_w=None, time_w=None, timestamps=None, num_buckets=128,
             alpha=1.0) -> Rab:
    return Rab(_ptr(pos_w), _ptr(time_w), _ptr(timestamps),
               int(num_buckets) if time_w is not None else 0, float(alpha))


def _check(rc: int):
    if rc != 0:
        raise HstuError(rc, last_error())


def hstu_jagged_attn_workspace_bytes(B, max_len, H, d, total_tokens, for_bwd,
                                     dtype_code, rab: Optional[Rab] = None) -> int:
    n = load_library().hstu_jagged_attn_workspace_bytes(
        int(B), int(max_len), int(H), int(d), int(total_tokens), int(for_bwd),
        int(dtype_code), ctypes.byref(rab) if rab is not None else None)
    if n == 0:
        raise HstuError(-1, last_error())
    return n


def hstu_jagged_attn_fwd(q, k, v, u, seq_offsets, B, max_len, H, d,
                         rab: Optional[Rab], out: FwdOut, stream=None) -> None:
    _check(load_library().hstu_jagged_attn_fwd(
        _ptr(q), _ptr(k), _ptr(v), _ptr(u), _ptr(seq_offsets), int(B),
        int(max_len), int(H), int(d), ctypes.byref(rab) if rab is not None else None,
        ctypes.byref(out), _stream(stream)))


def hstu_jagged_attn_fwd_noalloc(q, k, v, u, seq_offsets, B, max_len, H, d,
                                 rab: Optional[Rab], out: FwdOut, stream=None) -> None:
    """As hstu_jagged_attn_fwd on the library's fixed per-GPU scratch
    (out.workspace is ignored)."""
    _check(load_library().hstu_jagged_attn_fwd_noalloc(
        _ptr(q), _ptr(k), _ptr(v), _ptr(u), _ptr(seq_offsets), int(B),
        int(max_len), int(H), int(d), ctypes.byref(rab) if rab is not None else None,
        ctypes.byref(out), _stream(stream)))


def hstu_jagged_attn_bwd(q, k, v, u, seq_offsets, B, max_len, H, d,
                         rab: Optional[Rab], io: BwdIO, stream=None) -> None:
    _check(load_library().hstu_jagged_attn_bwd(
        _ptr(q), _ptr(k), _ptr(v), _ptr(u), _ptr(seq_offsets), int(B),
        int(max_len), int(H), int(d), ctypes.byref(rab) if rab is not None else None,
        ctypes.byref(io), _stream(stream)))


def hstu_jagged_schedule(seq_offsets, B, max_len, total_tokens, n_entries, list_q,
                         list_k, workspace, stream=None) -> None:
    _check(load_library().hstu_jagged_schedule(
        _ptr(seq_offsets), int(B), int(max_len), int(total_tokens), _ptr(n_entries),
        _ptr(list_q), _ptr(list_k), _ptr(workspace), workspace.numel(), _stream(stream)))


def hstu_layer_workspace_bytes(B, max_len, H, d, d_model, total_tokens, for_bwd,
                               dtype_code, rab: Optional[Rab] = None) -> int:
    n = load_library().hstu_layer_workspace_bytes(
        int(B), int(max_len), int(H), int(d), int(d_model), int(total_tokens),
        int(for_bwd), int(dtype_code), ctypes.byref(rab) if rab is not None else None)
    if n == 0:
        raise HstuError(-1, last_error())
    return n


def hstu_layer_fwd(x, w1, w2, seq_offsets, B, max_len, H, d, d_model,
                   rab: Optional[Rab], out: LayerFwdOut, stream=None) -> None:
    _check(load_library().hstu_layer_fwd(
        _ptr(x), _ptr(w1), _ptr(w2), _ptr(seq_offsets), int(B), int(max_len), int(H),
        int(d), int(d_model), ctypes.byref(rab) if rab is not None else None,
        ctypes.byref(out), _stream(stream)))


def hstu_layer_bwd(x, w1, w2, seq_offsets, B, max_len, H, d, d_model,
                   rab: Optional[Rab], io: LayerBwdIO, stream=None) -> None:
    _check(load_library().hstu_layer_bwd(
        _ptr(x), _ptr(w1), _ptr(w2), _ptr(seq_offsets), int(B), int(max_len), int(H),
        int(d), int(d_model), ctypes.byref(rab) if rab is not None else None,
        ctypes.byref(io), _stream(stream)))


def hstu_jagged_status(workspace, status, stream=None) -> None:
    """Enqueues the copy of the seq_offsets status word of the last call that
    used `workspace` into `status` (an int32 tensor of one element)."""
    _check(load_library().hstu_jagged_status(_ptr(workspace), _ptr(status), _stream(stream)))


def hstu_jagged_rab_workspace_bytes(B, max_len, H, rp: RabParams) -> int:
    n = load_library().hstu_jagged_rab_workspace_bytes(int(B), int(max_len), int(H),
                                                        ctypes.byref(rp))
    if n == 0:
        raise HstuError(-1, last_error())
    return n


def hstu_jagged_rab_fwd(seq_offsets, B, max_len, H, total_tokens, total_square,
                        rp: RabParams, rab, workspace, stream=None) -> None:
    _check(load_library().hstu_jagged_rab_fwd(
        _ptr(seq_offsets), int(B), int(max_len), int(H), int(total_tokens),
        int(total_square), ctypes.byref(rp), _ptr(rab), _ptr(workspace), workspace.numel(),
        _stream(stream)))


def hstu_jagged_rab_bwd(seq_offsets, B, max_len, H, total_tokens, total_square,
                        rp: RabParams, d_rab, d_pos_w, d_time_w, d_time_fn, workspace,
                        stream=None) -> None:
    _check(load_library().hstu_jagged_rab_bwd(
        _ptr(seq_offsets), int(B), int(max_len), int(H), int(total_tokens),
        int(total_square), ctypes.byref(rp), _ptr(d_rab), _ptr(d_pos_w), _ptr(d_time_w),
        _ptr(d_time_fn), _ptr(workspace), workspace.numel(), _stream(stream)))


class RabPlan:
    """Standalone RAB: parameters, workspace and output of one batch; the
    caller passes the square size (sum of squared lengths) from its host copy
    of the lengths."""

    def __init__(self, seq_offsets, max_len, H, total_tokens, total_square, pos_w=None,
                 time_w=None, time_fn=None, timestamps=None, num_buckets=128):
        self.B = seq_offsets.numel() - 1
        self.N, self.H, self.T, self.S = int(max_len), int(H), int(total_tokens), \
            int(total_square)
        self.rp = RabParams(_ptr(pos_w), _ptr(time_w), _ptr(time_fn), _ptr(timestamps),
                            int(num_buckets) if time_w is not None else 0)
        self._keep = (seq_offsets, pos_w, time_w, time_fn, timestamps)
        dev = seq_offsets.device
        self.ws = _workspace(hstu_jagged_rab_workspace_bytes(self.B, self.N, self.H, self.rp),
                             dev)
        self.rab = torch.empty(self.H, self.S, dtype=torch.float32, device=dev)
        self.d_pos = (torch.empty(self.H, 2 * self.N - 1, dtype=torch.float32, device=dev)
                      if pos_w is not None else None)
        self.d_time = (torch.empty(self.H, num_buckets, dtype=torch.float32, device=dev)
                       if time_w is not None else None)
        self.d_fn = (torch.empty(self.H, 2, dtype=torch.float32, device=dev)
                     if time_fn is not None else None)

    def forward(self, stream=None):
        hstu_jagged_rab_fwd(self._keep[0], self.B, self.N, self.H, self.T, self.S, self.rp,
                            self.rab, self.ws, stream)
        return self.rab

    def backward(self, d_rab, stream=None):
        hstu_jagged_rab_bwd(self._keep[0], self.B, self.N, self.H, self.T, self.S, self.rp,
                            d_rab, self.d_pos, self.d_time, self.d_fn, self.ws, stream)
        return self.d_pos, self.d_time, self.d_fn


def max_entries(B: int, max_len: int, total_tokens: int) -> int:
    """Capacity of a work list: min(B*ceil(N/64), (T + 63B)/64)."""
    return min(B * ((max_len + 63) // 64), (total_tokens + 63 * B) // 64)


def schedule(seq_offsets, max_len, total_tokens):
    """Runs the device scheduler; returns (q_list, k_list) as int32 [E, 2] CPU tensors."""
    B = seq_offsets.numel() - 1
    dev = seq_offsets.device
    cap = max(max_entries(B, max_len, total_tokens), 1)
    ws = _workspace(hstu_jagged_attn_workspace_bytes(B, max_len, 1, 64, total_tokens, 1,
                                                     HSTU_F32, None), dev)
    n = torch.zeros(1, dtype=torch.int32, device=dev)
    lq = torch.full((cap, 2), -1, dtype=torch.int32, device=dev)
    lk = torch.full((cap, 2), -1, dtype=torch.int32, device=dev)
    hstu_jagged_schedule(seq_offsets, B, max_len, total_tokens, n, lq, lk, ws)
    E = int(n.item())
    return lq[:E].cpu(), lk[:E].cpu()


# ---------------------------------------------------------------- helpers
@dataclass
class FwdResult:
    y: torch.Tensor
    o: torch.Tensor
    ln_mean: torch.Tensor
    ln_rstd: torch.Tensor


@dataclass
class BwdResult:
    dq: torch.Tensor
    dk: torch.Tensor
    dv: torch.Tensor
    du: torch.Tensor
    d_pos_w: Optional[torch.Tensor]
    d_time_w: Optional[torch.Tensor]


def _workspace(nbytes: int, device) -> torch.Tensor:
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
    assert ws.data_ptr() % 256 == 0
    return ws


class Plan:
    """Outputs + workspace for one problem shape, allocated once and reused."""

    def __init__(self, q, seq_offsets, max_len, pos_w=None, time_w=None,
                 timestamps=None, num_buckets=128, backward=True, alpha=1.0,
                 deterministic=False):
        T, H, d = q.shape
        dev = q.device
        self.B = seq_offsets.numel() - 1
        self.N, self.H, self.d, self.T = int(max_len), H, d, T
        self.rab = make_rab(pos_w, time_w, timestamps, num_buckets, alpha)
        self._keep = (pos_w, time_w, timestamps)
        code = _dtype_code(q)
        self.fwd_ws = _workspace(hstu_jagged_attn_workspace_bytes(
            self.B, self.N, H, d, T, 0, code, self.rab), dev)
        self.y = torch.empty(T, H * d, dtype=q.dtype, device=dev)
        self.o = torch.empty(T, H, d, dtype=q.dtype, device=dev)
        self.mean = torch.empty(T, dtype=torch.float32, device=dev)
        self.rstd = torch.empty(T, dtype=torch.float32, device=dev)
        self.out = FwdOut(code, T, _ptr(self.y), _ptr(self.o), _ptr(self.mean),
                          _ptr(self.rstd), _ptr(self.fwd_ws), self.fwd_ws.numel())
        self.io = None
        if backward:
            self.bwd_ws = _workspace(hstu_jagged_attn_workspace_bytes(
                self.B, self.N, H, d, T, 1, code, self.rab), dev)
            self.dq = torch.empty(T, H, d, dtype=q.dtype, device=dev)
            self.dk = torch.empty_like(self.dq)
            self.dv = torch.empty_like(self.dq)
            self.du = torch.empty(T, H * d, dtype=q.dtype, device=dev)
            self.d_pos = (torch.empty(H, 2 * self.N - 1, dtype=torch.float32, device=dev)
                          if pos_w is not None else None)
            self.d_time = (torch.empty(H, num_buckets, dtype=torch.float32, device=dev)
                           if time_w is not None else None)
            self.io = BwdIO(code, T, None, _ptr(self.o), _ptr(self.mean), _ptr(self.rstd),
                            _ptr(self.dq), _ptr(self.dk), _ptr(self.dv), _ptr(self.du),
                            _ptr(self.d_pos), _ptr(self.d_time), _ptr(self.bwd_ws),
                            self.bwd_ws.numel(), 1 if deterministic else 0)

    def status(self, backward=False, stream=None) -> int:
        """The seq_offsets status word (HSTU_SEQ_* bits) of the last forward
        (or backward) call; waits for the stream."""
        st = torch.full((1,), -1, dtype=torch.int32, device=self.fwd_ws.device)
        hstu_jagged_status(self.bwd_ws if backward else self.fwd_ws, st, stream)
        return int(st.item())

    def forward(self, q, k, v, u, seq_offsets, stream=None) -> FwdResult:
        hstu_jagged_attn_fwd(q, k, v, u, seq_offsets, self.B, self.N, self.H, self.d,
                             self.rab, self.out, stream)
        return FwdResult(self.y, self.o, self.mean, self.rstd)

    def backward(self, q, k, v, u, seq_offsets, dy, stream=None) -> BwdResult:
        self.io.dy = _ptr(dy)
        self._dy = dy
        hstu_jagged_attn_bwd(q, k, v, u, seq_offsets, self.B, self.N, self.H, self.d,
                             self.rab, self.io, stream)
        return BwdResult(self.dq, self.dk, self.dv, self.du, self.d_pos, self.d_time)


def forward(q, k, v, u, seq_offsets, max_len, pos_w=None, time_w=None,
            timestamps=None, num_buckets=128, alpha=1.0) -> FwdResult:
    plan = Plan(q, seq_offsets, max_len, pos_w, time_w, timestamps, num_buckets,
                backward=False, alpha=alpha)
    return plan.forward(q, k, v, u, seq_offsets)


def forward_backward(q, k, v, u, seq_offsets, max_len, dy, pos_w=None, time_w=None,
                     timestamps=None, num_buckets=128, alpha=1.0, deterministic=False):
    plan = Plan(q, seq_offsets, max_len, pos_w, time_w, timestamps, num_buckets,
                alpha=alpha, deterministic=deterministic)
    f = plan.forward(q, k, v, u, seq_offsets)
    g = plan.backward(q, k, v, u, seq_offsets, dy)
    return f, g


# ------------------------------------------------------------ layer shell
@dataclass
class LayerFwdResult:
    out: torch.Tensor       # [T, d_model]
    h: torch.Tensor         # [T, 4*H*d]   x . w1
    z: torch.Tensor         # [4, T, H, d] silu(h) planes U, V, Q, K
    y: torch.Tensor         # [T, H*d]
    o: torch.Tensor         # [T, H, d]
    ln_mean: torch.Tensor
    ln_rstd: torch.Tensor


@dataclass
class LayerBwdResult:
    dx: torch.Tensor
    dw1: torch.Tensor
    dw2: torch.Tensor
    d_pos_w: Optional[torch.Tensor]
    d_time_w: Optional[torch.Tensor]


class LayerPlan:
    """Saved state, gradients and workspaces of one HSTU layer shape."""

    def __init__(self, x, seq_offsets, max_len, H, d, pos_w=None, time_w=None,
                 timestamps=None, num_buckets=128, backward=True):
        T, D = x.shape
        dev = x.device
        self.B = seq_offsets.numel() - 1
        self.N, self.H, self.d, self.D, self.T = int(max_len), int(H), int(d), int(D), T
        C = H * d
        self.rab = make_rab(pos_w, time_w, timestamps, num_buckets)
        self._keep = (pos_w, time_w, timestamps)
        code = _dtype_code(x)
        self.fwd_ws = _workspace(hstu_layer_workspace_bytes(
            self.B, self.N, H, d, D, T, 0, code, self.rab), dev)
        bf = dict(dtype=x.dtype, device=dev)
        self.res = LayerFwdResult(
            out=torch.empty(T, D, **bf), h=torch.empty(T, 4 * C, **bf),
            z=torch.empty(4, T, H, d, **bf), y=torch.empty(T, C, **bf),
            o=torch.empty(T, H, d, **bf),
            ln_mean=torch.empty(T, dtype=torch.float32, device=dev),
            ln_rstd=torch.empty(T, dtype=torch.float32, device=dev))
        r = self.res
        self.out = LayerFwdOut(code, T, _ptr(r.out), _ptr(r.h), _ptr(r.z), _ptr(r.y),
                               _ptr(r.o), _ptr(r.ln_mean), _ptr(r.ln_rstd),
                               _ptr(self.fwd_ws), self.fwd_ws.numel())
        self.io = None
        if backward:
            self.bwd_ws = _workspace(hstu_layer_workspace_bytes(
                self.B, self.N, H, d, D, T, 1, code, self.rab), dev)
            self.grad = LayerBwdResult(
                dx=torch.empty(T, D, **bf), dw1=torch.empty(D, 4 * C, **bf),
                dw2=torch.empty(C, D, **bf),
                d_pos_w=(torch.empty(H, 2 * self.N - 1, dtype=torch.float32, device=dev)
                         if pos_w is not None else None),
                d_time_w=(torch.empty(H, num_buckets, dtype=torch.float32, device=dev)
                          if time_w is not None else None))
            g = self.grad
            self.io = LayerBwdIO(code, T, None, _ptr(r.h), _ptr(r.z), _ptr(r.y), _ptr(r.o),
                                 _ptr(r.ln_mean), _ptr(r.ln_rstd), _ptr(g.dx), _ptr(g.dw1),
                                 _ptr(g.dw2), _ptr(g.d_pos_w), _ptr(g.d_time_w),
                                 _ptr(self.bwd_ws), self.bwd_ws.numel())

    def forward(self, x, w1, w2, seq_offsets, stream=None) -> LayerFwdResult:
        hstu_layer_fwd(x, w1, w2, seq_offsets, self.B, self.N, self.H, self.d, self.D,
                       self.rab, self.out, stream)
        return self.res

    def backward(self, x, w1, w2, seq_offsets, dout, stream=None) -> LayerBwdResult:
        self.io.dout = _ptr(dout)
        self._dout = dout
        hstu_layer_bwd(x, w1, w2, seq_offsets, self.B, self.N, self.H, self.d, self.D,
                       self.rab, self.io, stream)
        return self.grad
