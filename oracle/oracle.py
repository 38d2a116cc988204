"""ctypes wrapper for the CPU oracle (libhstu_oracle.so).

TEST INFRASTRUCTURE ONLY: only tests, the smoke check and the benchmark's
CPU-baseline leg may import this module.  The HIP library never does, and
this module imports nothing from it.

Inputs are numpy arrays or CPU torch tensors of any float dtype; they are
upcast exactly to float64 before the call.  Outputs are float64 numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "hstu_oracle.c")
LIB = os.path.join(HERE, "libhstu_oracle.so")
EPS = 1e-6

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (strict IEEE double: no fast-math)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC",
                               "-shared", SRC, "-o", tmp, "-lm"])
        os.replace(tmp, LIB)
    return LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build(force=True)
        lib = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        lib.hstu_oracle_time_bucket.argtypes = [i64, i32]
        lib.hstu_oracle_time_bucket.restype = ctypes.c_int
        lib.hstu_oracle_fwd.argtypes = [P, P, P, P, P, i32, i32, i32, i32, P, P,
                                        P, i32, f64, f64, P, P, P, P]
        lib.hstu_oracle_fwd.restype = ctypes.c_int
        lib.hstu_oracle_bwd.argtypes = [P, P, P, P, P, i32, i32, i32, i32, P, P,
                                        P, i32, f64, f64, P, P, P, P, P, P, P]
        lib.hstu_oracle_bwd.restype = ctypes.c_int
        lib.hstu_oracle_num_threads.argtypes = []
        lib.hstu_oracle_num_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def _f64(x):
    if x is None:
        return None
    if hasattr(x, "detach"):          # torch tensor (CPU)
        import torch
        x = x.detach().to("cpu", torch.float64).numpy()
    return np.ascontiguousarray(x, dtype=np.float64)


def _i64(x):
    if x is None:
        return None
    if hasattr(x, "detach"):
        x = x.detach().cpu().numpy()
    return np.ascontiguousarray(x, dtype=np.int64)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def num_threads() -> int:
    return _load().hstu_oracle_num_threads()


def time_bucket(delta: int, num_buckets: int) -> int:
    return _load().hstu_oracle_time_bucket(int(delta), int(num_buckets))


def _common(q, k, v, u, seq_offsets, pos_w, time_w, timestamps):
    q, k, v, u = _f64(q), _f64(k), _f64(v), _f64(u)
    off = _i64(seq_offsets)
    T, H, d = q.shape
    for t in (k, v):
        assert t.shape == (T, H, d)
    u = u.reshape(T, H, d)
    return q, k, v, u, off, T, H, d, _f64(pos_w), _f64(time_w), _i64(timestamps)


def fwd(q, k, v, u, seq_offsets, max_len, pos_w=None, time_w=None,
        timestamps=None, num_buckets=128, eps=EPS, alpha=1.0):
    """Returns dict(o [T,H,d], y [T,H*d], mean [T], rstd [T])."""
    q, k, v, u, off, T, H, d, pos_w, time_w, ts = _common(
        q, k, v, u, seq_offsets, pos_w, time_w, timestamps)
    B = len(off) - 1
    assert off[-1] == T
    o = np.zeros((T, H, d)); y = np.zeros((T, H * d))
    mean = np.zeros(T); rstd = np.zeros(T)
    rc = _load().hstu_oracle_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(u), _ptr(off),
                                 B, int(max_len), H, d, _ptr(pos_w), _ptr(time_w),
                                 _ptr(ts), int(num_buckets), float(eps), float(alpha),
                                 _ptr(o), _ptr(y), _ptr(mean), _ptr(rstd))
    if rc != 0:
        raise ValueError(f"hstu_oracle_fwd rejected its arguments (rc={rc})")
    return dict(o=o, y=y, mean=mean, rstd=rstd)


def bwd(q, k, v, u, seq_offsets, max_len, dy, pos_w=None, time_w=None,
        timestamps=None, num_buckets=128, eps=EPS, alpha=1.0):
    """Returns dict(dq, dk, dv [T,H,d], du [T,H*d], d_pos, d_time)."""
    q, k, v, u, off, T, H, d, pos_w, time_w, ts = _common(
        q, k, v, u, seq_offsets, pos_w, time_w, timestamps)
    B = len(off) - 1
    dy = _f64(dy).reshape(T, H * d)
    dq = np.zeros((T, H, d)); dk = np.zeros((T, H, d)); dv = np.zeros((T, H, d))
    du = np.zeros((T, H * d))
    N = int(max_len)
    d_pos = np.zeros((H, 2 * N - 1)) if pos_w is not None else None
    d_time = np.zeros((H, int(num_buckets))) if time_w is not None else None
    rc = _load().hstu_oracle_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(u), _ptr(off),
                                 B, N, H, d, _ptr(pos_w), _ptr(time_w), _ptr(ts),
                                 int(num_buckets), float(eps), float(alpha), _ptr(dy),
                                 _ptr(dq), _ptr(dk), _ptr(dv), _ptr(du),
                                 _ptr(d_pos), _ptr(d_time))
    if rc != 0:
        raise ValueError(f"hstu_oracle_bwd failed (rc={rc})")
    return dict(dq=dq, dk=dk, dv=dv, du=du, d_pos=d_pos, d_time=d_time)


def fwd_workload(w, eps=EPS, alpha=1.0):
    """Oracle forward on a paper_2605_13433_amd.inputs.Workload."""
    return fwd(w.q, w.k, w.v, w.u, w.seq_offsets, w.N, w.pos_w, w.time_w,
               w.timestamps, w.num_buckets, eps, alpha)


def bwd_workload(w, eps=EPS, alpha=1.0):
    return bwd(w.q, w.k, w.v, w.u, w.seq_offsets, w.N, w.dy, w.pos_w,
               w.time_w, w.timestamps, w.num_buckets, eps, alpha)
