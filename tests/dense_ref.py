"""Independent padded-dense formulation of jagged HSTU attention (torch f64).

Used only to pin the CPU oracle: it pads every sequence to max_len, builds
the full score matrix with a batched matmul, applies the bias through index
gathers and the causal/validity mask as a matrix, normalises with
torch.nn.functional.layer_norm, and takes gradients with torch.autograd.
Nothing here is shared with the oracle or with the HIP path.
"""
from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as F


def time_bucket_frexp(delta: np.ndarray, num_buckets: int) -> np.ndarray:
    """Bucket rule written via frexp: x = f * 2**E, f in [0.5, 1).

    For x >= 4 the bucket is 4*(e-1) + floor(4*(x/2**e - 1)) with e = E-1,
    i.e. four equal-width buckets per octave; below 4 it is x itself.
    Exact in float64 for |delta| < 2**53.
    """
    x = np.abs(np.asarray(delta, dtype=np.int64)).astype(np.float64)
    f, E = np.frexp(x)
    e = E - 1
    frac = np.ldexp(x, -e) - 1.0                     # in [0, 1)
    big = 4 * (e - 1) + np.floor(4.0 * frac).astype(np.int64)
    out = np.where(x < 4, x.astype(np.int64), big)
    return np.minimum(out, num_buckets - 1)


def _pad(x, off, N):
    """[T, ...] -> [B, N, ...] zero padded, plus the validity mask [B, N]."""
    B = len(off) - 1
    out = x.new_zeros((B, N) + tuple(x.shape[1:]))
    valid = torch.zeros(B, N, dtype=torch.bool)
    for b in range(B):
        L = int(off[b + 1] - off[b])
        out[b, :L] = x[off[b]:off[b + 1]]
        valid[b, :L] = True
    return out, valid


def _unpad(x, off):
    return torch.cat([x[b, :int(off[b + 1] - off[b])] for b in range(len(off) - 1)], 0)


def forward(q, k, v, u, seq_offsets, N, pos_w=None, time_w=None,
            timestamps=None, num_buckets=128, eps=1e-6, return_a=False):
    """All tensors float64 torch (q,k,v,u [T,H,d]); returns o [T,H,d], y [T,H*d]."""
    off = [int(x) for x in seq_offsets]
    T, H, d = q.shape
    qp, valid = _pad(q, off, N)
    kp, _ = _pad(k, off, N)
    vp, _ = _pad(v, off, N)
    # scores [B, H, N(i), N(j)]
    s = torch.matmul(qp.permute(0, 2, 1, 3), kp.permute(0, 2, 3, 1))
    idx_i = torch.arange(N).view(N, 1)
    idx_j = torch.arange(N).view(1, N)
    if pos_w is not None:
        rel = (idx_j - idx_i + N - 1)                  # [N, N]
        s = s + pos_w[:, rel].unsqueeze(0)             # [1, H, N, N]
    if time_w is not None:
        tsp, _ = _pad(timestamps.view(-1, 1).to(torch.int64), off, N)
        tsp = tsp.squeeze(-1).numpy()                  # [B, N]
        delta = tsp[:, :, None] - tsp[:, None, :]      # [B, i, j]
        bk = torch.from_numpy(time_bucket_frexp(delta, num_buckets))
        tb = time_w[:, bk]                             # [H, B, N, N]
        s = s + tb.permute(1, 0, 2, 3)
    causal = (idx_j <= idx_i)
    mask = causal.view(1, 1, N, N) & valid.view(-1, 1, N, 1) & valid.view(-1, 1, 1, N)
    a = torch.where(mask, F.silu(s), torch.zeros_like(s)) / N
    op = torch.matmul(a, vp.permute(0, 2, 1, 3))       # [B, H, N, d]
    o = _unpad(op.permute(0, 2, 1, 3), off)            # [T, H, d]
    z = o.reshape(T, H * d)
    y = F.layer_norm(z, (H * d,), eps=eps) * u.reshape(T, H * d)
    if return_a:
        return o, y, a, mask
    return o, y


def forward_backward(q, k, v, u, seq_offsets, N, dy, pos_w=None, time_w=None,
                     timestamps=None, num_buckets=128, eps=1e-6):
    """Autograd gradients of sum(y * dy) w.r.t. q, k, v, u and the tables."""
    leaves = {}
    def leaf(name, t):
        if t is None:
            return None
        t = t.detach().clone().to(torch.float64).requires_grad_(True)
        leaves[name] = t
        return t
    q_, k_, v_, u_ = leaf("q", q), leaf("k", k), leaf("v", v), leaf("u", u)
    pw, tw = leaf("pos", pos_w), leaf("time", time_w)
    o, y = forward(q_, k_, v_, u_, seq_offsets, N, pw, tw, timestamps,
                   num_buckets, eps)
    (y * dy.to(torch.float64).reshape(y.shape)).sum().backward()
    out = dict(o=o.detach(), y=y.detach(), dq=q_.grad, dk=k_.grad, dv=v_.grad,
               du=u_.grad.reshape(y.shape))
    out["d_pos"] = pw.grad if pw is not None else None
    out["d_time"] = tw.grad if tw is not None else None
    return out
