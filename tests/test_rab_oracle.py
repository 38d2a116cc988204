"""Pins of the standalone RAB oracle (CPU only): a hand-worked fixture, an
element-by-element brute force that uses the C oracle's bucket function, the
fused attention oracle reproduced by a dense attention that adds the
materialized bias (so the standalone layout and indexing follow the fused
operator's definition), finite differences of every parameter gradient, and
the sum rules."""
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import rab as R
from paper_2605_13433_amd import inputs

HERE = os.path.dirname(os.path.abspath(__file__))


def test_golden_fixture():
    g = json.load(open(os.path.join(HERE, "golden", "rab_tiny.json")))
    out = R.rab_fwd(g["seq_offsets"], g["N"], 1, pos_w=g["pos_w"], timestamps=g["timestamps"],
                    time_fn=g["time_fn"])
    assert np.allclose(out, g["rab"], rtol=0, atol=1e-14)
    d_pos, d_time, d_fn = R.rab_bwd(np.ones((1, 9)), g["seq_offsets"], g["N"], 1,
                                    has_pos=True, timestamps=g["timestamps"],
                                    time_fn=g["time_fn"])
    assert np.array_equal(d_pos, np.array(g["d_pos"], dtype=np.float64))
    assert d_time is None
    assert np.allclose(d_fn, g["d_time_fn"], rtol=1e-14, atol=0)


def _case(seed, lengths, H=2, N=None, nb=32):
    N = N or max(lengths)
    w = inputs.make_workload(lengths, H=H, d=8, N=N, dtype=torch.float64, seed=seed,
                             num_buckets=nb)
    rng = np.random.default_rng(seed)
    fn = np.stack([rng.normal(0, 0.5, H), rng.uniform(0.1, 1.5, H)], axis=1)
    return w, fn


def test_brute_force_tiny(oracle_lib):
    w, fn = _case(1, [3, 0, 5, 1], N=6, nb=9)
    w.timestamps = w.timestamps * 7 + 3 * torch.arange(w.T) ** 2     # wider gaps
    out = R.rab_fwd(w.seq_offsets, w.N, w.H, w.pos_w, w.time_w, w.timestamps, w.num_buckets, fn)
    off, ts = w.seq_offsets.tolist(), w.timestamps.tolist()
    pos, tw = w.pos_w.tolist(), w.time_w.tolist()
    k = 0
    for b in range(len(off) - 1):
        L = off[b + 1] - off[b]
        for i in range(L):
            for j in range(L):
                dt = ts[off[b] + i] - ts[off[b] + j]
                for h in range(w.H):
                    ref = (pos[h][j - i + w.N - 1]
                           + tw[h][oracle_lib.time_bucket(dt, w.num_buckets)]
                           + fn[h][0] * (1.0 + abs(dt)) ** (-fn[h][1]))
                    assert abs(out[h, k] - ref) <= 1e-13 * max(1.0, abs(ref))
                k += 1
    assert k == out.shape[1]


def test_bucket_matches_c_oracle(oracle_lib):
    rng = np.random.default_rng(0)
    deltas = np.concatenate([np.arange(-70, 70), rng.integers(-2 ** 40, 2 ** 40, 500),
                             [2 ** 31 - 1, -(2 ** 31), 2 ** 62]])
    for nb in (1, 32, 128):
        got = R.time_bucket(deltas, nb)
        ref = [oracle_lib.time_bucket(int(x), nb) for x in deltas]
        assert got.tolist() == ref


def test_dense_attention_with_materialized_bias(oracle_lib):
    """The fused oracle's output equals masked SiLU attention whose scores add
    the standalone bias tensor."""
    w, _ = _case(4, [9, 1, 14, 6], H=2, N=16, nb=40)
    ref = oracle_lib.fwd_workload(w)["o"]
    rab = R.rab_fwd(w.seq_offsets, w.N, w.H, w.pos_w, w.time_w, w.timestamps, w.num_buckets)
    sq = R.square_offsets(w.seq_offsets)
    off = w.seq_offsets.tolist()
    q, k, v = (t.double().numpy() for t in (w.q, w.k, w.v))
    o = np.zeros_like(ref)
    for b in range(len(off) - 1):
        L = off[b + 1] - off[b]
        for h in range(w.H):
            S = q[off[b]:off[b + 1], h] @ k[off[b]:off[b + 1], h].T
            S = S + rab[h, sq[b]:sq[b + 1]].reshape(L, L)
            A = S / (1.0 + np.exp(-S)) / w.N * np.tril(np.ones((L, L)))
            o[off[b]:off[b + 1], h] = A @ v[off[b]:off[b + 1], h]
    assert np.abs(o - ref).max() <= 1e-12 * np.abs(ref).max()


def test_finite_differences():
    w, fn = _case(5, [4, 7], H=2, N=8, nb=16)
    w.timestamps = w.timestamps * 3
    S = int(R.square_offsets(w.seq_offsets)[-1])
    G = np.random.default_rng(2).standard_normal((w.H, S))
    pos, tw = w.pos_w.double().numpy(), w.time_w.double().numpy()

    def loss(pos_, tw_, fn_):
        return float((R.rab_fwd(w.seq_offsets, w.N, w.H, pos_, tw_, w.timestamps,
                                w.num_buckets, fn_) * G).sum())
    d_pos, d_time, d_fn = R.rab_bwd(G, w.seq_offsets, w.N, w.H, True, True, w.timestamps,
                                    w.num_buckets, fn)
    h = 1e-6
    for name, base, grad in (("pos", pos, d_pos), ("time", tw, d_time), ("fn", fn, d_fn)):
        flat = base.reshape(-1)
        for ix in range(flat.size):
            p, m = flat.copy(), flat.copy()
            p[ix] += h
            m[ix] -= h
            args_p = {"pos": (p.reshape(base.shape), tw, fn), "time": (pos, p.reshape(base.shape), fn),
                      "fn": (pos, tw, p.reshape(base.shape))}[name]
            args_m = {"pos": (m.reshape(base.shape), tw, fn), "time": (pos, m.reshape(base.shape), fn),
                      "fn": (pos, tw, m.reshape(base.shape))}[name]
            fd = (loss(*args_p) - loss(*args_m)) / (2 * h)
            an = float(grad.reshape(-1)[ix])
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, ix, fd, an)


def test_sum_rules_and_special_cases():
    w, fn = _case(6, [12, 3, 20], H=3, N=24, nb=64)
    S = int(R.square_offsets(w.seq_offsets)[-1])
    G = np.random.default_rng(3).standard_normal((w.H, S))
    d_pos, d_time, _ = R.rab_bwd(G, w.seq_offsets, w.N, w.H, True, True, w.timestamps,
                                 w.num_buckets, None)
    assert np.allclose(d_pos.sum(1), G.sum(1)) and np.allclose(d_time.sum(1), G.sum(1))
    # beta = 0: the functional term is the constant a_h; a = 0: no term
    fn0 = np.stack([np.array([0.5, -1.0, 2.0]), np.zeros(3)], axis=1)
    out = R.rab_fwd(w.seq_offsets, w.N, w.H, timestamps=w.timestamps, time_fn=fn0)
    assert np.array_equal(out, np.repeat(fn0[:, :1], S, axis=1))
    fnz = np.stack([np.zeros(3), np.ones(3)], axis=1)
    assert not R.rab_fwd(w.seq_offsets, w.N, w.H, timestamps=w.timestamps, time_fn=fnz).any()
