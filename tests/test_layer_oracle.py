"""Pins of the HSTU layer-shell oracle (oracle/layer.py) against things other
than itself.

* an independent torch f64 formulation of the whole layer (padded dense
  attention from dense_ref, torch matmul / silu / split) whose gradients come
  from torch.autograd rather than the oracle's hand-written chain rule;
* central finite differences of sum(out * dout) along random directions in
  every input and parameter (x, w1, w2, both bias tables);
* the split order U, V, Q, K, fixed by zeroing one column block of w1 at a
  time: a zero V block gives o = 0 exactly, a zero U block gives y = 0 with
  o != 0, and a zero Q (K) block makes the output independent of the K (Q)
  block -- a permuted split fails at least one of these.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from paper_2605_13433_amd import inputs
from tests import dense_ref


@pytest.fixture(scope="module")
def layer_oracle(oracle_lib):
    from oracle import layer
    return layer


def _rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-300))


def _small(lengths=(5, 1, 9, 0), H=2, d=4, N=10, D=12, seed=3, pos=True, time=True):
    w = inputs.make_workload(list(lengths), H, d, N, dtype=torch.float64, pos=pos,
                             time=time, seed=seed, layer_dim=D)
    return w


def _torch_layer(w, params):
    """Dense torch f64 layer; params = dict(x, w1, w2, pos, time) leaves."""
    H, d = w.H, w.d
    C = H * d
    T = params["x"].shape[0]
    h = params["x"] @ params["w1"]
    z = F.silu(h)
    u, v, q, k = torch.split(z, C, dim=1)
    o, y = dense_ref.forward(q.reshape(T, H, d), k.reshape(T, H, d),
                             v.reshape(T, H, d), u.reshape(T, H, d),
                             w.seq_offsets.tolist(), w.N, params.get("pos"),
                             params.get("time"), w.timestamps, w.num_buckets)
    return h, o, y, y @ params["w2"]


def _leaves(w):
    e = w.extra
    p = dict(x=e["x"], w1=e["w1"], w2=e["w2"], pos=w.pos_w, time=w.time_w)
    return {k: (None if t is None else t.detach().clone().to(torch.float64).requires_grad_(True))
            for k, t in p.items()}


@pytest.mark.parametrize("pos,time", [(True, True), (True, False), (False, True)])
def test_layer_oracle_matches_dense_autograd(layer_oracle, pos, time):
    w = _small(pos=pos, time=time)
    p = _leaves(w)
    h, o, y, out = _torch_layer(w, p)
    (out * w.extra["dout"]).sum().backward()
    g = layer_oracle.layer_bwd_workload(w)
    f = g["fwd"]
    assert _rel(f["h"], h.detach()) < 1e-13
    assert _rel(f["o"], o.detach()) < 1e-12
    assert _rel(f["y"], y.detach()) < 1e-12
    assert _rel(f["out"], out.detach()) < 1e-12
    assert _rel(g["dx"], p["x"].grad) < 1e-10
    assert _rel(g["dw1"], p["w1"].grad) < 1e-10
    assert _rel(g["dw2"], p["w2"].grad) < 1e-10
    if pos:
        assert _rel(g["d_pos"], p["pos"].grad) < 1e-10
    if time:
        assert _rel(g["d_time"], p["time"].grad) < 1e-10


def test_layer_oracle_finite_differences(layer_oracle):
    w = _small(lengths=(4, 6, 1), H=2, d=4, N=8, D=8, seed=11)
    e = w.extra
    base = dict(x=e["x"].numpy(), w1=e["w1"].numpy(), w2=e["w2"].numpy(),
                pos=w.pos_w.numpy(), time=w.time_w.numpy())
    dout = e["dout"].numpy()

    def loss(p):
        f = layer_oracle.layer_fwd(p["x"], p["w1"], p["w2"], w.seq_offsets, w.N, w.H,
                                   w.d, p["pos"], p["time"], w.timestamps, w.num_buckets)
        return float((f["out"] * dout).sum())

    g = layer_oracle.layer_bwd(base["x"], base["w1"], base["w2"], w.seq_offsets, w.N,
                               w.H, w.d, dout, base["pos"], base["time"], w.timestamps,
                               w.num_buckets)
    grads = dict(x=g["dx"], w1=g["dw1"], w2=g["dw2"], pos=g["d_pos"], time=g["d_time"])
    rng = np.random.default_rng(5)
    eps = 1e-6
    for name in base:
        for _ in range(2):
            dirn = rng.standard_normal(base[name].shape)
            plus = dict(base); plus[name] = base[name] + eps * dirn
            minus = dict(base); minus[name] = base[name] - eps * dirn
            fd = (loss(plus) - loss(minus)) / (2 * eps)
            an = float((grads[name] * dirn).sum())
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, fd, an)


def test_layer_oracle_split_order(layer_oracle):
    w = _small(lengths=(7, 3), H=2, d=4, N=8, D=8, seed=21)
    e = w.extra
    C = w.H * w.d
    x, w1, w2 = e["x"].numpy(), e["w1"].numpy().copy(), e["w2"].numpy()

    def run(w1m):
        return layer_oracle.layer_fwd(x, w1m, w2, w.seq_offsets, w.N, w.H, w.d,
                                      w.pos_w, w.time_w, w.timestamps, w.num_buckets)

    def zero(block, m=None):
        m = (w1 if m is None else m).copy()
        m[:, block * C:(block + 1) * C] = 0.0
        return m

    full = run(w1)
    assert np.abs(full["o"]).max() > 0 and np.abs(full["y"]).max() > 0
    # block 1 is V: silu(0) = 0 -> v = 0 -> o = 0 exactly
    f = run(zero(1))
    assert np.abs(f["o"]).max() == 0.0 and np.abs(f["out"]).max() == 0.0
    # block 0 is U: y = LN(o) * 0 = 0, o unchanged
    f = run(zero(0))
    assert np.abs(f["y"]).max() == 0.0 and np.array_equal(f["o"], full["o"])
    # block 2 is Q: with q = 0 the scores are the bias alone, so the K block
    # (3) no longer matters; symmetrically for a zero K block and Q
    rng = np.random.default_rng(0)
    for zb, other in ((2, 3), (3, 2)):
        a = zero(zb)
        b = a.copy()
        b[:, other * C:(other + 1) * C] = rng.standard_normal((w1.shape[0], C))
        assert np.array_equal(run(a)["out"], run(b)["out"])
        # ... while the same change with the block present does matter
        c = w1.copy()
        c[:, other * C:(other + 1) * C] = b[:, other * C:(other + 1) * C]
        assert not np.allclose(run(c)["out"], full["out"])
