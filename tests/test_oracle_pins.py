"""Pins of the CPU oracle against things other than itself.

The paper prints no worked numbers for the attention operator, so the oracle
is pinned by: the bucket rule's hand-worked table, closed forms (one-token
sequences, zero input, the linear regime of SiLU), an independent padded
dense formulation in torch f64 with library LayerNorm and autograd, central
finite differences, exact causality / isolation properties, sum rules of the
table gradients and LayerNorm invariants.  Each is chosen so that a dropped
term, a flipped sign or index or a transposed operand fails at least one.
"""
import itertools
import os

import numpy as np
import pytest
import torch

from paper_2605_13433_amd import inputs
from tests import dense_ref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "time_buckets.txt")


def _t64(x):
    return None if x is None else x.detach().to(torch.float64)


def _dense(w, bwd=False):
    args = (_t64(w.q), _t64(w.k), _t64(w.v), _t64(w.u), w.seq_offsets.tolist(), w.N)
    kw = dict(pos_w=_t64(w.pos_w), time_w=_t64(w.time_w), timestamps=w.timestamps,
              num_buckets=w.num_buckets)
    if bwd:
        return dense_ref.forward_backward(*args, _t64(w.dy), **kw)
    o, y = dense_ref.forward(*args, **kw)
    return dict(o=o, y=y)


def _rel(a, b):
    a = np.asarray(a, dtype=np.float64); b = np.asarray(b, dtype=np.float64)
    scale = max(np.abs(b).max(), 1e-300) if b.size else 1.0
    return float(np.abs(a - b).max() / scale) if a.size else 0.0


# ---------------------------------------------------------------- P11 buckets
def test_bucket_golden_table(oracle_lib):
    rows = [l.split() for l in open(GOLDEN) if l.strip() and not l.startswith("#")]
    assert len(rows) > 20
    for delta, want in rows:
        assert oracle_lib.time_bucket(int(delta), 128) == int(want), delta


def test_bucket_frexp_formulation_agrees(oracle_lib):
    rng = np.random.default_rng(0)
    xs = np.concatenate([np.arange(0, 5000), rng.integers(0, 2**40, 5000),
                         2 ** np.arange(0, 50), 2 ** np.arange(2, 50) - 1])
    ref = dense_ref.time_bucket_frexp(xs, 128)
    got = np.array([oracle_lib.time_bucket(int(x), 128) for x in xs])
    assert np.array_equal(got, ref)


def test_bucket_monotone_four_per_octave(oracle_lib):
    prev = -1
    for x in range(0, 1 << 14):
        b = oracle_lib.time_bucket(x, 1000)
        assert b >= prev and b - prev <= 1
        prev = b
    for e in range(2, 40):          # every octave [2^e, 2^(e+1)) holds 4 buckets
        vals = {oracle_lib.time_bucket(x, 1000) for x in
                np.linspace(2**e, 2**(e + 1) - 1, 64).astype(np.int64)}
        assert vals == set(range(4 * (e - 1), 4 * (e - 1) + 4))
    assert oracle_lib.time_bucket(1 << 60, 7) == 6          # clamp


# ------------------------------------------------------------- P1 closed form
def test_single_token_sequences_closed_form(oracle_lib):
    N, H, d = 16, 1, 8
    w = inputs.make_workload([1, 1, 1], H=H, d=d, N=N, dtype=torch.float64, seed=3)
    r = oracle_lib.fwd_workload(w)
    q, k, v, u = (x.numpy() for x in (w.q, w.k, w.v, w.u))
    pw, tw = w.pos_w.double().numpy(), w.time_w.double().numpy()
    for t in range(3):
        s = q[t, 0] @ k[t, 0] + pw[0, N - 1] + tw[0, 0]
        a = s / (1 + np.exp(-s)) / N
        np.testing.assert_allclose(r["o"][t, 0], a * v[t, 0], rtol=1e-14, atol=0)
        # one head: LN(a v) = sign(a) LN(v) up to eps
        vv = v[t, 0]
        ln = (vv - vv.mean()) / np.sqrt(vv.var() + 1e-6 / a**2)
        np.testing.assert_allclose(r["y"][t], np.sign(a) * ln * u[t, 0], rtol=1e-9, atol=1e-12)


# -------------------------------------------------------- P2 one-hot readout
def test_one_hot_v_reads_out_every_weight(oracle_lib):
    L, N, H = 7, 8, 2
    d = 8
    w = inputs.make_workload([L, 5], H=H, d=d, N=N, dtype=torch.float64, seed=5)
    eye = torch.zeros(w.T, H, d, dtype=torch.float64)
    for b, (s, e) in enumerate(zip(w.seq_offsets[:-1].tolist(), w.seq_offsets[1:].tolist())):
        for j in range(e - s):
            eye[s + j, :, j] = 1.0
    w.v = eye
    r = oracle_lib.fwd_workload(w)
    _, _, a, mask = dense_ref.forward(_t64(w.q), _t64(w.k), w.v, _t64(w.u),
                                      w.seq_offsets.tolist(), N, _t64(w.pos_w),
                                      _t64(w.time_w), w.timestamps, w.num_buckets,
                                      return_a=True)
    off = w.seq_offsets.tolist()
    for b in range(2):
        Lb = off[b + 1] - off[b]
        got = r["o"][off[b]:off[b + 1], :, :Lb]           # [i, h, j] = a_ij
        want = a[b, :, :Lb, :Lb].permute(1, 0, 2).numpy()
        np.testing.assert_allclose(got, want, rtol=1e-13, atol=0)
        iu = np.triu_indices(Lb, 1)
        assert np.all(got[iu[0], :, iu[1]] == 0.0)       # strictly causal zeros


# -------------------------------------------------------- P3 linear regime
def test_linear_regime_is_masked_matmul(oracle_lib):
    # with every score near +40, silu(s) = s (1 - O(e^-40)): a textbook
    # masked matmul ((Q K^T + R) . M) V / N
    N, H, d = 12, 2, 4
    lengths = [9, 12, 3]
    w = inputs.make_workload(lengths, H=H, d=d, N=N, dtype=torch.float64, seed=9,
                             time=False)
    w.q = w.q * 0.3
    w.pos_w = 40.0 + torch.arange(2 * N - 1, dtype=torch.float32).repeat(H, 1) * 0.25
    r = oracle_lib.fwd_workload(w)
    off = w.seq_offsets.tolist()
    for b, Lb in enumerate(lengths):
        sl = slice(off[b], off[b + 1])
        for h in range(H):
            Q = w.q[sl, h].numpy(); K = w.k[sl, h].numpy(); V = w.v[sl, h].numpy()
            i = np.arange(Lb)[:, None]; j = np.arange(Lb)[None, :]
            R = w.pos_w[h].double().numpy()[j - i + N - 1]
            M = np.tril(np.ones((Lb, Lb)))
            want = ((Q @ K.T + R) * M) @ V / N
            np.testing.assert_allclose(r["o"][sl, h], want, rtol=1e-12, atol=1e-12)


# -------------------------------------------------------- P4 zero input
def test_zero_queries_and_bias(oracle_lib):
    N, H, d = 8, 2, 4
    lengths = [5, 3]
    w = inputs.make_workload(lengths, H=H, d=d, N=N, dtype=torch.float64, seed=2,
                             pos=False, time=False)
    w.q = torch.zeros_like(w.q)
    r = oracle_lib.fwd_workload(w)
    assert np.all(r["o"] == 0) and np.all(r["y"] == 0)
    g = oracle_lib.bwd_workload(w)
    assert np.all(g["dv"] == 0) and np.all(g["du"] == 0)
    # n = 0, rstd = 1/sqrt(eps): dO = (g - mean g)/sqrt(eps); dS = dA * 0.5 / N
    T = w.T
    gg = (w.dy.double() * w.u.double().reshape(T, -1)).numpy()
    dO = ((gg - gg.mean(1, keepdims=True)) / np.sqrt(1e-6)).reshape(T, H, d)
    off = w.seq_offsets.tolist()
    for b in range(2):
        sl = slice(off[b], off[b + 1])
        for h in range(H):
            V = w.v[sl, h].numpy(); K = w.k[sl, h].numpy(); D = dO[sl, h]
            dS = np.tril(D @ V.T) * 0.5 / N
            np.testing.assert_allclose(g["dq"][sl, h], dS @ K, rtol=1e-10, atol=1e-9)
            np.testing.assert_allclose(g["dk"][sl, h], dS.T @ (w.q[sl, h].numpy()),
                                       atol=0)


# ------------------------------------------------ P5 independent dense formulation
@pytest.mark.parametrize("seed,lengths,H,d,N,pos,time", [
    (0, [5, 1, 7, 3], 2, 4, 8, True, True),
    (1, [16, 9, 1, 12], 3, 8, 16, True, True),
    (2, [4, 0, 6], 1, 5, 6, True, False),
    (3, [10, 10], 2, 6, 10, False, True),
    (4, [13, 2, 0, 8], 2, 3, 16, False, False),
])
def test_oracle_matches_dense_autograd(oracle_lib, seed, lengths, H, d, N, pos, time):
    w = inputs.make_workload(lengths, H=H, d=d, N=N, dtype=torch.float64,
                             pos=pos, time=time, seed=seed)
    if time:   # spread timestamps over many buckets
        w.timestamps = w.timestamps * 97 + torch.arange(w.T) ** 3
    f = oracle_lib.fwd_workload(w)
    g = oracle_lib.bwd_workload(w)
    ref = _dense(w, bwd=True)
    assert _rel(f["o"], ref["o"]) < 1e-12
    assert _rel(f["y"], ref["y"]) < 1e-12
    for name in ("dq", "dk", "dv", "du"):
        assert _rel(g[name], ref[name]) < 1e-11, name
    if pos:
        assert _rel(g["d_pos"], ref["d_pos"]) < 1e-11
    if time:
        assert _rel(g["d_time"], ref["d_time"]) < 1e-11


# --------------------------------------------------- P12 brute force offsets
def test_all_tiny_offset_vectors(oracle_lib):
    N, H, d = 4, 1, 3
    count = 0
    for B in range(0, 4):
        for lengths in itertools.product(range(0, 5), repeat=B):
            w = inputs.make_workload(list(lengths), H=H, d=d, N=N,
                                     dtype=torch.float64, seed=count)
            f = oracle_lib.fwd_workload(w)
            if w.T:
                ref = _dense(w)
                assert _rel(f["o"], ref["o"]) < 1e-12
                assert _rel(f["y"], ref["y"]) < 1e-12
            count += 1
    assert count == 1 + 5 + 25 + 125


# ------------------------------------------------------ P8 finite differences
def test_finite_differences(oracle_lib):
    N, H, d = 8, 2, 4
    w = inputs.make_workload([5, 2, 6], H=H, d=d, N=N, dtype=torch.float64, seed=11)
    w.timestamps = w.timestamps * 13 + torch.arange(w.T) ** 2
    g = oracle_lib.bwd_workload(w)
    dy = w.dy.double().numpy()

    def loss(**over):
        kw = dict(q=w.q, k=w.k, v=w.v, u=w.u, pos_w=w.pos_w.double(),
                  time_w=w.time_w.double())
        kw.update(over)
        r = oracle_lib.fwd(kw["q"], kw["k"], kw["v"], kw["u"], w.seq_offsets, N,
                           kw["pos_w"], kw["time_w"], w.timestamps, w.num_buckets)
        return float((r["y"] * dy).sum())

    rng = np.random.default_rng(0)
    h = 1e-6
    checks = [("q", "dq"), ("k", "dk"), ("v", "dv"), ("u", "du"),
              ("pos_w", "d_pos"), ("time_w", "d_time")]
    for name, gname in checks:
        base = dict(q=w.q, k=w.k, v=w.v, u=w.u, pos_w=w.pos_w.double(),
                    time_w=w.time_w.double())[name].double().clone()
        grad = g[gname].reshape(base.shape)
        flat = base.view(-1)
        if name == "pos_w":
            idx = [N - 1, N - 2, N - 4, N - 6, 2 * N - 1 + N - 1, 2 * N - 1 + N - 3, N + 2]
        elif name == "time_w":
            nz = np.flatnonzero(np.abs(grad.reshape(-1)) > 0)
            idx = list(nz[:6]) + [127]
        else:
            idx = rng.choice(flat.numel(), size=8, replace=False)
        for ix in idx:
            p = flat.clone(); p[ix] += h
            m = flat.clone(); m[ix] -= h
            fd = (loss(**{name: p.view(base.shape)}) - loss(**{name: m.view(base.shape)})) / (2 * h)
            an = float(grad.reshape(-1)[ix])
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, ix, fd, an)


def test_directional_derivative_mid_size(oracle_lib):
    N, H, d = 32, 2, 8
    w = inputs.make_workload([30, 17, 32, 4], H=H, d=d, N=N, dtype=torch.float64, seed=12)
    g = oracle_lib.bwd_workload(w)
    dy = w.dy.double().numpy()
    rng = np.random.default_rng(1)
    dirs = {n: torch.from_numpy(rng.standard_normal(tuple(getattr(w, n).shape)))
            for n in ("q", "k", "v", "u", "pos_w", "time_w")}
    grads = dict(q="dq", k="dk", v="dv", u="du", pos_w="d_pos", time_w="d_time")
    an = sum(float((g[grads[n]].reshape(-1) * dirs[n].numpy().reshape(-1)).sum())
             for n in dirs)

    def at(t):
        x = {n: getattr(w, n).double() + t * dirs[n] for n in dirs}
        r = oracle_lib.fwd(x["q"], x["k"], x["v"], x["u"], w.seq_offsets, N,
                           x["pos_w"], x["time_w"], w.timestamps, w.num_buckets)
        return float((r["y"] * dy).sum())
    h = 1e-5
    fd = (at(h) - at(-h)) / (2 * h)
    assert abs(fd - an) <= 1e-6 * abs(an)


# ---------------------------------------------------------- P6 causality
def test_causality_bitwise(oracle_lib):
    N, H, d = 16, 2, 4
    w = inputs.make_workload([12, 9], H=H, d=d, N=N, dtype=torch.float64, seed=21)
    base = oracle_lib.fwd_workload(w)
    t = 5                               # perturb token 5 of sequence 0
    for name in ("q", "k", "v", "u"):
        x = getattr(w, name).clone(); x[t] += 1.0
        old = getattr(w, name); setattr(w, name, x)
        r = oracle_lib.fwd_workload(w)
        setattr(w, name, old)
        assert np.array_equal(r["o"][:t], base["o"][:t]), name
        assert np.array_equal(r["y"][:t], base["y"][:t]), name
        assert np.array_equal(r["o"][12:], base["o"][12:]), name   # other sequence
    ts = w.timestamps.clone(); ts[t:12] += 1000
    old = w.timestamps; w.timestamps = ts
    r = oracle_lib.fwd_workload(w); w.timestamps = old
    assert np.array_equal(r["o"][:t], base["o"][:t])


def test_prefix_rows_are_exact_on_their_own(oracle_lib):
    """o, y, dQ and dU of a sequence's first n rows depend on those rows
    alone (causality; LayerNorm is per row): the oracle on the prefix as a
    batch of its own, with the same N, gives them bit for bit.  dK and dV of
    those rows do not (later queries reach them).  This is the premise of
    the GPU check of the 65536-token batch, and it checks inputs.prefix."""
    N, H, d = 40, 2, 4
    w = inputs.make_workload([7, 33, 5], H=H, d=d, N=N, dtype=torch.float64, seed=23)
    full_f, full_b = oracle_lib.fwd_workload(w), oracle_lib.bwd_workload(w)
    off = w.seq_offsets.numpy()
    n = 20
    p = inputs.prefix(w, 1, n)
    assert p.lengths.tolist() == [n] and p.N == N
    pf, pb = oracle_lib.fwd_workload(p), oracle_lib.bwd_workload(p)
    r = slice(off[1], off[1] + n)
    for name in ("o", "y"):
        assert np.array_equal(pf[name], full_f[name][r]), name
    for name in ("dq", "du"):
        assert np.array_equal(pb[name], full_b[name][r]), name
    assert not np.allclose(pb["dk"], full_b["dk"][r])


def test_device_workload_recipe():
    """The device-drawn inputs (drawn here on the CPU generator): seeded and
    reproducible, the documented shapes and dtypes, per-sequence clocks
    strictly increasing from 0, and inputs.prefix of a whole sequence equal
    to inputs.subset of it."""
    kw = dict(H=2, d=8, N=70, seed=3, num_buckets=16, device="cpu")
    w = inputs.device_workload([5, 0, 70], **kw)
    w2 = inputs.device_workload([5, 0, 70], **kw)
    for n in ("q", "k", "v", "u", "dy", "pos_w", "time_w", "timestamps"):
        assert torch.equal(getattr(w, n), getattr(w2, n)), n
    assert w.q.shape == (75, 2, 8) and w.dy.shape == (75, 16) and w.q.dtype == torch.bfloat16
    assert w.pos_w.shape == (2, 139) and w.time_w.shape == (2, 16)
    ts, off = w.timestamps.numpy(), w.seq_offsets.numpy()
    for b in range(3):
        seg = ts[off[b]:off[b + 1]]
        if len(seg):
            assert seg[0] == 0 and np.all(np.diff(seg) > 0)
    p, sb = inputs.prefix(w, 2, 70), inputs.subset(w, [2])
    assert p.lengths.tolist() == sb.lengths.tolist() == [70]
    for n in ("q", "k", "v", "u", "dy", "timestamps", "seq_offsets"):
        assert torch.equal(getattr(p, n), getattr(sb, n)), n


# ------------------------------------------------- P7 isolation / permutation
def test_isolation_and_permutation(oracle_lib):
    N, H, d = 16, 2, 4
    lengths = [7, 16, 3, 11]
    w = inputs.make_workload(lengths, H=H, d=d, N=N, dtype=torch.float64, seed=31)
    f = oracle_lib.fwd_workload(w)
    g = oracle_lib.bwd_workload(w)
    perm = [2, 0, 3, 1]
    wp = inputs.subset(w, perm)
    fp = oracle_lib.fwd_workload(wp)
    gp = oracle_lib.bwd_workload(wp)
    off = w.seq_offsets.tolist(); offp = wp.seq_offsets.tolist()
    for newb, b in enumerate(perm):
        a, c = slice(off[b], off[b + 1]), slice(offp[newb], offp[newb + 1])
        for key in ("o", "y"):
            assert np.array_equal(f[key][a], fp[key][c])
        for key in ("dq", "dk", "dv", "du"):
            assert np.array_equal(g[key][a], gp[key][c])
    assert _rel(g["d_pos"], gp["d_pos"]) < 1e-13
    assert _rel(g["d_time"], gp["d_time"]) < 1e-13
    # splitting the batch: tables add up
    g1 = oracle_lib.bwd_workload(inputs.subset(w, [0, 1]))
    g2 = oracle_lib.bwd_workload(inputs.subset(w, [2, 3]))
    assert _rel(g1["d_pos"] + g2["d_pos"], g["d_pos"]) < 1e-13


# ------------------------------------------------------- P9 sum rules
def test_table_gradient_sum_rules(oracle_lib):
    N, H, d = 16, 2, 4
    w = inputs.make_workload([16, 5, 9], H=H, d=d, N=N, dtype=torch.float64, seed=41)
    g = oracle_lib.bwd_workload(w)
    # every dS lands once in each table
    np.testing.assert_allclose(g["d_pos"].sum(1), g["d_time"].sum(1), rtol=1e-12)
    # j - i + N - 1 >= N is unreachable under causality
    assert np.all(g["d_pos"][:, N:] == 0)
    # the diagonal entry of d_pos sums dS_ii, each of which is dA_ii silu'(s_ii)/N
    wq = inputs.make_workload([1] * 6, H=H, d=d, N=N, dtype=torch.float64, seed=42)
    gq = oracle_lib.bwd_workload(wq)
    assert np.all(gq["d_pos"][:, :N - 1] == 0)
    np.testing.assert_allclose(gq["d_pos"][:, N - 1], gq["d_time"][:, 0], rtol=1e-12)
    # single tokens: dq_i = dS_ii k_i, so dS_ii = <dq_i, k_i>/|k_i|^2 summed = d_pos
    dS = (gq["dq"] * wq.k.numpy()).sum(-1) / (wq.k.numpy() ** 2).sum(-1)
    np.testing.assert_allclose(dS.sum(0), gq["d_pos"][:, N - 1], rtol=1e-10)


# ------------------------------------------------------- P10 LayerNorm invariants
def test_layernorm_invariants(oracle_lib):
    N, H, d = 16, 4, 8
    w = inputs.make_workload([16, 7], H=H, d=d, N=N, dtype=torch.float64, seed=51)
    w.u = torch.ones_like(w.u)
    r = oracle_lib.fwd_workload(w)
    y = r["y"]
    np.testing.assert_allclose(y.mean(1), 0, atol=1e-12)
    z = r["o"].reshape(w.T, -1)
    var = z.var(1)
    np.testing.assert_allclose((y ** 2).mean(1), var / (var + 1e-6), rtol=1e-10)
    np.testing.assert_allclose(r["mean"], z.mean(1), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(r["rstd"], 1 / np.sqrt(var + 1e-6), rtol=1e-12)


def test_mistakes_are_caught(oracle_lib):
    """Planted mistakes in a copy of the computation fail the dense pin.

    The perturbations stand for plausible oracle bugs (mask off by one,
    reversed position index, missing 1/N); each makes the dense comparison
    fail, showing the pin has teeth."""
    N, H, d = 8, 2, 4
    w = inputs.make_workload([6, 8], H=H, d=d, N=N, dtype=torch.float64, seed=61)
    ref = _dense(w)["o"].numpy()
    f = oracle_lib.fwd_workload(w)
    assert _rel(f["o"], ref) < 1e-12
    # reversed position index: flip the table
    w2 = inputs.make_workload([6, 8], H=H, d=d, N=N, dtype=torch.float64, seed=61)
    w2.pos_w = torch.flip(w2.pos_w, dims=[1])
    assert _rel(oracle_lib.fwd_workload(w2)["o"], ref) > 1e-3
    # missing 1/N: scale by N
    assert _rel(f["o"] * N, ref) > 1e-3


# ------------------------------------------------ optional scale alpha on QK^T
def test_alpha_is_a_query_scaling(oracle_lib):
    """s = alpha <q, k> + rab equals the plain operator on queries alpha*q:
    forward outputs agree, dq(alpha, q) = alpha dq(1, alpha q), every other
    gradient agrees (a scale left out of the forward, dq or dk fails)."""
    w = inputs.make_workload([7, 1, 13, 0, 9], H=2, d=8, N=16, dtype=torch.float64, seed=21)
    alpha = 0.37
    f = oracle_lib.fwd_workload(w, alpha=alpha)
    g = oracle_lib.bwd_workload(w, alpha=alpha)
    qa = w.q.double() * alpha
    f1 = oracle_lib.fwd(qa, w.k, w.v, w.u, w.seq_offsets, w.N, w.pos_w, w.time_w,
                        w.timestamps, w.num_buckets)
    g1 = oracle_lib.bwd(qa, w.k, w.v, w.u, w.seq_offsets, w.N, w.dy, w.pos_w, w.time_w,
                        w.timestamps, w.num_buckets)
    for n in ("o", "y"):
        assert _rel(f[n], f1[n]) < 1e-13, n
    assert _rel(g["dq"], alpha * g1["dq"]) < 1e-12
    for n in ("dk", "dv", "du", "d_pos", "d_time"):
        assert _rel(g[n], g1[n]) < 1e-12, n
    # and alpha = 1 is the plain operator
    f0 = oracle_lib.fwd_workload(w)
    assert np.array_equal(f0["o"], oracle_lib.fwd_workload(w, alpha=1.0)["o"])


def test_alpha_finite_differences(oracle_lib):
    N, H, d = 8, 2, 4
    w = inputs.make_workload([5, 6], H=H, d=d, N=N, dtype=torch.float64, seed=22)
    alpha = -1.7
    g = oracle_lib.bwd_workload(w, alpha=alpha)
    dy = w.dy.double().numpy()

    def loss(q, k):
        r = oracle_lib.fwd(q, k, w.v, w.u, w.seq_offsets, N, w.pos_w, w.time_w,
                           w.timestamps, w.num_buckets, alpha=alpha)
        return float((r["y"] * dy).sum())
    h = 1e-6
    rng = np.random.default_rng(3)
    for name, gname in (("q", "dq"), ("k", "dk")):
        base = getattr(w, name).double().clone()
        flat = base.view(-1)
        for ix in rng.choice(flat.numel(), size=8, replace=False):
            p = flat.clone(); p[ix] += h
            m = flat.clone(); m[ix] -= h
            args_p = (p.view(base.shape), w.k) if name == "q" else (w.q, p.view(base.shape))
            args_m = (m.view(base.shape), w.k) if name == "q" else (w.q, m.view(base.shape))
            fd = (loss(*args_p) - loss(*args_m)) / (2 * h)
            an = float(g[gname].reshape(-1)[ix])
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, ix, fd, an)
