"""GPU parity: the HIP path against the CPU oracle, element by element.

Tolerance per output tensor: max|gpu - ref| <= 2e-2 max|ref| for bf16 and
1e-5 max|ref| for fp32, on y, o, dq, dk, dv, du, d_pos and d_time (o is
checked as well as y: LayerNorm is scale-invariant, so a wrong global scale
of o would hide in y).  Small cases span several 64-row tiles, ragged tails,
empty and single-token sequences and L = max_len; the five workloads run at
full size in the launch configuration the benchmark times, with the oracle
on every row and both tables for workloads 1-4, and on sampled whole
sequences (always the longest ones) for the 1024-sequence Zipf batch.
Sequence handling (offsets, masks, isolation) is checked bit-exactly.
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2605_13433_amd import hstu, inputs
from tests.gpu_util import TOL, check, rows_of, run_gpu, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.build(force=False)


def compare(w, got, ref_f, ref_b=None, rows=None, tables=True):
    tol = TOL[w.dtype]
    sel = (lambda a: a) if rows is None else (lambda a: a[rows])
    check("o", sel(got["o"]), ref_f["o"], tol)
    check("y", sel(got["y"]), ref_f["y"], tol)
    if ref_b is not None:
        for n in ("dq", "dk", "dv", "du"):
            check(n, sel(got[n]), ref_b[n], tol)
        if tables and w.pos_w is not None:
            check("d_pos", got["d_pos"], ref_b["d_pos"], tol)
        if tables and w.time_w is not None:
            check("d_time", got["d_time"], ref_b["d_time"], tol)


SMALL = [
    # lengths, H, d, N, pos, time
    ([1, 63, 64, 65, 130, 0, 200, 17, 256], 2, 64, 256, True, True),
    ([1, 63, 64, 65, 130, 0, 200, 17, 256], 2, 128, 256, True, True),
    ([129, 5, 64, 191], 3, 64, 192, True, False),
    ([100, 33, 0, 7], 1, 128, 128, False, True),
    ([77, 250, 3], 2, 64, 250, False, False),
    ([2, 1, 1, 3, 64], 4, 64, 64, True, True),
    ([1, 40, 64, 90, 5, 0], 2, 64, 128, False, True),   # one-tile sequences, time bias only
]


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_small_bf16(case):
    lengths, H, d, N, pos, time = SMALL[case]
    say(f"small bf16 case {case}: lengths={lengths} H={H} d={d} N={N} pos={pos} time={time}")
    w = inputs.make_workload(lengths, H=H, d=d, N=N, pos=pos, time=time, seed=100 + case)
    got = run_gpu(w)
    compare(w, got, oracle.fwd_workload(w), oracle.bwd_workload(w))


# Mean length >= 256 tokens: the bf16 d=64 forward takes items of two query
# tiles (the pair list; the d=128 cases run the same batches through the
# one-tile items).  Odd and even tile counts (the last pair of an odd count
# has no upper tile), one-tile and empty sequences, L = max_len.
PAIRS = [
    ([256, 320, 64, 65, 1, 767, 0, 639], 2, 64, 768, True, True),
    ([256, 320, 64, 65, 1, 767, 0, 639], 2, 128, 768, True, True),
    ([300, 1, 511], 3, 64, 512, True, False),
    ([190, 700, 129], 1, 128, 700, False, True),
    ([190, 700, 129], 2, 64, 700, False, True),
    ([640, 64, 257, 100], 2, 64, 640, False, False),
]


@pytest.mark.parametrize("case", range(len(PAIRS)))
def test_pair_items_bf16(case):
    lengths, H, d, N, pos, time = PAIRS[case]
    assert sum(lengths) >= 256 * len(lengths)
    say(f"pair-item bf16 case {case}: lengths={lengths} H={H} d={d} N={N} pos={pos} time={time}")
    w = inputs.make_workload(lengths, H=H, d=d, N=N, pos=pos, time=time, seed=300 + case)
    got = run_gpu(w)
    compare(w, got, oracle.fwd_workload(w), oracle.bwd_workload(w))


# Enough 64-row tiles that the backward runs as two launches (a dK/dV
# kernel, then a dQ kernel) rather than the combined one, at d=64 with
# every bias combination: 600 short sequences (one to three tiles) and two
# long ones (16 and 11 tiles: long runs of streamed tiles through the dQ
# kernel's double buffers).
@pytest.mark.parametrize("pos,time", [(True, True), (True, False), (False, True),
                                      (False, False)])
def test_split_backward_d64(pos, time):
    from paper_2605_13433_amd import hstu
    rng = np.random.default_rng(77)
    lengths = [1000, 700] + rng.integers(20, 141, size=600).tolist()
    w = inputs.make_workload(lengths, H=4, d=64, N=1024, pos=pos, time=time, seed=400)
    say(f"split backward d=64 pos={pos} time={time}: B={w.B} T={w.T}")
    # the library takes the combined launch below 4 items per work-group of
    # its grid (CUs x occupancy, at most 4 work-groups per CU here)
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    assert hstu.max_entries(w.B, w.N, w.T) * w.H >= 4 * 4 * n_cu
    got = run_gpu(w)
    compare(w, got, oracle.fwd_workload(w), oracle.bwd_workload(w))


# The same at d=128 (two launches there too), every bias combination.
@pytest.mark.parametrize("pos,time", [(True, True), (True, False), (False, True),
                                      (False, False)])
def test_split_backward_d128(pos, time):
    from paper_2605_13433_amd import hstu
    rng = np.random.default_rng(81)
    lengths = [800, 300] + rng.integers(20, 141, size=600).tolist()
    w = inputs.make_workload(lengths, H=4, d=128, N=800, pos=pos, time=time, seed=403)
    say(f"split backward d=128 pos={pos} time={time}: B={w.B} T={w.T}")
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    assert hstu.max_entries(w.B, w.N, w.T) * w.H >= 4 * 4 * n_cu
    got = run_gpu(w)
    compare(w, got, oracle.fwd_workload(w), oracle.bwd_workload(w))


def test_pair_items_cover_every_tile():
    """The 1024-sequence Zipf batch (sequence-major pair list): every row of
    o is written (o starts as NaN), complementing the sampled parity below."""
    from paper_2605_13433_amd import hstu
    from tests.gpu_util import to_dev
    w = inputs.workload(5)
    say(f"  pair coverage, workload 5 {w.name}: T={w.T}")
    q, k, v, u = (to_dev(x) for x in (w.q, w.k, w.v, w.u))
    off = to_dev(w.seq_offsets)
    plan = hstu.Plan(q, off, w.N, to_dev(w.pos_w), to_dev(w.time_w), to_dev(w.timestamps),
                     w.num_buckets, backward=False)
    plan.o.fill_(float("nan"))
    f = plan.forward(q, k, v, u, off)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(f.o).all())


@pytest.mark.parametrize("d", [32, 64, 128])
def test_small_f32(d):
    lengths = [1, 70, 0, 33, 128]
    say(f"small fp32 d={d}: lengths={lengths}")
    w = inputs.make_workload(lengths, H=2, d=d, N=128, dtype=torch.float32, seed=200 + d)
    got = run_gpu(w)
    compare(w, got, oracle.fwd_workload(w), oracle.bwd_workload(w))


def far_timestamps(lengths, seed):
    """Timestamps that drive the exact time-bucket path: per sequence (in
    order) mostly small gaps with a few of 2^22..2^31 s (tiles go from near
    to far of the sequence's first timestamp part-way), every gap about 2^26 s
    (deltas beyond 32 bits), small gaps only (fast path), and small gaps in
    shuffled order (negative deltas, non-monotone index runs)."""
    rng = np.random.default_rng(seed)
    out = []
    for b, L in enumerate(lengths):
        kind = b % 4
        g = 1 + np.floor(rng.exponential(600.0, size=L)).astype(np.int64)
        if kind == 0:
            big = rng.random(L) < 0.05
            g[big] = rng.integers(1 << 22, 1 << 31, size=int(big.sum()))
        elif kind == 1:
            g = rng.integers(1 << 25, 1 << 27, size=L)
        ts = np.cumsum(g)
        ts -= ts[0] if L else 0
        if kind == 3:
            rng.shuffle(ts)
        out.append(ts)
    return torch.from_numpy(np.concatenate(out).astype(np.int64))


@pytest.mark.parametrize("d,dtype", [(64, torch.bfloat16), (128, torch.bfloat16),
                                     (64, torch.float32)])
def test_far_timestamps(d, dtype):
    lengths = [200, 130, 65, 150, 64, 1, 250, 190]
    say(f"far timestamps d={d} {dtype}: lengths={lengths}")
    w = inputs.make_workload(lengths, H=2, d=d, N=256, dtype=dtype, seed=300 + d)
    w.timestamps = far_timestamps(lengths, seed=301)
    ts = w.timestamps.numpy()
    off = w.seq_offsets.numpy()
    far = sum(int((np.abs(ts[off[b]:off[b + 1]] - ts[off[b]]) >= 1 << 23).any())
              for b in range(len(lengths)) if off[b + 1] > off[b])
    assert far >= 3
    got = run_gpu(w)
    compare(w, got, oracle.fwd_workload(w), oracle.bwd_workload(w))


def test_long_sequence():
    """One sequence longer than any workload's (141 tiles, ragged last tile)
    beside short ones: tile indices, bias-table spans and scheduler bins past
    the workloads' range."""
    lengths = [9000, 300, 1, 64]
    say(f"long sequence: lengths={lengths}")
    w = inputs.make_workload(lengths, H=1, d=64, N=9000, seed=400)
    got = run_gpu(w)
    compare(w, got, oracle.fwd_workload(w), oracle.bwd_workload(w))


def test_workload1_fp32_forward():
    w = inputs.workload(1)
    say(f"workload 1 {w.name}: T={w.T} pairs/head={w.pairs}")
    got = run_gpu(w, bwd=False)
    compare(w, got, oracle.fwd_workload(w))


def test_workload2_full():
    w = inputs.workload(2)
    say(f"workload 2 {w.name}: T={w.T} pairs/head={w.pairs}")
    got = run_gpu(w)
    compare(w, got, oracle.fwd_workload(w), oracle.bwd_workload(w))


def assert_finite(got):
    """Every element of every output of a full-size run is finite (the
    oracle comparisons of sampled runs only see the sampled rows)."""
    for n, a in got.items():
        if a is not None:
            assert np.all(np.isfinite(a)), f"non-finite values in {n}"


def test_workload3_full():
    """Long-tail batch (d=128, lengths to 2048): every row and both
    full-batch tables against the oracle."""
    w = inputs.workload(3)
    say(f"workload 3 {w.name}: T={w.T} pairs/head={w.pairs} max L={int(w.lengths.max())}")
    got = run_gpu(w)
    assert_finite(got)
    compare(w, got, oracle.fwd_workload(w), oracle.bwd_workload(w))


def test_workload4_attention_full():
    """Layer batch's attention (d=128, lengths to 4096): every row and both
    full-batch tables against the oracle."""
    w = inputs.workload(4)
    say(f"workload 4 {w.name}: T={w.T} pairs/head={w.pairs} max L={int(w.lengths.max())}")
    got = run_gpu(w)
    assert_finite(got)
    compare(w, got, oracle.fwd_workload(w), oracle.bwd_workload(w))


def test_workload5_sampled():
    """Zipf batch (1024 sequences to 8192 tokens) at full size.  The oracle
    runs on whole sequences: the four longest (they hold most of the causal
    pairs), two more above 2M pairs, the two shortest and random picks.
    Table gradients sum over every sequence; the oracle checks them three
    ways: on the sampled sub-batch run by itself; on the full batch at every
    diagonal m >= L of the fifth-longest sequence (only the four sampled
    longest sequences reach those diagonals, so there the full batch's
    d_pos equals the sub-batch oracle's); and the full batch's table must be
    the sum of the sample's and the complement's (additivity)."""
    w = inputs.workload(5)
    say(f"workload 5 {w.name}: T={w.T} pairs/head={w.pairs} (full-size GPU run)")
    got = run_gpu(w)
    assert_finite(got)
    L = w.lengths
    order = np.argsort(L, kind="stable")
    rng = np.random.default_rng(5)
    chosen = set(int(b) for b in order[:2]) | set(int(b) for b in order[-4:])
    big = [int(b) for b in order[:-4] if L[b] * (L[b] + 1) // 2 > 2_000_000]
    chosen |= set(int(b) for b in rng.choice(big, size=2, replace=False))
    chosen |= set(int(b) for b in rng.choice(order[:-4], size=6, replace=False))
    seqs = sorted(chosen)
    sub = inputs.subset(w, seqs)
    say(f"  sampled sequences {seqs} lengths {L[seqs].tolist()} "
        f"({100.0 * sub.pairs / w.pairs:.1f}% of the causal pairs)")
    ref_f = oracle.fwd_workload(sub)
    ref_b = oracle.bwd_workload(sub)
    rows = rows_of(w, seqs)
    compare(w, got, ref_f, ref_b, rows=rows, tables=False)
    m0 = int(L[order[-5]])                         # fifth-longest length
    hi = w.N - 1 - m0 + 1                          # index j - i + N - 1 <= N - 1 - m0
    say(f"  full-batch d_pos at diagonals m >= {m0} (only sampled sequences reach them):")
    check("d_pos[m>=m0]", got["d_pos"][:, :hi], ref_b["d_pos"][:, :hi], TOL[w.dtype])
    assert np.all(got["d_pos"][:, w.N:] == 0)      # j > i: no causal pair
    say("  tables on the sampled sub-batch:")
    got_sub = run_gpu(sub)
    compare(sub, got_sub, ref_f, ref_b)
    rest = [b for b in range(w.B) if b not in chosen]
    got_rest = run_gpu(inputs.subset(w, rest))
    for n in ("d_pos", "d_time"):
        if got[n] is not None:
            check(n + "+", got_sub[n] + got_rest[n], got[n], 1e-3)


def test_long_sequence_d128():
    """One 4096-token sequence at d=128 with both biases (64 tiles; the
    dK/dV and dQ items of its first tiles stream 64 tiles each)."""
    lengths = [4096, 1, 700]
    say(f"long sequence d=128: lengths={lengths}")
    w = inputs.make_workload(lengths, H=2, d=128, N=4096, seed=410)
    got = run_gpu(w)
    compare(w, got, oracle.fwd_workload(w), oracle.bwd_workload(w))


def test_max_size_batch():
    """Every size limit at once: four sequences of max_len = 65536 tokens
    (1024 tiles each) at H = 64 heads of d = 128, so that one head's rows
    of a sequence span 2^30 bytes (the bound of the kernels' 32-bit
    in-sequence offsets) and element offsets pass 2^31; H * num_buckets =
    4096; both biases; then short sequences that start at element 2^31.
    The inputs are drawn on the GPU.  The oracle cannot run a 65536-token
    sequence, so it checks what causality isolates exactly: o, y, dQ and dU
    of the first rows of the first and the last long sequence depend on
    those rows alone, and the short sequences are checked whole.  Every
    element of every output must be finite and d_pos zero for j > i."""
    N, H, d, nb = 65536, 64, 128, 64
    lengths = [N] * 4 + [333, 1, 64]
    say(f"max-size batch: lengths={lengths} H={H} d={d} N={N} num_buckets={nb}")
    w = inputs.device_workload(lengths, H, d, N, seed=430, num_buckets=nb)
    off = w.seq_offsets.numpy()
    assert off[4] * H * d == 1 << 31
    dev = w.q.device
    offd, ts = w.seq_offsets.to(dev), w.timestamps.to(dev)
    plan = hstu.Plan(w.q, offd, N, w.pos_w.to(dev), w.time_w.to(dev), ts, nb)
    f = plan.forward(w.q, w.k, w.v, w.u, offd)
    g = plan.backward(w.q, w.k, w.v, w.u, offd, w.dy)
    torch.cuda.synchronize()
    say("  GPU run done")
    outs = dict(o=f.o, y=f.y, dq=g.dq, dk=g.dk, dv=g.dv, du=g.du, d_pos=g.d_pos_w,
                d_time=g.d_time_w)
    for n, t in outs.items():
        assert bool(torch.isfinite(t).all()), f"non-finite values in {n}"
    assert bool((g.d_pos_w[:, N:] == 0).all())

    def rows(t, r):
        return t.index_select(0, torch.from_numpy(r).to(dev)).to("cpu", torch.float64).numpy()

    tol = TOL[w.dtype]
    for b, n in ((0, 200), (3, 200)):
        say(f"  first {n} rows of sequence {b} (rows from {off[b]})")
        pw = inputs.prefix(w, b, n)
        ref_f, ref_b = oracle.fwd_workload(pw), oracle.bwd_workload(pw)
        r = np.arange(off[b], off[b] + n, dtype=np.int64)
        check("o", rows(f.o, r), ref_f["o"], tol)
        check("y", rows(f.y, r), ref_f["y"], tol)
        check("dq", rows(g.dq, r), ref_b["dq"], tol)
        check("du", rows(g.du, r), ref_b["du"], tol)
    say("  short sequences 4-6, every output row")
    sw = inputs.subset(w, [4, 5, 6])
    ref_f, ref_b = oracle.fwd_workload(sw), oracle.bwd_workload(sw)
    r = rows_of(w, [4, 5, 6])
    for n, t in outs.items():
        if n in ("o", "y"):
            check(n, rows(t, r), ref_f[n], tol)
        elif n not in ("d_pos", "d_time"):
            check(n, rows(t, r), ref_b[n], tol)
    del plan, f, g, outs, w
    torch.cuda.empty_cache()


def test_fp32_past_2g_elements():
    """The fp32 path with element offsets past 2^31: 4096 sequences of 64
    tokens at H = 64, d = 128 (8.6 GB per operand), then short sequences
    that start at element 2^31, both biases, inputs drawn on the GPU.  The
    sequences are independent, so whole sequences at the start, the middle
    and the end are checked against the oracle; every output element is
    finite and d_pos zero for j > i."""
    H, d, N = 64, 128, 333
    lengths = [64] * 4096 + [333, 1, 64]
    say(f"fp32 past 2^31 elements: 4096 x 64 + [333, 1, 64] tokens, H={H} d={d} N={N}")
    w = inputs.device_workload(lengths, H, d, N, dtype=torch.float32, seed=440)
    off = w.seq_offsets.numpy()
    assert off[4096] * H * d == 1 << 31
    dev = w.q.device
    offd, ts = w.seq_offsets.to(dev), w.timestamps.to(dev)
    plan = hstu.Plan(w.q, offd, N, w.pos_w.to(dev), w.time_w.to(dev), ts, w.num_buckets)
    f = plan.forward(w.q, w.k, w.v, w.u, offd)
    g = plan.backward(w.q, w.k, w.v, w.u, offd, w.dy)
    torch.cuda.synchronize()
    say("  GPU run done")
    outs = dict(o=f.o, y=f.y, dq=g.dq, dk=g.dk, dv=g.dv, du=g.du, d_pos=g.d_pos_w,
                d_time=g.d_time_w)
    for n, t in outs.items():
        assert bool(torch.isfinite(t).all()), f"non-finite values in {n}"
    assert bool((g.d_pos_w[:, N:] == 0).all())
    seqs = [0, 2047, 4095, 4096, 4097, 4098]
    say(f"  sequences {seqs}, every output row")
    sw = inputs.subset(w, seqs)
    ref_f, ref_b = oracle.fwd_workload(sw), oracle.bwd_workload(sw)
    r = torch.from_numpy(rows_of(w, seqs)).to(dev)
    tol = TOL[w.dtype]
    for n, t in outs.items():
        if n in ("d_pos", "d_time"):
            continue
        got = t.index_select(0, r).to("cpu", torch.float64).numpy()
        check(n, got, (ref_f if n in ("o", "y") else ref_b)[n], tol)
    del plan, f, g, outs, w
    torch.cuda.empty_cache()


@pytest.mark.parametrize("nb", [32, 1])
@pytest.mark.parametrize("d,dtype", [(64, torch.bfloat16), (128, torch.bfloat16),
                                     (64, torch.float32)])
def test_num_buckets(nb, d, dtype):
    """Bucket counts other than 128: with 32 buckets (HSTU's count) the
    seeded gaps reach buckets past 31, which clamp to the last one; with one
    bucket every pair reads bucket 0.  Far timestamps in two sequences drive
    the exact path's clamp as well."""
    lengths = [200, 130, 65, 150, 64, 1, 250, 190]
    say(f"num_buckets={nb} d={d} {dtype}: lengths={lengths}")
    w = inputs.make_workload(lengths, H=2, d=d, N=256, dtype=dtype, num_buckets=nb,
                             seed=500 + nb + d)
    w.timestamps = far_timestamps(lengths, seed=501)
    got = run_gpu(w)
    compare(w, got, oracle.fwd_workload(w), oracle.bwd_workload(w))


# ---------------------------------------------------- bit-exact jagged handling
def _fwd_bits(w):
    got = run_gpu(w, bwd=False)
    return got["o"], got["y"]


def test_causality_and_isolation_bitwise():
    lengths = [150, 70, 129]
    w = inputs.make_workload(lengths, H=2, d=64, N=256, seed=7)
    say("bitwise causality / isolation, lengths=" + str(lengths))
    o0, y0 = _fwd_bits(w)
    t = 40                       # perturb token 40 of sequence 0 (and later ones)
    for name in ("q", "k", "v", "u"):
        x = getattr(w, name).clone()
        x[t] += 1.0
        old = getattr(w, name)
        setattr(w, name, x)
        o1, y1 = _fwd_bits(w)
        setattr(w, name, old)
        assert np.array_equal(o1[:t], o0[:t]) and np.array_equal(y1[:t], y0[:t]), name
        assert np.array_equal(o1[150:], o0[150:]) and np.array_equal(y1[150:], y0[150:]), name
    ts = w.timestamps.clone()
    ts[t:150] += 5000
    old = w.timestamps
    w.timestamps = ts
    o1, _ = _fwd_bits(w)
    w.timestamps = old
    assert np.array_equal(o1[:t], o0[:t]) and np.array_equal(o1[150:], o0[150:])


def test_split_and_permute_bitwise():
    lengths = [65, 1, 200, 0, 64, 33]
    w = inputs.make_workload(lengths, H=2, d=128, N=256, seed=8)
    say("bitwise split / permutation, lengths=" + str(lengths))
    o0, y0 = _fwd_bits(w)
    off = w.seq_offsets.numpy()
    for part in ([0, 1, 2], [3, 4, 5], [5, 2, 0, 4, 1, 3]):
        sub = inputs.subset(w, part)
        o1, y1 = _fwd_bits(sub)
        rows = np.concatenate([np.arange(off[b], off[b + 1]) for b in part]).astype(int)
        assert np.array_equal(o1, o0[rows]) and np.array_equal(y1, y0[rows]), part


def test_forward_deterministic_and_guard_bands():
    from paper_2605_13433_amd import hstu
    w = inputs.make_workload([100, 64, 3], H=2, d=64, N=128, seed=9)
    say("determinism + guard bands")
    dev = lambda t: t.contiguous().cuda()
    q, k, v, u, off = (dev(x) for x in (w.q, w.k, w.v, w.u, w.seq_offsets))
    pos, tw, ts = dev(w.pos_w), dev(w.time_w), dev(w.timestamps)
    plan = hstu.Plan(q, off, w.N, pos, tw, ts, w.num_buckets, backward=False)
    T, H, d = q.shape
    pad = 4096
    canary = torch.full((T * H * d + 2 * pad,), -12345.0, dtype=torch.bfloat16, device="cuda")
    o_view = canary[pad:pad + T * H * d].view(T, H, d)
    plan.o = o_view
    plan.out.o = o_view.data_ptr()
    r1 = plan.forward(q, k, v, u, off).y.clone()
    r2 = plan.forward(q, k, v, u, off).y.clone()
    torch.cuda.synchronize()
    assert torch.equal(r1, r2)
    assert torch.all(canary[:pad] == -12345.0) and torch.all(canary[pad + T * H * d:] == -12345.0)


def test_degenerate_batches():
    say("degenerate: all-empty batch backward writes zero tables; L = N; B = 1")
    w = inputs.make_workload([0, 0, 0], H=2, d=64, N=64, seed=10)
    got = run_gpu(w)
    assert np.all(got["d_pos"] == 0) and np.all(got["d_time"] == 0)
    w = inputs.make_workload([64], H=1, d=64, N=64, seed=11)
    got = run_gpu(w)
    compare(w, got, oracle.fwd_workload(w), oracle.bwd_workload(w))
