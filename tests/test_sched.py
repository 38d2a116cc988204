"""seq_offsets tile scheduler: a host reference enumerator, its properties,
and the device scheduler's work lists checked against it bit for bit (as
multisets), with their order.  The scheduler takes one of two orders:
cost-major (every entry longest first) unless the causal work per nominal
work-group is at least SLACK times the longest entry, then sequence-major
(sequence by sequence, longest sequence first, order among equal lengths
free, each sequence's tiles longest first)."""
import itertools

import numpy as np
import pytest
import torch

TILE = 64
SLACK = 4          # work per work-group over the longest entry for sequence-major


def reference_lists(lengths, N):
    """Entries (b, tile) with their causal cost, sorted longest first."""
    q, k = [], []
    for b, L in enumerate(lengths):
        L = max(0, min(int(L), N))
        nt = (L + TILE - 1) // TILE
        for t in range(nt):
            q.append((t + 1, b, t))        # q-tile t visits key tiles 0..t
            k.append((nt - t, b, t))       # key tile t is visited by q-tiles t..nt-1
    q.sort(key=lambda x: -x[0])
    k.sort(key=lambda x: -x[0])
    return q, k


def tile_pairs(lengths, N):
    """Every (b, qt, kt) with kt <= qt < ntiles_b: the lower-triangular work."""
    out = set()
    for b, L in enumerate(lengths):
        nt = (min(int(L), N) + TILE - 1) // TILE
        out |= {(b, qt, kt) for qt in range(nt) for kt in range(qt + 1)}
    return out


def lpt_makespan(costs, m):
    loads = [0] * m
    for c in sorted(costs, reverse=True):
        i = loads.index(min(loads))
        loads[i] += c
    return max(loads)


def opt_makespan(costs, m):
    best = sum(costs)
    for assign in itertools.product(range(m), repeat=len(costs)):
        loads = [0] * m
        for c, a in zip(costs, assign):
            loads[a] += c
        best = min(best, max(loads))
    return best


@pytest.mark.parametrize("lengths,N", [([0, 1, 64, 65, 130, 512], 512),
                                       ([8192, 1, 4000], 8192),
                                       (list(range(0, 300, 7)), 300)])
def test_reference_covers_each_tile_pair_once(lengths, N):
    q, k = reference_lists(lengths, N)
    pairs_q = [(b, t, kt) for _, b, t in q for kt in range(t + 1)]
    assert len(pairs_q) == len(set(pairs_q))
    assert set(pairs_q) == tile_pairs(lengths, N)
    nts = {b: (min(L, N) + TILE - 1) // TILE for b, L in enumerate(lengths)}
    pairs_k = [(b, qt, t) for _, b, t in k for qt in range(t, nts[b])]
    assert len(pairs_k) == len(set(pairs_k)) and set(pairs_k) == tile_pairs(lengths, N)
    assert sum(c for c, _, _ in q) == len(tile_pairs(lengths, N))
    assert all(q[i][0] >= q[i + 1][0] for i in range(len(q) - 1))


def test_lpt_within_graham_bound_bruteforce():
    rng = np.random.default_rng(0)
    for _ in range(40):
        n, m = int(rng.integers(2, 8)), int(rng.integers(2, 4))
        costs = [int(c) for c in rng.integers(1, 20, size=n)]
        assert lpt_makespan(costs, m) <= (4 / 3 - 1 / (3 * m)) * opt_makespan(costs, m) + 1e-9


def sequence_major(lengths, N, H, grid):
    """The scheduler's choice of order: causal tile pairs over all heads
    against SLACK times the longest entry on every work-group."""
    nt = (np.minimum(np.asarray(lengths), N) + TILE - 1) // TILE
    if nt.size == 0 or nt.max() == 0:
        return False
    work = int((nt * (nt + 1) // 2).sum())
    return work * H >= SLACK * int(nt.max()) * grid


def check_order(got, nts, seq_major):
    """got: [(cost, b, tile)] in pop order."""
    if not seq_major:
        costs = [c for c, _, _ in got]
        assert costs == sorted(costs, reverse=True)
        return
    # contiguous per-sequence blocks, in non-increasing tile count
    blocks = []
    for c, b, t in got:
        if not blocks or blocks[-1][0] != b:
            assert all(b != bb for bb, _ in blocks), "sequence split across blocks"
            blocks.append((b, []))
        blocks[-1][1].append(c)
    sizes = [int(nts[b]) for b, _ in blocks]
    assert sizes == sorted(sizes, reverse=True)
    # inside a block: costs nt, nt-1, ..., 1 (longest first)
    for b, costs in blocks:
        assert costs == list(range(int(nts[b]), 0, -1))


def test_order_choice():
    grid = 1024
    assert not sequence_major([512] * 128, 512, 4, grid)      # 8 tiles, little work
    assert sequence_major([8192] * 1024, 8192, 4, grid)       # deep batch
    assert not sequence_major([], 64, 4, grid)
    assert not sequence_major([0, 0], 64, 4, grid)
    # the threshold itself: one sequence of nt tiles, nt (nt + 1) / 2 pairs
    nt = 7
    need = SLACK * nt * grid            # pairs x H
    H = -(-need // (nt * (nt + 1) // 2))
    assert not sequence_major([nt * TILE], nt * TILE, H - 1, grid)
    assert sequence_major([nt * TILE], nt * TILE, H, grid)


@pytest.mark.gpu
@pytest.mark.parametrize("seed,B,N", [(0, 7, 256), (1, 300, 512), (2, 1024, 8192), (3, 5, 64)])
def test_device_lists_match_reference(seed, B, N):
    from paper_2605_13433_amd import hstu
    rng = np.random.default_rng(seed)
    lengths = rng.integers(0, N + 1, size=B)
    lengths[: min(3, B)] = [0, N, 1][: min(3, B)]
    off = np.zeros(B + 1, dtype=np.int64)
    np.cumsum(lengths, out=off[1:])
    print(f"schedule seed={seed} B={B} N={N} T={off[-1]}", flush=True)
    lq, lk = hstu.schedule(torch.from_numpy(off).cuda(), N, int(off[-1]))
    q, k = reference_lists(lengths, N)
    assert len(lq) == len(q)
    nts = (np.minimum(lengths, N) + TILE - 1) // TILE
    got_q = [(t + 1, b, t) for b, t in lq.tolist()]
    got_k = [(int(nts[b]) - t, b, t) for b, t in lk.tolist()]
    assert sorted(got_q) == sorted(q) and sorted(got_k) == sorted(k)
    grid = 4 * torch.cuda.get_device_properties(0).multi_processor_count
    seq_major = sequence_major(lengths, N, 1, grid)
    print(f"  order: {'sequence' if seq_major else 'cost'}-major", flush=True)
    for got in (got_q, got_k):
        check_order(got, nts, seq_major)
