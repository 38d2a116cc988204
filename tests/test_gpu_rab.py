"""GPU parity of the standalone RAB operator (materialised jagged bias and
its backward into the position table, the time-bucket table and the
functional time encoding) against oracle/rab.py.

Float32 output: max|gpu - ref| <= 1e-5 max|ref| per tensor, element by
element.  Cases span several 64 x 64 tiles with ragged edges, empty and
one-token sequences, L = max_len, each parameter alone and all together,
gaps that reach the exact 64-bit bucket path, num_buckets = 1, and the
power-law batch (workload 2) in full; the backward is checked to repeat
bit for bit.
"""
import numpy as np
import pytest
import torch

from oracle import rab as R
from paper_2605_13433_amd import hstu, inputs
from tests.gpu_util import check, say, to_dev

pytestmark = pytest.mark.gpu

TOL = 1e-5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _fn(H, seed):
    rng = np.random.default_rng(seed)
    return torch.from_numpy(np.stack([rng.normal(0, 0.5, H), rng.uniform(0.1, 1.5, H)],
                                     axis=1).astype(np.float32))


def run_case(w, pos=True, time=True, fn=True, seed=0):
    H = w.H
    pos_w = w.pos_w if pos else None
    time_w = w.time_w if time else None
    time_fn = _fn(H, seed) if fn else None
    S = int(R.square_offsets(w.seq_offsets)[-1])
    plan = hstu.RabPlan(to_dev(w.seq_offsets), w.N, H, w.T, S, to_dev(pos_w), to_dev(time_w),
                        to_dev(time_fn), to_dev(w.timestamps), w.num_buckets)
    rab = plan.forward().clone()
    G = torch.from_numpy(np.random.default_rng(seed + 1).standard_normal((H, S))
                         .astype(np.float32))
    d1 = [None if t is None else t.clone() for t in plan.backward(to_dev(G))]
    d2 = [None if t is None else t.clone() for t in plan.backward(to_dev(G))]
    torch.cuda.synchronize()
    ref = R.rab_fwd(w.seq_offsets, w.N, H, pos_w, time_w, w.timestamps, w.num_buckets,
                    time_fn)
    check("rab", rab.cpu().double().numpy(), ref, TOL)
    rp, rt, rf = R.rab_bwd(G.double().numpy(), w.seq_offsets, w.N, H, pos, time,
                           w.timestamps, w.num_buckets, time_fn)
    for name, got, again, want in (("d_pos", d1[0], d2[0], rp), ("d_time", d1[1], d2[1], rt),
                                   ("d_fn", d1[2], d2[2], rf)):
        if want is None:
            assert got is None
            continue
        check(name, got.cpu().double().numpy(), want, TOL)
        assert torch.equal(got.view(torch.int32), again.view(torch.int32)), name


@pytest.mark.parametrize("pos,time,fn", [(True, True, True), (True, False, False),
                                         (False, True, False), (False, False, True)])
def test_small(pos, time, fn):
    w = inputs.make_workload([70, 1, 130, 0, 64, 200], H=2, d=64, N=200, seed=41, num_buckets=48)
    say(f"  rab small pos={pos} time={time} fn={fn}")
    run_case(w, pos, time, fn, seed=1)


def test_far_gaps_and_one_bucket():
    w = inputs.make_workload([90, 150, 3], H=3, d=64, N=160, seed=42)
    gaps = torch.randint(1, 2 ** 31, (w.T,), generator=torch.Generator().manual_seed(0))
    w.timestamps = torch.cumsum(gaps, 0)
    run_case(w, seed=2)
    w1 = inputs.make_workload([65, 7], H=1, d=64, N=80, seed=43, num_buckets=1)
    run_case(w1, seed=3)


def test_workload2_full():
    w = inputs.workload(2)
    say(f"  rab workload 2 {w.name}: T={w.T}")
    run_case(w, seed=4)
