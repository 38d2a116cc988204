"""HSTU_VALIDATE=1: the scheduler checks the seq_offsets contract on the
device and reports violations through the workspace status word, without
the host waiting on the device during the call.

Every offsets array below stays inside [0, total_tokens], so the kernels'
own clamps keep every access in bounds whether or not the check runs; the
check only adds the report (and skips the attention work on a violation).
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2605_13433_amd import hstu, inputs
from tests.gpu_util import TOL, check, say, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.build(force=False)


@pytest.fixture
def validate_on(monkeypatch):
    monkeypatch.setenv("HSTU_VALIDATE", "1")


def _plan(w, off):
    q, k, v, u = (to_dev(x) for x in (w.q, w.k, w.v, w.u))
    pos, tw, ts = to_dev(w.pos_w), to_dev(w.time_w), to_dev(w.timestamps)
    plan = hstu.Plan(q, off, w.N, pos, tw, ts, w.num_buckets, backward=True)
    return plan, (q, k, v, u)


def test_valid_offsets_report_zero_and_match_oracle(validate_on):
    w = inputs.make_workload([70, 1, 0, 130], H=2, d=64, N=160, seed=600)
    say("HSTU_VALIDATE=1, valid offsets")
    off = to_dev(w.seq_offsets)
    plan, (q, k, v, u) = _plan(w, off)
    f = plan.forward(q, k, v, u, off)
    assert plan.status() == 0
    g = plan.backward(q, k, v, u, off, to_dev(w.dy))
    assert plan.status(backward=True) == 0
    torch.cuda.synchronize()
    ref = oracle.fwd_workload(w)
    check("o", f.o.double().cpu().numpy(), ref["o"], TOL[w.dtype])
    refb = oracle.bwd_workload(w)
    check("dq", g.dq.double().cpu().numpy(), refb["dq"], TOL[w.dtype])


def test_unchecked_without_env(monkeypatch):
    monkeypatch.delenv("HSTU_VALIDATE", raising=False)
    w = inputs.make_workload([70, 30], H=1, d=64, N=128, seed=601)
    off = to_dev(w.seq_offsets)
    plan, (q, k, v, u) = _plan(w, off)
    plan.forward(q, k, v, u, off)
    assert plan.status() == hstu.HSTU_SEQ_UNCHECKED


@pytest.mark.parametrize("offsets,bits", [
    ([5, 40, 100], hstu.HSTU_SEQ_FIRST_NOT_ZERO),          # off[0] != 0
    ([0, 60, 40, 100], hstu.HSTU_SEQ_DECREASING),           # a negative length
    ([0, 10, 100], hstu.HSTU_SEQ_TOO_LONG),                 # 90 > max_len = 64
    ([0, 30, 90], hstu.HSTU_SEQ_LAST_NOT_T),                # off[B] = 90 != T = 100
    ([3, 2, 100], hstu.HSTU_SEQ_FIRST_NOT_ZERO | hstu.HSTU_SEQ_DECREASING
     | hstu.HSTU_SEQ_TOO_LONG),
])
def test_violations_are_reported(validate_on, offsets, bits):
    say(f"HSTU_VALIDATE=1, offsets {offsets}, expected status {bits:#x}")
    T = 100
    w = inputs.make_workload([T], H=2, d=64, N=64, seed=602)   # tensors of T rows
    off = torch.tensor(offsets, dtype=torch.int64, device="cuda")
    plan, (q, k, v, u) = _plan(w, torch.tensor([0, T], dtype=torch.int64, device="cuda"))
    plan.B = len(offsets) - 1
    # the plan's workspaces were sized for B = 1; size them for this B
    code = hstu._dtype_code(q)
    plan.fwd_ws = hstu._workspace(hstu.hstu_jagged_attn_workspace_bytes(
        plan.B, plan.N, plan.H, plan.d, T, 0, code, plan.rab), q.device)
    plan.out.workspace, plan.out.workspace_bytes = plan.fwd_ws.data_ptr(), plan.fwd_ws.numel()
    plan.bwd_ws = hstu._workspace(hstu.hstu_jagged_attn_workspace_bytes(
        plan.B, plan.N, plan.H, plan.d, T, 1, code, plan.rab), q.device)
    plan.io.workspace, plan.io.workspace_bytes = plan.bwd_ws.data_ptr(), plan.bwd_ws.numel()
    plan.forward(q, k, v, u, off)
    assert plan.status() == bits
    g = plan.backward(q, k, v, u, off, to_dev(w.dy))
    assert plan.status(backward=True) == bits
    torch.cuda.synchronize()
    # the table gradients are still written (no causal pair was processed)
    assert np.all(np.isfinite(g.d_pos_w.cpu().numpy()))
