"""hstu_jagged_attn_fwd_noalloc: the forward on the library's fixed per-GPU
scratch matches hstu_jagged_attn_fwd (same kernels: bit for bit, which is
within the bf16 tolerance of the parity tests a fortiori) on two calls in a
row, the second with a smaller input, and a problem too large for the
scratch is rejected before anything runs."""
import pytest
import torch

from paper_2605_13433_amd import hstu, inputs
from tests.gpu_util import say, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _both(w):
    q, k, v, u, off = (to_dev(x) for x in (w.q, w.k, w.v, w.u, w.seq_offsets))
    pos, tw, ts = to_dev(w.pos_w), to_dev(w.time_w), to_dev(w.timestamps)
    plan = hstu.Plan(q, off, w.N, pos, tw, ts, w.num_buckets, backward=False)
    ref = plan.forward(q, k, v, u, off)
    T, H, d = q.shape
    y = torch.full((T, H * d), 7.0, dtype=q.dtype, device="cuda")
    o = torch.full((T, H, d), 7.0, dtype=q.dtype, device="cuda")
    mean = torch.full((T,), 7.0, dtype=torch.float32, device="cuda")
    rstd = torch.full((T,), 7.0, dtype=torch.float32, device="cuda")
    out = hstu.FwdOut(hstu._dtype_code(q), T, y.data_ptr(), o.data_ptr(), mean.data_ptr(),
                      rstd.data_ptr(), None, 0)
    hstu.hstu_jagged_attn_fwd_noalloc(q, k, v, u, off, w.B, w.N, H, d, plan.rab, out)
    torch.cuda.synchronize()
    for name, a, b in (("y", y, ref.y), ("o", o, ref.o), ("mean", mean, ref.ln_mean),
                       ("rstd", rstd, ref.ln_rstd)):
        assert torch.equal(a, b), name


def test_noalloc_matches_forward_twice_shrinking():
    big = inputs.make_workload([300, 1, 64, 129, 0, 700], H=4, d=64, N=768, seed=700)
    # mean length >= 256 at d=64: the forward's two-query-tile items
    pairs = inputs.make_workload([600, 1, 64, 129, 0, 900, 300], H=4, d=64, N=900, seed=703)
    small = inputs.make_workload([65, 2], H=2, d=128, N=128, seed=701)
    say("no-alloc forward: large batch, a pair-item batch, then a smaller one (d=64, then d=128)")
    _both(big)
    _both(pairs)
    _both(small)
    f32 = inputs.make_workload([40, 3], H=2, d=32, N=64, dtype=torch.float32, seed=702)
    _both(f32)


def test_noalloc_rejects_oversize():
    # 64 sequences of 8192 tokens need 64 * 128 work-list entries of 24 bytes
    # plus records: still small; 1 M one-token sequences need ~40 MB
    B, N = 1 << 20, 64
    q = torch.zeros(B, 1, 64, dtype=torch.bfloat16, device="cuda")
    off = torch.arange(B + 1, dtype=torch.int64, device="cuda")
    out = hstu.FwdOut(hstu.HSTU_BF16, B, q.data_ptr(), q.data_ptr(), q.data_ptr(),
                      q.data_ptr(), None, 0)
    with pytest.raises(hstu.HstuError) as ei:
        hstu.hstu_jagged_attn_fwd_noalloc(q, q, q, q, off, B, N, 1, 64, None, out)
    assert ei.value.code == -3 and "scratch" in str(ei.value)
