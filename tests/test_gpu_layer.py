"""GPU parity of the HSTU layer shell (hstu_layer_fwd / hstu_layer_bwd)
against the layer oracle, element by element.

Every tensor the layer returns or saves is checked at the bf16 tolerance
max|gpu - ref| <= 2e-2 max|ref|: out, h (= x w1), the four silu'd planes
U, V, Q, K, o, y, dx, dw1, dw2 and both table gradients.  The oracle runs in
float64 on the bf16 inputs with no intermediate rounding, so the bound also
covers the bf16 rounding of h, z, y and the GEMM outputs on the GPU side.
The 32-sequence layer workload runs at full size and is checked on every
token row and on its full weight and table gradients.
"""
import numpy as np
import pytest
import torch

from oracle import layer as layer_oracle
from oracle import oracle
from paper_2605_13433_amd import hstu, inputs
from tests.gpu_util import check, say, to_dev

pytestmark = pytest.mark.gpu

TOL = 2e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.build(force=False)


def run_layer(w, bwd=True):
    e = w.extra
    x, w1, w2 = to_dev(e["x"]), to_dev(e["w1"]), to_dev(e["w2"])
    off = to_dev(w.seq_offsets)
    pos, tw, ts = to_dev(w.pos_w), to_dev(w.time_w), to_dev(w.timestamps)
    plan = hstu.LayerPlan(x, off, w.N, w.H, w.d, pos, tw, ts, w.num_buckets,
                          backward=bwd)
    f = plan.forward(x, w1, w2, off)
    got = dict(out=f.out, h=f.h, u=f.z[0], v=f.z[1], q=f.z[2], k=f.z[3], o=f.o, y=f.y)
    if bwd:
        g = plan.backward(x, w1, w2, off, to_dev(e["dout"]))
        got.update(dx=g.dx, dw1=g.dw1, dw2=g.dw2, d_pos=g.d_pos_w, d_time=g.d_time_w)
    torch.cuda.synchronize()
    return {n: (None if t is None else t.detach().to("cpu", torch.float64).numpy())
            for n, t in got.items()}


def compare_layer(w, got, ref, rows=None, sums=True):
    f = ref["fwd"]
    sel = (lambda a: a) if rows is None else (lambda a: a[rows])
    for n in ("out", "h", "u", "v", "q", "k", "o", "y"):
        check(n, sel(got[n]), f[n], TOL)
    check("dx", sel(got["dx"]), ref["dx"], TOL)
    if sums:
        check("dw1", got["dw1"], ref["dw1"], TOL)
        check("dw2", got["dw2"], ref["dw2"], TOL)
        if w.pos_w is not None:
            check("d_pos", got["d_pos"], ref["d_pos"], TOL)
        if w.time_w is not None:
            check("d_time", got["d_time"], ref["d_time"], TOL)


SMALL = [
    # lengths, H, d, N, D, pos, time
    ([1, 70, 130, 0, 64], 2, 64, 160, 128, True, True),
    ([300, 64, 129], 4, 128, 512, 512, True, True),     # the layer workload's head geometry
    ([5, 200, 63], 1, 128, 256, 64, True, False),       # d_model < H*d
    ([17, 90], 2, 64, 128, 40, False, True),            # d_model not a multiple of 64
]


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_layer_small(case):
    lengths, H, d, N, D, pos, time = SMALL[case]
    say(f"layer case {case}: lengths={lengths} H={H} d={d} N={N} D={D} pos={pos} time={time}")
    w = inputs.make_workload(lengths, H=H, d=d, N=N, pos=pos, time=time,
                             seed=300 + case, layer_dim=D)
    got = run_layer(w)
    compare_layer(w, got, layer_oracle.layer_bwd_workload(w))


def test_layer_split_k_weight_gradients():
    """Enough tokens (T = 2 x 1050 + 1) that dW1 and dW2 run as split-K
    products (two row blocks in one strided batch plus a one-row
    remainder), checked in full against the oracle."""
    lengths = [700, 700, 701]
    say(f"layer split-K: lengths={lengths}")
    w = inputs.make_workload(lengths, H=1, d=64, N=704, seed=320, layer_dim=64)
    got = run_layer(w)
    compare_layer(w, got, layer_oracle.layer_bwd_workload(w))


def test_layer_split_backward_d64():
    """A d=64 layer on enough tiles that the attention backward runs as the
    dK/dV and dQ launches (not the combined one): the dQ kernel's fused
    silu' store into dh, checked with every other output against the
    oracle."""
    rng = np.random.default_rng(78)
    lengths = [900] + rng.integers(20, 141, size=600).tolist()
    w = inputs.make_workload(lengths, H=4, d=64, N=960, seed=321, layer_dim=128)
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    assert hstu.max_entries(w.B, w.N, w.T) * w.H >= 4 * 4 * n_cu
    say(f"layer split backward d=64: B={w.B} T={w.T}")
    got = run_layer(w)
    compare_layer(w, got, layer_oracle.layer_bwd_workload(w))


def test_layer_workload4_full():
    """The 32-sequence layer workload (lengths to 4096) at full size: every
    token row, both weight gradients and both tables against the oracle."""
    w = inputs.workload(4)
    say(f"layer workload {w.name}: T={w.T} pairs/head={w.pairs} max L={int(w.lengths.max())}")
    got = run_layer(w)
    for n, a in got.items():
        if a is not None:
            assert np.all(np.isfinite(a)), f"non-finite values in {n}"
    compare_layer(w, got, layer_oracle.layer_bwd_workload(w))


def test_layer_routes_planes_into_attention_bitwise():
    """The layer's o and y equal a direct attention call on its own U, V, Q, K
    planes, bit for bit (the planes reach the right attention arguments)."""
    w = inputs.make_workload([100, 37, 64], H=2, d=64, N=128, seed=310, layer_dim=128)
    say("layer -> attention plane routing (bitwise)")
    e = w.extra
    x, w1, w2, off = to_dev(e["x"]), to_dev(e["w1"]), to_dev(e["w2"]), to_dev(w.seq_offsets)
    pos, tw, ts = to_dev(w.pos_w), to_dev(w.time_w), to_dev(w.timestamps)
    lp = hstu.LayerPlan(x, off, w.N, w.H, w.d, pos, tw, ts, w.num_buckets, backward=False)
    f = lp.forward(x, w1, w2, off)
    z = f.z
    ap = hstu.Plan(z[2], off, w.N, pos, tw, ts, w.num_buckets, backward=False)
    a = ap.forward(z[2], z[3], z[1], z[0], off)
    torch.cuda.synchronize()
    assert torch.equal(a.o, f.o) and torch.equal(a.y, f.y)


def test_layer_empty_batch_zero_gradients():
    w = inputs.make_workload([0, 0], H=2, d=64, N=64, seed=320, layer_dim=64)
    say("layer with T = 0: weight and table gradients written as zeros")
    e = w.extra
    dev = "cuda"
    x = torch.empty(0, 64, dtype=torch.bfloat16, device=dev)
    w1, w2, off = to_dev(e["w1"]), to_dev(e["w2"]), to_dev(w.seq_offsets)
    pos, tw = to_dev(w.pos_w), to_dev(w.time_w)
    ts = torch.empty(0, dtype=torch.int64, device=dev)
    lp = hstu.LayerPlan(x, off, w.N, w.H, w.d, pos, tw, ts, w.num_buckets)
    lp.forward(x, w1, w2, off)
    for t in (lp.grad.dw1, lp.grad.dw2, lp.grad.d_pos_w, lp.grad.d_time_w):
        t.fill_(7.0)
    g = lp.backward(x, w1, w2, off, torch.empty(0, 64, dtype=torch.bfloat16, device=dev))
    torch.cuda.synchronize()
    for t in (g.dw1, g.dw2, g.d_pos_w, g.d_time_w):
        assert torch.count_nonzero(t).item() == 0
