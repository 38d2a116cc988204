"""GPU parity of the jagged embedding lookup against the CPU oracle.

Forward rows are copies, so they are compared bit for bit; the distinct-row
list and count of the backward are compared exactly; the float32 gradient
sums against the float64 oracle at max|gpu - ref| <= 1e-5 max|ref|.  Rows no
valid id touches must keep what the caller left in the gradient buffer (a
NaN fill here).  Cases: flat and token layouts, float32 and bf16, row
widths 8 .. 512 (including 136, whose 34 slices per row do not divide a
work-group), invalid ids, empty tables, runs of one row that start, end and
span 32-position chunk boundaries, a row repeated 5000 times, determinism
(two backward calls give identical bits), and the full multi-table sequence
batch.
"""
import numpy as np
import pytest
import torch

from oracle import embedding as E
from paper_2605_13433_amd import emb_inputs
from paper_2605_13433_amd import embedding as emb
from tests.gpu_util import say

pytestmark = pytest.mark.gpu

TOL = 1e-5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def run(b, layout="flat", dout=None):
    """Forward and backward of batch `b` through the C ABI."""
    dev = "cuda"
    W = b.weights.to(dev)
    ids = b.ids.to(dev)
    ro, io = b.row_offsets.to(dev), b.id_offsets.to(dev)
    p = emb.plan(W, ro, io, b.total_rows, b.n, layout)
    out = emb.lookup(p, W, ids)
    if dout is None:
        dout = b.dout if layout == "flat" else emb_inputs.token_layout(b.dout, b.F)
    g = torch.full((b.total_rows, b.D), float("nan"), device=dev)
    uniq = torch.full((max(b.n, 1),), -7, dtype=torch.int64, device=dev)
    cnt = torch.full((1,), -7, dtype=torch.int32, device=dev)
    emb.lookup_backward(p, ids, dout.contiguous().to(dev), g, uniq, cnt)
    torch.cuda.synchronize()
    return out.cpu(), g.cpu(), uniq.cpu(), int(cnt.item()), p, (W, ids, dout)


def compare(b, layout="flat"):
    say(f"  case {b.name}: F={b.F} n={b.n} D={b.D} {b.dtype} layout={layout}")
    out, g, uniq, cnt, _, _ = run(b, layout)
    ref = E.embedding_fwd(b.weights, b.row_offsets, b.ids, b.id_offsets, layout)
    got = out.to(torch.float64).numpy()
    assert np.array_equal(got, ref), "forward rows differ"
    dout = b.dout if layout == "flat" else emb_inputs.token_layout(b.dout, b.F)
    rows, grads = E.embedding_bwd(dout, b.row_offsets, b.ids, b.id_offsets, layout)
    assert cnt == len(rows), (cnt, len(rows))
    assert np.array_equal(uniq[:cnt].numpy(), rows)
    gd = g.to(torch.float64).numpy()
    touched = gd[rows]
    assert np.isfinite(touched).all()
    scale = np.abs(grads).max() if grads.size else 1.0
    err = np.abs(touched - grads).max() / scale if grads.size else 0.0
    say(f"    grad max|gpu-ref|/max|ref| = {err:.3e} over {len(rows)} rows")
    assert err <= TOL
    mask = np.ones(b.total_rows, dtype=bool)
    mask[rows] = False
    assert np.isnan(gd[mask]).all(), "an untouched row was written"
    return out, g


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("D", [8, 64, 128, 136, 512])
def test_small_flat(dtype, D):
    b = emb_inputs.make_batch((5, 300, 1, 77), (40, 700, 9, 0), D, dtype, seed=D, alpha=1.1,
                              name=f"small_D{D}")
    ids = b.ids.clone()
    ids[3], ids[50], ids[700] = -1, 300, 10 ** 9          # invalid ids
    b.ids = ids
    compare(b)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_token_layout(dtype):
    b = emb_inputs.make_batch((64, 1 << 12, 3), (333, 333, 333), 128, dtype, seed=3,
                              name="token3")
    compare(b, "token")


def test_runs_across_chunk_boundaries():
    # sorted runs [0,31) [31,64) [64,128) [128,129) [129,161) then a long run
    ids = [0] * 31 + [1] * 33 + [2] * 64 + [3] + [4] * 32 + [5] * 5000 + [6] * 3
    rng = np.random.default_rng(0)
    ids = np.array(ids)[rng.permutation(len(ids))]
    for dtype in (torch.float32, torch.bfloat16):
        b = emb_inputs.make_batch((8,), (len(ids),), 128, dtype, seed=1, ids=ids,
                                  name="runs")
        compare(b)


def test_backward_is_deterministic():
    b = emb_inputs.make_batch((1 << 10, 16), (20000, 20000), 128, torch.float32, seed=9,
                              alpha=1.2, name="det")
    _, g1, u1, c1, p, (W, ids, dout) = run(b)
    g2 = torch.full_like(g1, float("nan"), device="cuda")
    emb.lookup_backward(p, ids, dout.contiguous().cuda(), g2)
    torch.cuda.synchronize()
    g2 = g2.cpu()
    rows = u1[:c1]
    assert torch.equal(g1[rows].view(torch.int32), g2[rows].view(torch.int32))


def test_degenerate():
    # every id invalid: zero rows, nothing touched
    b = emb_inputs.make_batch((4, 4), (3, 2), 64, torch.float32, seed=0,
                              ids=[-1, 4, 99, 7, -3], name="all_invalid")
    out, g, uniq, cnt, _, _ = run(b)
    assert cnt == 0 and not out.any() and torch.isnan(g).all()
    # an empty table between two others
    b = emb_inputs.make_batch((10, 20, 30), (50, 0, 60), 64, torch.bfloat16, seed=2,
                              name="empty_middle")
    compare(b)
    # no ids at all
    b = emb_inputs.make_batch((10,), (0,), 64, torch.float32, seed=0, name="no_ids")
    out, g, uniq, cnt, _, _ = run(b)
    assert cnt == 0 and out.numel() == 0


_FULL = {}


def _full_batch(dtype):
    # drawn once (about 20 s for 2.9 GB of weights); the bf16 batch is the
    # same draw rounded, exactly as sequence_batch(dtype=bf16) produces it
    if "f32" not in _FULL:
        _FULL["f32"] = emb_inputs.sequence_batch(dtype=torch.float32)
    b = _FULL["f32"]
    if dtype == torch.float32:
        return b
    import dataclasses
    return dataclasses.replace(b, weights=b.weights.to(dtype), dout=b.dout.to(dtype),
                               dtype=dtype, name=b.name.replace("f32", "bf16"))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_sequence_batch_full(dtype):
    """The benchmark's batch: 8 tables (128 .. 4 M rows), 32 sequences of up
    to 4160 tokens, D = 128, token-major output; every row of both passes."""
    compare(_full_batch(dtype), "token")
