"""Host-side argument checks of the embedding lookup C ABI (no GPU needed:
every case below is rejected before the library touches a device)."""
import ctypes
import os

import pytest

from paper_2605_13433_amd import embedding as emb
from paper_2605_13433_amd import hstu

pytestmark = pytest.mark.skipif(not os.path.exists(hstu.LIB_PATH),
                                reason="libhstu_jagged.so not built")

FAKE = 0x1000   # never dereferenced


def _desc(**kw):
    d = dict(dtype=hstu.HSTU_F32, num_tables=2, dim=128, row_offsets=FAKE, id_offsets=FAKE,
             total_rows=100, num_ids=10, layout=emb.HSTU_EMB_FLAT)
    d.update(kw)
    return emb.EmbDesc(d["dtype"], d["num_tables"], d["dim"], d["row_offsets"],
                       d["id_offsets"], d["total_rows"], d["num_ids"], d["layout"])


@pytest.mark.parametrize("kw,frag", [
    (dict(dtype=5), "dtype"),
    (dict(num_tables=-1), "num_tables"),
    (dict(num_tables=2000), "num_tables"),
    (dict(dim=12), "dim"),
    (dict(dim=0), "dim"),
    (dict(dim=8192), "dim"),
    (dict(num_ids=-2), "num_ids"),
    (dict(num_ids=1 << 31), "num_ids"),
    (dict(total_rows=-1), "total_rows"),
    (dict(layout=3), "layout"),
    (dict(num_tables=0), "no tables"),
    (dict(layout=emb.HSTU_EMB_TOKEN, num_tables=3), "multiple"),
    (dict(row_offsets=None), "non-null"),
])
def test_invalid_descriptor(kw, frag):
    lib = emb._lib()
    d = _desc(**kw)
    rc = lib.hstu_jagged_embedding_fwd(ctypes.byref(d), FAKE, FAKE, FAKE, None)
    assert rc == -1
    assert frag in hstu.last_error()
    rc = lib.hstu_jagged_embedding_bwd(ctypes.byref(d), FAKE, FAKE, FAKE, None, None,
                                       FAKE, 1 << 30, None)
    assert rc == -1 and frag in hstu.last_error()
    assert lib.hstu_jagged_embedding_bwd_workspace_bytes(ctypes.byref(d)) == 0


def test_null_tensors_rejected():
    lib = emb._lib()
    d = _desc()
    assert lib.hstu_jagged_embedding_fwd(ctypes.byref(d), None, FAKE, FAKE, None) == -1
    assert "non-null" in hstu.last_error()


def test_empty_forward_is_a_no_op():
    lib = emb._lib()
    d = _desc(num_ids=0)
    assert lib.hstu_jagged_embedding_fwd(ctypes.byref(d), None, None, None, None) == 0
