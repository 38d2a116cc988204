"""The C-ABI library loads, exports every declared symbol and validates its
arguments on the host (no GPU needed: every case below is rejected before
the library touches a device)."""
import ctypes
import os
import re

import pytest

from paper_2605_13433_amd import hstu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", f) for f in sorted(os.listdir(os.path.join(ROOT, "include")))
           if f.endswith(".h")]

pytestmark = pytest.mark.skipif(not os.path.exists(hstu.LIB_PATH),
                                reason="libhstu_jagged.so not built")


def declared_functions():
    src = "\n".join(open(h).read() for h in HEADERS)
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(hstu_\w+)\s*\(", src, flags=re.M)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert {"hstu_jagged_attn_fwd", "hstu_jagged_attn_bwd",
            "hstu_jagged_attn_workspace_bytes", "hstu_last_error",
            "hstu_jagged_embedding_fwd", "hstu_jagged_embedding_bwd",
            "hstu_jagged_embedding_bwd_workspace_bytes"} <= set(names)
    lib = ctypes.CDLL(hstu.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert hstu.load_library().hstu_version().decode().startswith("hstu_jagged")


FAKE = 0x1000   # never dereferenced: every call below fails validation first


def _fwd(B=2, N=64, H=2, d=64, dtype=hstu.HSTU_BF16, T=10, rab=None, null=()):
    ptrs = {n: (None if n in null else FAKE) for n in ("q", "k", "v", "u", "off")}
    out = hstu.FwdOut(dtype, T, None if "y" in null else FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30)
    lib = hstu.load_library()
    return lib.hstu_jagged_attn_fwd(ptrs["q"], ptrs["k"], ptrs["v"], ptrs["u"], ptrs["off"],
                                    B, N, H, d, ctypes.byref(rab) if rab else None,
                                    ctypes.byref(out), None)


@pytest.mark.parametrize("kw,code,frag", [
    (dict(B=-1), -1, "B = -1"),
    (dict(H=0), -1, "H = 0"),
    (dict(N=0), -1, "max_len"),
    (dict(d=48), -1, "d = 48"),
    (dict(d=32), -2, "bf16"),
    (dict(dtype=7), -1, "dtype"),
    (dict(T=-3), -1, "total_tokens"),
    (dict(B=0, T=5), -1, "B = 0"),
    (dict(N=70000), -2, "max_len"),
    (dict(H=65), -2, "H = 65"),
    (dict(null=("q",)), -1, "non-null"),
    (dict(null=("q",), T=0), 0, ""),
    (dict(null=("off",)), -1, "non-null"),
    (dict(null=("y",)), -1, "out->y"),
])
def test_fwd_validation(kw, code, frag):
    assert _fwd(**kw) == code
    assert frag in hstu.last_error()


def test_rab_validation():
    r = hstu.Rab(None, FAKE, None, 128)
    assert _fwd(rab=r) == -1 and "timestamps" in hstu.last_error()
    r = hstu.Rab(None, FAKE, FAKE, 0)
    assert _fwd(rab=r) == -1 and "num_buckets" in hstu.last_error()
    r = hstu.Rab(None, FAKE, FAKE, 1025)
    assert _fwd(H=4, rab=r) == -2 and "4096" in hstu.last_error()


def test_empty_batch_is_noop_without_device():
    # T = 0 forward enqueues nothing and touches no device
    assert _fwd(B=3, T=0) == 0
    assert _fwd(B=0, T=0) == 0


def test_bwd_validation():
    lib = hstu.load_library()
    io = hstu.BwdIO(hstu.HSTU_BF16, 10, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                    None, None, FAKE, 1 << 30)
    r = hstu.Rab(FAKE, None, None, 0)
    rc = lib.hstu_jagged_attn_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, 2, 64, 2, 64,
                                  ctypes.byref(r), ctypes.byref(io), None)
    assert rc == -1 and "d_pos_w" in hstu.last_error()
    io.du = None
    rc = lib.hstu_jagged_attn_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, 2, 64, 2, 64, None,
                                  ctypes.byref(io), None)
    assert rc == -1
    assert lib.hstu_jagged_attn_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, 2, 64, 2, 64, None,
                                    None, None) == -1


def test_workspace_query_rejects_bad_sizes():
    lib = hstu.load_library()
    assert lib.hstu_jagged_attn_workspace_bytes(2, 64, 2, 48, 10, 0, 0, None) == 0
    assert "d = 48" in hstu.last_error()


def _layer_fwd(B=2, N=64, H=2, d=64, D=128, dtype=hstu.HSTU_BF16, T=10, null=()):
    p = {n: (None if n in null else FAKE) for n in ("x", "w1", "w2", "off", "z", "out")}
    out = hstu.LayerFwdOut(dtype, T, p["out"], FAKE, p["z"], FAKE, FAKE, FAKE, FAKE,
                           FAKE, 1 << 40)
    return hstu.load_library().hstu_layer_fwd(p["x"], p["w1"], p["w2"], p["off"], B, N, H,
                                              d, D, None, ctypes.byref(out), None)


@pytest.mark.parametrize("kw,code,frag", [
    (dict(dtype=hstu.HSTU_F32), -2, "HSTU_BF16 only"),
    (dict(D=12), -1, "d_model = 12"),
    (dict(D=0), -1, "d_model = 0"),
    (dict(D=65544), -1, "d_model"),
    (dict(d=32), -2, "bf16"),
    (dict(H=0), -1, "H = 0"),
    (dict(null=("x",)), -1, "x, w1 and w2"),
    (dict(null=("w2",)), -1, "x, w1 and w2"),
    (dict(null=("z",)), -1, "non-null"),
    (dict(null=("out",)), -1, "out->out"),
    (dict(null=("x", "w1", "w2", "z", "out"), T=0), 0, ""),
])
def test_layer_fwd_validation(kw, code, frag):
    assert _layer_fwd(**kw) == code
    assert frag in hstu.last_error()


def test_layer_bwd_validation():
    lib = hstu.load_library()
    io = hstu.LayerBwdIO(hstu.HSTU_BF16, 10, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                         FAKE, None, FAKE, None, None, FAKE, 1 << 40)
    rc = lib.hstu_layer_bwd(FAKE, FAKE, FAKE, FAKE, 2, 64, 2, 64, 128, None,
                            ctypes.byref(io), None)
    assert rc == -1 and "dw1" in hstu.last_error()
    io.dw1 = FAKE
    r = hstu.Rab(FAKE, None, None, 0)
    rc = lib.hstu_layer_bwd(FAKE, FAKE, FAKE, FAKE, 2, 64, 2, 64, 128, ctypes.byref(r),
                            ctypes.byref(io), None)
    assert rc == -1 and "d_pos_w" in hstu.last_error()
    io.dx = None
    rc = lib.hstu_layer_bwd(FAKE, FAKE, FAKE, FAKE, 2, 64, 2, 64, 128, None,
                            ctypes.byref(io), None)
    assert rc == -1 and "dx" in hstu.last_error()
    assert lib.hstu_layer_bwd(FAKE, FAKE, FAKE, FAKE, 2, 64, 2, 64, 128, None,
                              None, None) == -1


def test_layer_workspace_query_rejects_bad_sizes():
    lib = hstu.load_library()
    assert lib.hstu_layer_workspace_bytes(2, 64, 2, 64, 100, 10, 1, 0, None) == 0
    assert "d_model = 100" in hstu.last_error()
    assert lib.hstu_layer_workspace_bytes(2, 64, 2, 64, 128, 10, 0, 1, None) == 0
    assert "HSTU_BF16" in hstu.last_error()


def test_alpha_must_be_finite():
    lib = hstu.load_library()
    for bad in (float("nan"), float("inf"), -float("inf")):
        r = hstu.Rab(FAKE, None, None, 0, bad)
        out = hstu.FwdOut(hstu.HSTU_BF16, 10, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30)
        rc = lib.hstu_jagged_attn_fwd(FAKE, FAKE, FAKE, FAKE, FAKE, 2, 64, 2, 64,
                                      ctypes.byref(r), ctypes.byref(out), None)
        assert rc == -1 and "alpha" in hstu.last_error()
