"""CPU-side checks of the C ABI: the library loads, exports every declared symbol, and
rejects bad arguments on the host before touching a device (no compute calls here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "imbd.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b([a-z_][a-z0-9_]*)\s*\([^;{]*\)\s*;", text)
    return sorted(set(n for n in names if n not in ("sizeof",)))


@pytest.fixture(scope="module")
def lib():
    import paper_1712_04432_amd as m
    return m.load()


def test_header_declares_the_boundary():
    names = _declared_functions()
    for n in ("mlp_fwd", "mlp_bwd", "sgd_step", "mlp_local_fwd", "mlp_local_bwd", "softmax_xent",
              "cast_f32_bf16", "conv3x3_tile_fwd", "conv3x3_tile_dgrad", "conv3x3_tile_wgrad",
              "mlp_workspace_bytes", "imbd_status_string"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    from paper_1712_04432_amd._abi import SIGNATURES
    for n in _declared_functions():
        assert hasattr(lib, n), n
        assert n in SIGNATURES, f"{n} is declared but not bound in Python"


def test_status_strings(lib):
    assert lib.imbd_status_string(0) == b"ok"
    assert lib.imbd_status_string(-1) == b"invalid argument"
    assert lib.imbd_status_string(12345) == b"unknown status"
    assert lib.imbd_version() >= 100


def test_workspace_sizing_and_offsets():
    import paper_1712_04432_amd as m
    net = m.MLP((784, 256, 128, 10), 64, "f32")
    n = m.mlp_workspace_bytes(net)
    offs = [m.mlp_workspace_offset(net, m.IMBD_WS_ACT, 1), m.mlp_workspace_offset(net, m.IMBD_WS_ACT, 2),
            m.mlp_workspace_offset(net, m.IMBD_WS_LOGITS), m.mlp_workspace_offset(net, m.IMBD_WS_DY, 1),
            m.mlp_workspace_offset(net, m.IMBD_WS_DY, 3), m.mlp_workspace_offset(net, m.IMBD_WS_ROWLOSS)]
    assert all(o % 256 == 0 for o in offs)
    assert offs == sorted(offs) and offs[-1] + 64 * 4 <= n
    # regions do not overlap
    assert offs[1] - offs[0] >= 64 * 256 * 4
    with pytest.raises(m.ImbdError):
        m.mlp_workspace_offset(net, m.IMBD_WS_ACT, 3)      # the top layer has logits, not X_{L+1}
    with pytest.raises(m.ImbdError):
        m.mlp_workspace_offset(net, 9, 1)
    big = m.MLP((9216, 4096, 4096, 1000), 256, "bf16")
    assert m.mlp_workspace_bytes(big) > 256 * (4096 * 2 + 1000) * 2


@pytest.mark.parametrize("desc", [
    dict(dims=(), batch=4),                 # no layers
    dict(dims=(4, 0, 2), batch=4),          # zero width
    dict(dims=(4, 3), batch=0),             # empty batch: the mean of Eq. (1) is undefined
    dict(dims=(4, 3), batch=4, dtype=7),    # unknown dtype
])
def test_bad_descriptions_are_rejected(lib, desc):
    from paper_1712_04432_amd._abi import MlpDesc
    dims = desc["dims"]
    arr = (ctypes.c_int * max(len(dims), 1))(*dims)
    d = MlpDesc(max(len(dims) - 1, 0), arr, desc["batch"], desc.get("dtype", 1))
    assert lib.mlp_workspace_bytes(ctypes.byref(d)) == 0
    assert lib.mlp_fwd(ctypes.byref(d), None, None, None, None, 0, None, None) == -1
    assert lib.imbd_last_error() != b""


def test_validation_errors_before_any_launch(lib):
    import paper_1712_04432_amd as m
    net = m.MLP((8, 4, 2), 4, "bf16")
    # null layer array
    assert lib.mlp_fwd(net.desc, None, ctypes.c_void_p(16), ctypes.c_void_p(16), ctypes.c_void_p(256), 1 << 20,
                       ctypes.c_void_p(16), None) == m.IMBD_EINVAL
    # SGD: negative count, NaN learning rate, bf16 copy with a wrong type code
    assert lib.sgd_step(ctypes.c_void_p(16), None, 1, ctypes.c_void_p(16), -1, 0.1, 1.0, None) == m.IMBD_EINVAL
    assert lib.sgd_step(ctypes.c_void_p(16), None, 1, ctypes.c_void_p(16), 4, float("nan"), 1.0, None) == m.IMBD_EINVAL
    assert lib.sgd_step(ctypes.c_void_p(16), ctypes.c_void_p(16), 0, ctypes.c_void_p(16), 4, 0.1, 1.0, None) == m.IMBD_EINVAL
    assert lib.sgd_step(None, None, 1, None, 0, 0.1, 1.0, None) == m.IMBD_OK      # n == 0 is a no-op
    assert lib.cast_f32_bf16(None, None, -3, None) == m.IMBD_EINVAL
    assert lib.cast_f32_bf16(None, None, 0, None) == m.IMBD_OK
    # softmax: ld smaller than the row
    assert lib.softmax_xent(4, 10, ctypes.c_void_p(16), 5, ctypes.c_void_p(16), 0.25, ctypes.c_void_p(16),
                            ctypes.c_void_p(16), None, 10, 0, None) == m.IMBD_EINVAL
    # local blocks: bad grid, ld < row, unknown dtype
    p = ctypes.c_void_p(256)
    assert lib.mlp_local_fwd(1, 0, 0, 4, 8, 8, 4, p, 8, None, p, 8, p, 8, 1, None, 0, None) == m.IMBD_EINVAL
    assert lib.mlp_local_fwd(1, 0, 2, 4, 8, 8, 4, p, 7, None, p, 8, p, 8, 1, None, 0, None) == m.IMBD_EINVAL
    assert lib.mlp_local_fwd(5, 0, 2, 4, 8, 8, 4, p, 8, None, p, 8, p, 8, 1, None, 0, None) == m.IMBD_EINVAL
    assert lib.mlp_local_bwd(1, 2, 4, 8, 8, 4, p, 8, p, 8, p, 8, None, 8, None, None, 8, 0, None, 0,
                             None) == m.IMBD_EINVAL                              # dw_part missing
    assert lib.mlp_local_fwd(1, 0, 2, 4, 8, 8, 0, None, 0, None, None, 0, None, 0, 1, None, 0, None) == m.IMBD_OK
    # conv: bad sizes
    assert lib.conv3x3_tile_fwd(1, 0, 4, 8, 8, p, p, p, 1, None) == m.IMBD_EINVAL
    assert lib.imbd_timing_end(None, None) == m.IMBD_EINVAL


def test_workspace_too_small_is_reported(lib):
    import paper_1712_04432_amd as m
    net = m.MLP((8, 4, 2), 4, "bf16")
    layers = m._layers([{"w": _Fake(256), "w_lp": _Fake(512), "b": _Fake(768)}] * 2)
    rc = lib.mlp_fwd(net.desc, layers, ctypes.c_void_p(256), ctypes.c_void_p(256), ctypes.c_void_p(256), 16,
                     ctypes.c_void_p(256), None)
    assert rc == m.IMBD_EWORKSPACE
    assert b"workspace" in lib.imbd_last_error()


class _Fake:
    """Stands in for a tensor on the host-validation path (only data_ptr is read)."""

    def __init__(self, addr):
        self.addr = addr

    def data_ptr(self):
        return self.addr
