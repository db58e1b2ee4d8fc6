"""CPU-side checks of the C ABI: the library loads, exports every declared symbol, and
rejects bad arguments on the host before touching a device (no compute calls here)."""
import ctypes

import numpy as np
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


def test_workspace_regions_of_random_networks():
    """For seeded random networks (2-5 layers, widths 1-5000, batches 1-3000, fp32 and bf16),
    every workspace region is 256-byte aligned, lies inside the size the library reports
    and overlaps no other region; the split-K partials come after all of them."""
    import paper_1712_04432_amd as m
    rng = np.random.default_rng(2024)
    for _ in range(200):
        L = int(rng.integers(1, 5))
        dims = tuple(int(v) for v in rng.integers(1, 5001, size=L + 1))
        B = int(rng.integers(1, 3001))
        dt = "bf16" if rng.random() < 0.5 else "f32"
        esz = 2 if dt == "bf16" else 4
        net = m.MLP(dims, B, dt)
        total = m.mlp_workspace_bytes(net)
        regions = [(m.mlp_workspace_offset(net, m.IMBD_WS_ACT, i), B * dims[i] * esz) for i in range(1, L)]
        regions.append((m.mlp_workspace_offset(net, m.IMBD_WS_LOGITS, 0), B * dims[L] * 4))
        regions += [(m.mlp_workspace_offset(net, m.IMBD_WS_DY, i), B * dims[i] * esz) for i in range(1, L + 1)]
        regions.append((m.mlp_workspace_offset(net, m.IMBD_WS_ROWLOSS, 0), B * 4))
        regions.sort()
        for (o, n), (o2, _) in zip(regions, regions[1:] + [(total, 0)]):
            assert o % 256 == 0 and o + n <= o2, (dims, B, dt, o, n, o2)


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


_OPTION_DEFAULTS = {"SKINNY_OFF": 0, "SKINNY_SPLITS": 0, "TOP_UNFUSED": 0, "WIDE_OFF": 0, "WIDE_SPLITS": 0,
                    "DW_WIDE_MIN_K": 257, "DW_STREAM": 1, "DW_GENERIC": 0, "GEMM_CFG": -1, "GEMM_SPLITS": 0,
                    "CONV_NT": 1, "SKINNY_NB": 0, "DW_WIDE_DUAL": -1, "LOCAL_PAIR": 1, "REDUCE_TAIL": 1}


def _options_in_child(env_extra):
    """Option values seen by a fresh process whose environment has only env_extra of the
    IMBD_* variables."""
    import json
    import subprocess
    import sys
    env = {k: v for k, v in os.environ.items() if not k.startswith("IMBD_")}
    env.update(env_extra)
    code = ("import json, paper_1712_04432_amd as m\n"
            "print(json.dumps({m.option_name(k)[5:]: m.get_option(k) for k in range(m.IMBD_OPT_COUNT)}))")
    out = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                         check=True, timeout=120)
    return json.loads(out.stdout.strip().splitlines()[-1])


def test_options_defaults_and_environment_read_once():
    assert _options_in_child({}) == _OPTION_DEFAULTS
    got = _options_in_child({"IMBD_DW_WIDE_MIN_K": "500", "IMBD_WIDE_SPLITS": "3", "IMBD_CONV_NT": "7"})
    assert got["DW_WIDE_MIN_K"] == 500 and got["WIDE_SPLITS"] == 3
    assert got["CONV_NT"] == 1          # out of range: the default stays


def test_options_set_get_and_validation(lib, monkeypatch):
    import paper_1712_04432_amd as m
    assert m.option_name(m.IMBD_OPT_DW_WIDE_MIN_K) == "IMBD_DW_WIDE_MIN_K"
    assert m.option_name(m.IMBD_OPT_COUNT) == ""
    old = m.get_option(m.IMBD_OPT_WIDE_SPLITS)
    # the environment is not read after load
    monkeypatch.setenv("IMBD_WIDE_SPLITS", "5")
    assert m.get_option(m.IMBD_OPT_WIDE_SPLITS) == old
    with m.options(wide_splits=3, dw_stream=0):
        assert m.get_option(m.IMBD_OPT_WIDE_SPLITS) == 3 and m.get_option(m.IMBD_OPT_DW_STREAM) == 0
    assert m.get_option(m.IMBD_OPT_WIDE_SPLITS) == old and m.get_option(m.IMBD_OPT_DW_STREAM) == 1
    assert lib.imbd_set_option(m.IMBD_OPT_SKINNY_OFF, 2) == m.IMBD_EINVAL
    assert lib.imbd_set_option(m.IMBD_OPT_GEMM_CFG, -2) == m.IMBD_EINVAL
    assert lib.imbd_set_option(m.IMBD_OPT_COUNT, 0) == m.IMBD_EINVAL
    assert lib.imbd_set_option(-1, 0) == m.IMBD_EINVAL
    assert lib.imbd_get_option(0, None) == m.IMBD_EINVAL
    assert m.get_option(m.IMBD_OPT_SKINNY_OFF) == 0


def test_workspace_follows_a_split_option(lib):
    """A forced K split changes the partial sums a product needs; the workspace sized under
    the option covers it."""
    import paper_1712_04432_amd as m
    net = m.MLP((1032, 264, 136), 777, "bf16")
    base = m.mlp_workspace_bytes(net)
    with m.options(wide_splits=8):
        more = m.mlp_workspace_bytes(net)
    assert more > base and m.mlp_workspace_bytes(net) == base


def test_conv_bwd_validates_before_enqueueing(lib):
    import paper_1712_04432_amd as m
    p = ctypes.c_void_p(256)
    # dw missing; bad sizes; unknown dx dtype; workspace too small for the weight gradient
    assert lib.conv3x3_tile_bwd(2, 56, 56, 256, 256, p, p, p, p, 1, None, p, 1 << 30, None) == m.IMBD_EINVAL
    assert lib.conv3x3_tile_bwd(2, 0, 56, 256, 256, p, p, p, p, 1, p, p, 1 << 30, None) == m.IMBD_EINVAL
    assert lib.conv3x3_tile_bwd(2, 56, 56, 256, 256, p, p, p, p, 9, p, p, 1 << 30, None) == m.IMBD_EINVAL
    need = lib.conv3x3_wgrad_workspace_bytes(32, 56, 56, 256, 256)
    assert need > 0
    assert lib.conv3x3_tile_bwd(32, 56, 56, 256, 256, p, p, p, p, 1, p, p, need - 1, None) == m.IMBD_EWORKSPACE
    assert lib.mlp_status_string(-4) == lib.imbd_status_string(-4)


def test_static_scratch_refuses_oversized_network_on_the_host(lib):
    import paper_1712_04432_amd as m
    net = m.MLP((9216, 4096, 4096, 1000), 2048, "bf16")
    assert m.mlp_workspace_bytes(net) > m.IMBD_STATIC_SCRATCH_BYTES
    p = ctypes.c_void_p(256)
    layers = m._layers([{"w": _Fake(256), "w_lp": _Fake(512), "b": _Fake(768)}] * 3)
    assert lib.mlp_train_step_static(net.desc, layers, p, p, 0.01, p, None) == m.IMBD_EWORKSPACE
    assert b"static scratch" in lib.imbd_last_error()
    bad = m.MLP((8, 0, 2), 4, "bf16")
    assert lib.mlp_train_step_static(bad.desc, layers, p, p, 0.01, p, None) == m.IMBD_EINVAL
