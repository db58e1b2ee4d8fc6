"""ctypes declarations of include/imbd.h (one-to-one with the C ABI)."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libimbd.so")

IMBD_OK, IMBD_EINVAL, IMBD_EUNSUPPORTED, IMBD_EHIP, IMBD_EWORKSPACE = 0, -1, -2, -3, -4
IMBD_F32, IMBD_BF16 = 0, 1
IMBD_WS_ACT, IMBD_WS_LOGITS, IMBD_WS_DY, IMBD_WS_ROWLOSS = 0, 1, 2, 3
(IMBD_OPT_SKINNY_OFF, IMBD_OPT_SKINNY_SPLITS, IMBD_OPT_TOP_UNFUSED, IMBD_OPT_WIDE_OFF, IMBD_OPT_WIDE_SPLITS,
 IMBD_OPT_DW_WIDE_MIN_K, IMBD_OPT_DW_STREAM, IMBD_OPT_DW_GENERIC, IMBD_OPT_GEMM_CFG, IMBD_OPT_GEMM_SPLITS,
 IMBD_OPT_CONV_NT, IMBD_OPT_SKINNY_NB, IMBD_OPT_DW_WIDE_DUAL, IMBD_OPT_LOCAL_PAIR,
 IMBD_OPT_REDUCE_TAIL) = range(15)
IMBD_OPT_COUNT = 15
IMBD_STATIC_SCRATCH_BYTES = 64 << 20
(IMBD_K_GEMM_FWD, IMBD_K_GEMM_DX, IMBD_K_GEMM_DW, IMBD_K_SPLITK, IMBD_K_SOFTMAX, IMBD_K_BIAS,
 IMBD_K_SGD, IMBD_K_CAST, IMBD_K_CONV_FWD, IMBD_K_CONV_DGRAD, IMBD_K_CONV_WGRAD) = range(11)

# every function the header declares: name -> (restype, argtypes)
_i, _l, _p, _f, _d, _z = ctypes.c_int, ctypes.c_int64, ctypes.c_void_p, ctypes.c_float, ctypes.c_double, ctypes.c_size_t


class MlpDesc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int), ("dims", ctypes.POINTER(ctypes.c_int)),
                ("batch", ctypes.c_int), ("dtype", ctypes.c_int)]


class Layer(ctypes.Structure):
    _fields_ = [("w", _p), ("w_lp", _p), ("b", _p), ("dw", _p), ("db", _p)]


_PD = ctypes.POINTER(MlpDesc)
_PL = ctypes.POINTER(Layer)

SIGNATURES = {
    "imbd_status_string": (ctypes.c_char_p, [_i]),
    "mlp_status_string": (ctypes.c_char_p, [_i]),
    "imbd_last_error": (ctypes.c_char_p, []),
    "imbd_version": (_i, []),
    "mlp_workspace_bytes": (_z, [_PD]),
    "mlp_workspace_offset": (_l, [_PD, _i, _i]),
    "mlp_fwd": (_i, [_PD, _PL, _p, _p, _p, _z, _p, _p]),
    "mlp_bwd": (_i, [_PD, _PL, _p, _p, _z, _i, _f, _p, _p]),
    "mlp_train_step": (_i, [_PD, _PL, _p, _p, _p, _z, _f, _p, _p]),
    "mlp_train_step_static": (_i, [_PD, _PL, _p, _p, _f, _p, _p]),
    "sgd_step": (_i, [_p, _p, _i, _p, _l, _f, _f, _p]),
    "cast_f32_bf16": (_i, [_p, _p, _l, _p]),
    "softmax_xent": (_i, [_i, _i, _p, _l, _p, _f, _p, _p, _p, _l, _i, _p]),
    "mlp_local_fwd": (_i, [_i, _i, _i, _i, _i, _i, _i, _p, _l, _p, _p, _l, _p, _l, _i, _p, _z, _p]),
    "mlp_local_bwd": (_i, [_i, _i, _i, _i, _i, _i, _p, _l, _p, _l, _p, _l, _p, _l, _p, _p, _l, _i,
                           _p, _z, _p]),
    "mlp_local_workspace_bytes": (_z, [_i, _i, _i, _i, _i]),
    "conv3x3_tile_fwd": (_i, [_i, _i, _i, _i, _i, _p, _p, _p, _i, _p]),
    "conv3x3_tile_dgrad": (_i, [_i, _i, _i, _i, _i, _p, _p, _p, _i, _p]),
    "conv3x3_tile_wgrad": (_i, [_i, _i, _i, _i, _i, _p, _p, _p, _p, _z, _p]),
    "conv3x3_wgrad_workspace_bytes": (_z, [_i, _i, _i, _i, _i]),
    "conv3x3_tile_bwd": (_i, [_i, _i, _i, _i, _i, _p, _p, _p, _p, _i, _p, _p, _z, _p]),
    "imbd_set_option": (_i, [_i, _i]),
    "imbd_get_option": (_i, [_i, ctypes.POINTER(ctypes.c_int)]),
    "imbd_option_name": (ctypes.c_char_p, [_i]),
    "imbd_timing_begin": (_i, [_i, _i, _i]),
    "imbd_timing_end": (_i, [ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_double)]),
}

_lib = None


def load(path: str = LIB_PATH):
    """Load libimbd.so. Raises if it has not been built: there is no fallback path."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing; build it with `python -m paper_1712_04432_amd.build`")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


class ImbdError(RuntimeError):
    def __init__(self, status: int, where: str):
        lib = load()
        msg = lib.imbd_last_error().decode()
        super().__init__(f"{where}: {lib.imbd_status_string(status).decode()} ({status}): {msg}")
        self.status = status


def check(status: int, where: str) -> int:
    if status != IMBD_OK:
        raise ImbdError(status, where)
    return status
