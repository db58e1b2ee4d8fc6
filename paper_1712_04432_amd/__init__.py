"""Python binding of libimbd.so: the gfx950 hot path of integrated model/batch/domain
parallel SGD (Gholami et al., arXiv:1712.04432).

Functions carry the names of the C ABI in include/imbd.h and only marshal arguments:
torch tensors supply device pointers and the current HIP stream; every step of the path
runs in the library's kernels. Missing library -> RuntimeError (no fallback).

bf16 tensors are torch.bfloat16 (the bytes are bf16 bit patterns), fp32 tensors
torch.float32. Activations are [B][d] (one sample per row, the paper's column-major
X_i); weights [d_out][d_in].
"""
from __future__ import annotations

import ctypes

from ._abi import (IMBD_BF16, IMBD_F32, IMBD_K_BIAS, IMBD_K_CAST, IMBD_K_CONV_DGRAD,  # noqa: F401
                   IMBD_K_CONV_FWD, IMBD_K_CONV_WGRAD, IMBD_K_GEMM_DW, IMBD_K_GEMM_DX,
                   IMBD_K_GEMM_FWD, IMBD_K_SGD, IMBD_K_SOFTMAX, IMBD_K_SPLITK, IMBD_OK,
                   IMBD_EINVAL, IMBD_EUNSUPPORTED, IMBD_EHIP, IMBD_EWORKSPACE,
                   IMBD_WS_ACT, IMBD_WS_DY, IMBD_WS_LOGITS, IMBD_WS_ROWLOSS, ImbdError, Layer,
                   MlpDesc, check, load)
from ._abi import IMBD_STATIC_SCRATCH_BYTES  # noqa: F401
from ._abi import (IMBD_OPT_CONV_NT, IMBD_OPT_COUNT, IMBD_OPT_DW_GENERIC, IMBD_OPT_DW_STREAM,  # noqa: F401
                   IMBD_OPT_DW_WIDE_DUAL, IMBD_OPT_DW_WIDE_MIN_K, IMBD_OPT_LOCAL_PAIR, IMBD_OPT_GEMM_CFG, IMBD_OPT_GEMM_SPLITS, IMBD_OPT_SKINNY_OFF,
                   IMBD_OPT_SKINNY_NB, IMBD_OPT_SKINNY_SPLITS, IMBD_OPT_TOP_UNFUSED, IMBD_OPT_WIDE_OFF,
                   IMBD_OPT_WIDE_SPLITS, IMBD_OPT_REDUCE_TAIL)

__all__ = [
    "load", "ImbdError", "MLP", "mlp_workspace_bytes", "mlp_workspace_offset", "mlp_fwd",
    "mlp_bwd", "mlp_train_step", "mlp_train_step_static", "sgd_step", "cast_f32_bf16", "softmax_xent", "mlp_local_fwd",
    "mlp_local_bwd", "mlp_local_workspace_bytes", "conv3x3_tile_fwd", "conv3x3_tile_dgrad",
    "conv3x3_tile_wgrad", "conv3x3_tile_bwd", "conv3x3_wgrad_workspace_bytes", "timing_begin",
    "timing_end",
    "ws_view", "dtype_code", "set_option", "get_option", "option_name", "options",
]


def _torch():
    import torch
    return torch


def dtype_code(t_or_dtype) -> int:
    torch = _torch()
    dt = t_or_dtype.dtype if hasattr(t_or_dtype, "dtype") else t_or_dtype
    if dt == torch.bfloat16:
        return IMBD_BF16
    if dt == torch.float32:
        return IMBD_F32
    raise TypeError(f"unsupported dtype {dt}")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


class MLP:
    """Shape of a network: widths d_0..d_L, batch B, operand type ('bf16' or 'f32')."""

    def __init__(self, dims, batch: int, dtype: str = "bf16"):
        self.dims = [int(d) for d in dims]
        self.batch = int(batch)
        self.dtype = dtype
        self.code = IMBD_BF16 if dtype == "bf16" else IMBD_F32
        self._dims_arr = (ctypes.c_int * len(self.dims))(*self.dims)
        self._desc = MlpDesc(len(self.dims) - 1, self._dims_arr, self.batch, self.code)

    @property
    def n_layers(self):
        return len(self.dims) - 1

    @property
    def desc(self):
        return ctypes.byref(self._desc)

    def torch_dtype(self):
        torch = _torch()
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32


def _layers(layers):
    """layers: sequence of dicts with keys w, w_lp, b, (dw, db) -> ctypes Layer array."""
    arr = (Layer * len(layers))()
    for i, l in enumerate(layers):
        arr[i].w = l["w"].data_ptr()
        arr[i].w_lp = l["w_lp"].data_ptr()
        arr[i].b = l["b"].data_ptr()
        arr[i].dw = l["dw"].data_ptr() if l.get("dw") is not None else None
        arr[i].db = l["db"].data_ptr() if l.get("db") is not None else None
    return arr


def mlp_workspace_bytes(net: MLP) -> int:
    n = load().mlp_workspace_bytes(net.desc)
    if n == 0:
        raise ImbdError(IMBD_EINVAL, "mlp_workspace_bytes")
    return n


def mlp_workspace_offset(net: MLP, kind: int, layer: int = 0) -> int:
    off = load().mlp_workspace_offset(net.desc, kind, layer)
    if off < 0:
        raise ImbdError(IMBD_EINVAL, "mlp_workspace_offset")
    return off


def ws_view(net: MLP, ws, kind: int, layer: int = 0):
    """A tensor view of one workspace region (activations, logits, Delta_Y, row losses)."""
    torch = _torch()
    off = mlp_workspace_offset(net, kind, layer)
    B = net.batch
    if kind == IMBD_WS_ACT:
        shape, dt = (B, net.dims[layer]), net.torch_dtype()
    elif kind == IMBD_WS_LOGITS:
        shape, dt = (B, net.dims[-1]), torch.float32
    elif kind == IMBD_WS_DY:
        shape, dt = (B, net.dims[layer]), net.torch_dtype()
    else:
        shape, dt = (B,), torch.float32
    esz = torch.empty((), dtype=dt).element_size()
    n = 1
    for s in shape:
        n *= s
    return ws[off:off + n * esz].view(dt).view(shape)


def mlp_fwd(net: MLP, layers, x, labels, ws, loss, stream=None):
    lib = load()
    arr = _layers(layers)
    check(lib.mlp_fwd(net.desc, arr, _ptr(x), _ptr(labels), _ptr(ws), ws.numel() * ws.element_size(),
                      _ptr(loss), _stream(stream)), "mlp_fwd")


def mlp_bwd(net: MLP, layers, x, ws, fuse_sgd: bool, lr: float, dx1=None, stream=None):
    lib = load()
    arr = _layers(layers)
    check(lib.mlp_bwd(net.desc, arr, _ptr(x), _ptr(ws), ws.numel() * ws.element_size(), int(bool(fuse_sgd)),
                      float(lr), _ptr(dx1), _stream(stream)), "mlp_bwd")


def mlp_train_step(net: MLP, layers, x, labels, ws, lr: float, loss, stream=None):
    lib = load()
    arr = _layers(layers)
    check(lib.mlp_train_step(net.desc, arr, _ptr(x), _ptr(labels), _ptr(ws), ws.numel() * ws.element_size(),
                             float(lr), _ptr(loss), _stream(stream)), "mlp_train_step")


def mlp_train_step_static(net: MLP, layers, x, labels, lr: float, loss, stream=None):
    """mlp_train_step on the library's static scratch (no workspace argument, no allocation)."""
    lib = load()
    arr = _layers(layers)
    check(lib.mlp_train_step_static(net.desc, arr, _ptr(x), _ptr(labels), float(lr), _ptr(loss), _stream(stream)),
          "mlp_train_step_static")


def sgd_step(w, grad, lr: float, grad_scale: float = 1.0, w_lp=None, stream=None):
    lib = load()
    check(lib.sgd_step(_ptr(w), _ptr(w_lp), IMBD_BF16 if w_lp is not None else IMBD_F32, _ptr(grad),
                       w.numel(), float(lr), float(grad_scale), _stream(stream)), "sgd_step")


def cast_f32_bf16(src, dst, stream=None):
    lib = load()
    check(lib.cast_f32_bf16(_ptr(src), _ptr(dst), src.numel(), _stream(stream)), "cast_f32_bf16")


def softmax_xent(logits, labels, inv_batch: float, loss, row_loss, dz=None, stream=None):
    lib = load()
    B, C = logits.shape
    check(lib.softmax_xent(B, C, _ptr(logits), logits.stride(0), _ptr(labels), float(inv_batch), _ptr(loss),
                           _ptr(row_loss), _ptr(dz), dz.stride(0) if dz is not None else C,
                           dtype_code(dz) if dz is not None else IMBD_F32, _stream(stream)), "softmax_xent")


def mlp_local_workspace_bytes(which: int, dtype_: int, d_out_blk: int, d_in: int, b_blk: int) -> int:
    return load().mlp_local_workspace_bytes(which, dtype_, d_out_blk, d_in, b_blk)


def _ld(t):
    return t.stride(0) if t is not None else 0


def mlp_local_fwd(w_blk, x_blk, y_blk, P_r: int, P_c: int, bias=None, relu: bool = False, ws=None,
                  stream=None):
    """Y_blk = W_blk X_blk (+bias, ReLU) for one process of the P_r x P_c grid."""
    lib = load()
    d_out, d_in = w_blk.shape
    b_blk = x_blk.shape[0]
    check(lib.mlp_local_fwd(dtype_code(w_blk), int(relu), P_r, P_c, d_out, d_in, b_blk, _ptr(w_blk),
                            _ld(w_blk), _ptr(bias), _ptr(x_blk), _ld(x_blk), _ptr(y_blk), _ld(y_blk),
                            dtype_code(y_blk), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                            _stream(stream)), "mlp_local_fwd")


def mlp_local_bwd(w_blk, dy_blk, x_blk, dw_part, P_r: int, P_c: int, db_part=None, dx_part=None,
                  mask_relu: bool = False, ws=None, stream=None):
    lib = load()
    d_out, d_in = w_blk.shape
    b_blk = x_blk.shape[0]
    check(lib.mlp_local_bwd(dtype_code(w_blk), P_r, P_c, d_out, d_in, b_blk, _ptr(w_blk), _ld(w_blk),
                            _ptr(dy_blk), _ld(dy_blk), _ptr(x_blk), _ld(x_blk), _ptr(dw_part), _ld(dw_part),
                            _ptr(db_part), _ptr(dx_part), _ld(dx_part), int(bool(mask_relu)), _ptr(ws),
                            0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)),
          "mlp_local_bwd")


def conv3x3_tile_fwd(x_pad, w, y, stream=None):
    lib = load()
    N, Hp, Wp, Ci = x_pad.shape
    check(lib.conv3x3_tile_fwd(N, Hp - 2, Wp - 2, Ci, w.shape[0], _ptr(x_pad), _ptr(w), _ptr(y),
                               dtype_code(y), _stream(stream)), "conv3x3_tile_fwd")


def conv3x3_tile_dgrad(dy_pad, w, dx, stream=None):
    lib = load()
    N, Hp, Wp, Co = dy_pad.shape
    check(lib.conv3x3_tile_dgrad(N, Hp - 2, Wp - 2, w.shape[3], Co, _ptr(dy_pad), _ptr(w), _ptr(dx),
                                 dtype_code(dx), _stream(stream)), "conv3x3_tile_dgrad")


def conv3x3_wgrad_workspace_bytes(N, H, W, Ci, Co) -> int:
    return load().conv3x3_wgrad_workspace_bytes(N, H, W, Ci, Co)


def conv3x3_tile_wgrad(x_pad, dy_pad, dw, ws=None, stream=None):
    lib = load()
    N, Hp, Wp, Ci = x_pad.shape
    check(lib.conv3x3_tile_wgrad(N, Hp - 2, Wp - 2, Ci, dy_pad.shape[3], _ptr(x_pad), _ptr(dy_pad), _ptr(dw),
                                 _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                                 _stream(stream)), "conv3x3_tile_wgrad")


def conv3x3_tile_bwd(x_pad, w, dy_pad, dw, dx=None, ws=None, stream=None):
    """Input gradient (skipped when dx is None) and partial weight gradient of the tile."""
    lib = load()
    N, Hp, Wp, Ci = x_pad.shape
    check(lib.conv3x3_tile_bwd(N, Hp - 2, Wp - 2, Ci, dy_pad.shape[3], _ptr(x_pad), _ptr(w), _ptr(dy_pad),
                               _ptr(dx), dtype_code(dx) if dx is not None else IMBD_BF16, _ptr(dw), _ptr(ws),
                               0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)),
          "conv3x3_tile_bwd")


def timing_begin(kernel_class: int, layer: int = -1, max_launches: int = 1000):
    check(load().imbd_timing_begin(kernel_class, layer, max_launches), "imbd_timing_begin")


def timing_end():
    n = ctypes.c_int(0)
    ms = ctypes.c_double(0.0)
    check(load().imbd_timing_end(ctypes.byref(n), ctypes.byref(ms)), "imbd_timing_end")
    return n.value, ms.value


def set_option(key: int, value: int):
    check(load().imbd_set_option(int(key), int(value)), "imbd_set_option")


def get_option(key: int) -> int:
    v = ctypes.c_int(0)
    check(load().imbd_get_option(int(key), ctypes.byref(v)), "imbd_get_option")
    return v.value


def option_name(key: int) -> str:
    return load().imbd_option_name(int(key)).decode()


class options:
    """Context manager: set options (key -> value) for a block, restore them after."""

    def __init__(self, **kv):
        import sys
        mod = sys.modules[__name__]
        self.kv = {getattr(mod, "IMBD_OPT_" + k.upper()): int(v) for k, v in kv.items() if v is not None}
        self.old = {}

    def __enter__(self):
        for k, v in self.kv.items():
            self.old[k] = get_option(k)
            set_option(k, v)
        return self

    def __exit__(self, *exc):
        for k, v in self.old.items():
            set_option(k, v)
