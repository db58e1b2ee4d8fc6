"""Reference oracle for the hot path -- TEST INFRASTRUCTURE, NOT PRODUCT CODE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py``
may import this package. It never imports the device package and the device package
never imports it; the two share nothing but the seeded generators in ``synthdata``.

The arithmetic lives in ``oracle.c`` (naive loops in double precision). This module
loads it with ctypes and composes the steps of one SGD iteration in the order the
paper gives them (Sec. 1: forward ``Y_i = W_i X_i, X_{i+1} = f(Y_i)``, backward
``Delta_X = W^T Delta_Y`` and ``Delta_W = Delta_Y X^T``, then the mini-batch update of
Eq. (1); Appendix A for the same products on a process's blocks).

Arrays are numpy float64, one sample per row (``X[b, k]`` is the paper's X(k, b)).

Precision modes of :func:`train_step`:

``"f64"``
    everything in double; the ground truth.
``"bf16"``
    mirrors the storage points of the bf16 device path: the GEMM operands are the
    bf16 copy of each fp32 master weight, post-ReLU activations and every Delta_Y are
    rounded to bf16, logits, gradients, masters and biases to fp32.
``"f32"``
    the same storage points rounded to binary32 (the fp32 device path).

Readings of the paper used here, where it is silent or ambiguous:

* The mean 1/B of Eq. (1) is folded into the top-layer gradient, so every lower
  gradient is already the mini-batch mean; B is a power of two in every workload, so
  the placement does not change a bit.
* ReLU hidden layers, softmax cross-entropy at the top, biases present (zero-initialised
  and updated by the same SGD rule).
* f'(0) = 0.
* A local block's weight-gradient partial carries 1/B_global (passed as ``scale``) so
  the partials of a process column sum to the global mean gradient.
* Delta_X of the first layer is not needed (Sec. 2.2 notes the backward sum starts at
  layer 2); it is computed only on request.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
# ORACLE_LIB names another build of oracle.c to load (the sanitizer build of the tests)
_SO = os.environ.get("ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_lib = None

# AddressSanitizer + UndefinedBehaviorSanitizer, every finding fatal (host code only).
SANITIZE_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                  "-fno-sanitize-recover=all"]

_MODES = {"f64": 0, "bf16": 1, "f32": 2}


def build(out: str | None = None, sanitize: bool = False) -> str:
    """Compile the oracle with gcc (host only, no device code). sanitize: the
    AddressSanitizer / UndefinedBehaviorSanitizer build (load it with ORACLE_LIB and the
    sanitizer runtime preloaded)."""
    out = out or _SO
    opt = SANITIZE_FLAGS if sanitize else ["-O2"]
    cmd = ["gcc", *opt, "-fopenmp", "-shared", "-fPIC", "-Wall", _SRC, "-o", out + ".tmp", "-lm"]
    subprocess.check_call(cmd)
    os.replace(out + ".tmp", out)
    return out


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_SO)
    d, i, l, p = ctypes.c_double, ctypes.c_int, ctypes.c_int64, ctypes.c_void_p
    sig = {
        "orc_threads": (i, []),
        "orc_set_threads": (None, [i]),
        "orc_round_bf16": (d, [d]),
        "orc_round_f32": (d, [d]),
        "orc_round_array": (None, [p, l, i]),
        "orc_affine_fwd": (None, [i, i, i, p, l, p, l, p, p, l]),
        "orc_relu": (None, [p, l]),
        "orc_softmax_xent": (None, [i, i, p, l, p, d, p, p, l, p]),
        "orc_weight_grad": (None, [i, i, i, p, l, p, l, d, p, l, p]),
        "orc_input_grad": (None, [i, i, i, p, l, p, l, p, l]),
        "orc_relu_mask": (None, [i, i, p, l, p, l]),
        "orc_sgd": (None, [p, p, l, d]),
        "orc_conv3x3_fwd": (None, [i, i, i, i, i, p, p, p]),
        "orc_conv3x3_dgrad": (None, [i, i, i, i, i, p, p, p]),
        "orc_conv3x3_wgrad": (None, [i, i, i, i, i, p, p, p]),
        "orc_conv3x3_fwd_at": (None, [i, i, i, i, i, p, p, p, l, p]),
        "orc_conv3x3_dgrad_at": (None, [i, i, i, i, i, p, p, p, l, p]),
        "orc_conv3x3_wgrad_at": (None, [i, i, i, i, i, p, p, p, l, p]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def threads() -> int:
    return _load().orc_threads()


def set_threads(n: int) -> None:
    """OpenMP threads of the loops that follow (the results do not depend on it)."""
    _load().orc_set_threads(int(n))


# ----------------------------------------------------------------------------- rounding
def round_to(a, mode: str) -> np.ndarray:
    out = _f64(a).copy()
    _load().orc_round_array(_ptr(out), out.size, _MODES[mode])
    return out


def round_bf16(a) -> np.ndarray:
    return round_to(a, "bf16")


def bf16_bits_of(a) -> np.ndarray:
    """bf16 bit patterns of values that are already bf16-representable (or inf/nan)."""
    r = np.ascontiguousarray(a, dtype=np.float64).astype(np.float32)
    return (r.view(np.uint32) >> 16).astype(np.uint16)


# ------------------------------------------------------------------- per-layer primitives
def affine_fwd(W, X, bias=None) -> np.ndarray:
    """Y[b, m] = sum_k W[m, k] X[b, k] + bias[m]   (Sec. 1; Appendix A.1)."""
    W, X = _f64(W), _f64(X)
    dout, din = W.shape
    B = X.shape[0]
    assert X.shape[1] == din
    Y = np.empty((B, dout))
    bb = None if bias is None else _f64(bias)
    _load().orc_affine_fwd(dout, din, B, _ptr(W), din, _ptr(X), din,
                           None if bb is None else _ptr(bb), _ptr(Y), dout)
    return Y


def relu(Y) -> np.ndarray:
    out = _f64(Y).copy()
    _load().orc_relu(_ptr(out), out.size)
    return out


def softmax_xent(Z, labels, inv_batch: float):
    """Returns (mean loss, dZ, per-sample loss) for logits Z [B][C]."""
    Z = _f64(Z)
    B, C = Z.shape
    lab = np.ascontiguousarray(labels, dtype=np.int32)
    dZ = np.empty_like(Z)
    rows = np.empty(B)
    loss = ctypes.c_double(0.0)
    _load().orc_softmax_xent(C, B, _ptr(Z), C, _ptr(lab), inv_batch, ctypes.byref(loss),
                             _ptr(dZ), C, _ptr(rows))
    return loss.value, dZ, rows


def weight_grad(dY, X, scale: float = 1.0):
    """dW[m, k] = s sum_b dY[b, m] X[b, k];  db[m] = s sum_b dY[b, m]   (Sec. 1; App. A.2)."""
    dY, X = _f64(dY), _f64(X)
    B, dout = dY.shape
    din = X.shape[1]
    assert X.shape[0] == B
    dW = np.empty((dout, din))
    db = np.empty(dout)
    _load().orc_weight_grad(dout, din, B, _ptr(dY), dout, _ptr(X), din, scale, _ptr(dW), din,
                            _ptr(db))
    return dW, db


def input_grad(W, dY) -> np.ndarray:
    """dX[b, k] = sum_m W[m, k] dY[b, m]   (Sec. 1; App. A.2)."""
    W, dY = _f64(W), _f64(dY)
    dout, din = W.shape
    B = dY.shape[0]
    dX = np.empty((B, din))
    _load().orc_input_grad(dout, din, B, _ptr(W), din, _ptr(dY), dout, _ptr(dX), din)
    return dX


def relu_mask(dX, Xf) -> np.ndarray:
    """dX * [Xf > 0] (chain rule through ReLU, mask read from the stored activation)."""
    out = _f64(dX).copy()
    Xf = _f64(Xf)
    B, din = out.shape
    _load().orc_relu_mask(din, B, _ptr(out), din, _ptr(Xf), din)
    return out


def sgd(w, g, eta: float) -> np.ndarray:
    """Eq. (1): w - eta * g."""
    out = _f64(w).copy()
    gg = _f64(g)
    assert gg.size == out.size
    _load().orc_sgd(_ptr(out), _ptr(gg), out.size, eta)
    return out


# ---------------------------------------------------------------------- full iteration
def forward(ws, bs, x, labels, mode: str = "f64"):
    """Forward pass and loss. ws: fp32 master weights (float arrays), x: input values.

    Returns dict with the operand weights, activations X_1..X_L, logits and the loss.
    """
    L = len(ws)
    B = x.shape[0]
    wop = [round_to(w, "bf16") if mode == "bf16" else _f64(w) for w in ws]
    xs = [_f64(x)]                 # X_1 arrives already in the path's input format
    for i in range(L):
        Y = affine_fwd(wop[i], xs[i], bs[i])
        if i < L - 1:
            xs.append(round_to(relu(Y), mode if mode != "f64" else "f64"))
        else:
            logits = round_to(Y, "f32") if mode != "f64" else Y
    loss, dZ, rows = softmax_xent(logits, labels, 1.0 / B)
    return {"w_op": wop, "acts": xs, "logits": logits, "loss": loss, "dZ": dZ, "row_loss": rows}


def train_step(ws, bs, x, labels, eta: float, mode: str = "f64", want_dx1: bool = False,
               relu_decisions=None):
    """One SGD iteration, Sec. 1 and Eq. (1), in the order the paper gives it.

    ws, bs: lists of fp32 master weights [d_i][d_{i-1}] and biases [d_i]. x: [B][d_0]
    input values (for "bf16" the bf16 values themselves). Returns a dict with
    activations, loss, every Delta_Y, dW, db, the updated masters/biases and, for
    "bf16", the updated bf16 weight copies (as values).

    relu_decisions: optional list indexed like the activations; entry i (i >= 1), when
    not None, is a [B][d_i] array whose positive entries mark where f'(Y_{i-1}) = 1, used
    in place of this iteration's own [X_i > 0]. The derivative of ReLU is a 0/1 decision
    taken on the sign of a sum; a caller comparing two implementations whose sums differ
    by rounding passes one side's decisions so that both sides take the same one. Nothing
    else of the iteration changes.
    """
    L = len(ws)
    st = forward(ws, bs, x, labels, mode)
    store = (lambda a: round_to(a, mode)) if mode != "f64" else (lambda a: a)
    store32 = (lambda a: round_to(a, "f32")) if mode != "f64" else (lambda a: a)
    dY = [None] * L
    dY[L - 1] = store(st["dZ"])
    dWs, dbs = [None] * L, [None] * L
    dx1 = None
    for i in range(L - 1, -1, -1):
        dW, db = weight_grad(dY[i], st["acts"][i], 1.0)
        dWs[i], dbs[i] = dW, db
        if i >= 1:
            dX = input_grad(st["w_op"][i], dY[i])
            dec = None if relu_decisions is None else relu_decisions[i]
            dY[i - 1] = store(relu_mask(dX, st["acts"][i] if dec is None else dec))
        elif want_dx1:
            dx1 = store(input_grad(st["w_op"][0], dY[0]))
    new_w = [store32(sgd(ws[i], dWs[i], eta)) for i in range(L)]
    new_b = [store32(sgd(bs[i], dbs[i], eta)) for i in range(L)]
    out = dict(st)
    out.update({"dY": dY, "dW": [store32(a) for a in dWs], "db": [store32(a) for a in dbs],
                "dW_exact": dWs, "w": new_w, "b": new_b, "dx1": dx1})
    if mode == "bf16":
        out["w_bf16"] = [round_to(w, "bf16") for w in new_w]
    return out


def loss_only(ws, bs, x, labels) -> float:
    """Loss of the network in fp64 (used by the finite-difference pins)."""
    return forward(ws, bs, x, labels, "f64")["loss"]


# --------------------------------------------------------------- local blocks of the grid
def block_rows(n: int, parts: int, idx: int) -> slice:
    """The idx-th of ``parts`` equal contiguous pieces of range(n) (even splits only,
    as in Sec. 2.3)."""
    if n % parts:
        raise ValueError(f"{n} is not divisible by {parts}")
    s = n // parts
    return slice(idx * s, (idx + 1) * s)


def local_fwd(W_blk, X_blk, b_blk=None, apply_relu: bool = False):
    """Process (r, c) forward: Y_blk = W_blk X_blk (+bias), App. A.1 model-parallel form
    on the process's column block; the block is complete and awaits the all-gather."""
    Y = affine_fwd(W_blk, X_blk, b_blk)
    return relu(Y) if apply_relu else Y


def local_bwd(W_blk, dY_blk, X_blk, scale: float, mask_src=None, want_dx: bool = True):
    """Process (r, c) backward, App. A.2: the weight-gradient partial over its B/P_c
    samples (awaits the all-reduce over P_c) and the activation-gradient partial
    W_blk^T dY_blk (awaits the all-reduce over P_r). If mask_src is given, the ReLU
    mask [mask_src > 0] is applied to the partial (the mask is the same on every row of
    the process column, so it commutes with the sum)."""
    dW, db = weight_grad(dY_blk, X_blk, scale)
    dX = None
    if want_dx:
        dX = input_grad(W_blk, dY_blk)
        if mask_src is not None:
            dX = relu_mask(dX, mask_src)
    return dW, db, dX


def grid_layer(W, b, X, dY, P_r: int, P_c: int, scale: float, mask_src=None, apply_relu=False):
    """Software P_r x P_c grid for one layer: run every process's local block and apply
    the collectives of Sec. 2.3 in software (all-gather = concatenation over r,
    all-reduce = summation). Returns assembled Y, dW, db, dX."""
    dout, din = W.shape
    B = X.shape[0]
    Ys = [[None] * P_c for _ in range(P_r)]
    dW = np.zeros((dout, din))
    db = np.zeros(dout)
    dX = np.zeros((B, din))
    for r in range(P_r):
        rs = block_rows(dout, P_r, r)
        for c in range(P_c):
            cs = block_rows(B, P_c, c)
            Ys[r][c] = local_fwd(W[rs], X[cs], None if b is None else b[rs], apply_relu)
            m = None if mask_src is None else mask_src[cs]
            dWp, dbp, dXp = local_bwd(W[rs], dY[cs][:, rs], X[cs], scale, m)
            dW[rs] += dWp          # all-reduce over the P_c processes of row r
            db[rs] += dbp
            dX[cs] += dXp          # all-reduce over the P_r processes of column c
    Y = np.concatenate([np.concatenate([Ys[r][c] for r in range(P_r)], axis=1)
                        for c in range(P_c)], axis=0)   # all-gather over r, columns stacked
    return Y, dW, db, dX


# ------------------------------------------------------------------- conv tile (Sec. 2.2)
def conv3x3_fwd(x_pad, w):
    x_pad, w = _f64(x_pad), _f64(w)
    N, Hp, Wp, Ci = x_pad.shape
    Co = w.shape[0]
    y = np.empty((N, Hp - 2, Wp - 2, Co))
    _load().orc_conv3x3_fwd(N, Hp - 2, Wp - 2, Ci, Co, _ptr(x_pad), _ptr(w), _ptr(y))
    return y


def conv3x3_dgrad(dy_pad, w):
    dy_pad, w = _f64(dy_pad), _f64(w)
    N, Hp, Wp, Co = dy_pad.shape
    Ci = w.shape[3]
    dx = np.empty((N, Hp - 2, Wp - 2, Ci))
    _load().orc_conv3x3_dgrad(N, Hp - 2, Wp - 2, Ci, Co, _ptr(dy_pad), _ptr(w), _ptr(dx))
    return dx


def conv3x3_wgrad(x_pad, dy_pad):
    x_pad, dy_pad = _f64(x_pad), _f64(dy_pad)
    N, Hp, Wp, Ci = x_pad.shape
    Co = dy_pad.shape[3]
    dw = np.empty((Co, 3, 3, Ci))
    _load().orc_conv3x3_wgrad(N, Hp - 2, Wp - 2, Ci, Co, _ptr(x_pad), _ptr(dy_pad), _ptr(dw))
    return dw


def _at(fn, a, b, N, H, W, Ci, Co, idx):
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.size)
    fn(N, H, W, Ci, Co, _ptr(a), _ptr(b), _ptr(idx), idx.size, _ptr(out))
    return out


def conv3x3_fwd_at(x_pad, w, idx):
    x_pad, w = _f64(x_pad), _f64(w)
    N, Hp, Wp, Ci = x_pad.shape
    return _at(_load().orc_conv3x3_fwd_at, x_pad, w, N, Hp - 2, Wp - 2, Ci, w.shape[0], idx)


def conv3x3_dgrad_at(dy_pad, w, idx):
    dy_pad, w = _f64(dy_pad), _f64(w)
    N, Hp, Wp, Co = dy_pad.shape
    return _at(_load().orc_conv3x3_dgrad_at, dy_pad, w, N, Hp - 2, Wp - 2, w.shape[3], Co, idx)


def conv3x3_wgrad_at(x_pad, dy_pad, idx):
    x_pad, dy_pad = _f64(x_pad), _f64(dy_pad)
    N, Hp, Wp, Ci = x_pad.shape
    return _at(_load().orc_conv3x3_wgrad_at, x_pad, dy_pad, N, Hp - 2, Wp - 2, Ci,
               dy_pad.shape[3], idx)
