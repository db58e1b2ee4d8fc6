"""Seeded synthetic workloads for the fully connected hot path and the conv tile.

This module is shared by the tests, the benchmark and the oracle-side checks. It
only draws random numbers and holds the workload shapes; it contains none of the
method's arithmetic (no products, no activations, no losses, no updates).

Workloads (shapes follow the paper's AlexNet/VGG fully connected stacks, which
the paper describes in Sec. 3 only by parameter count; the layer widths are the
usual ones for those networks):

* ``mlp784_b64_f32``       784-256-128-10, B=64, fp32, ReLU, softmax-xent,
                            W ~ N(0, 2/fan_in), b = 0, x ~ U(0,1), labels U{0..9},
                            one SGD step, eta = 0.01.
* ``alexnet_fc_b256``      9216-4096-4096-1000, B=256, bf16 operands, fp32
                            accumulation and fp32 master weights; x = max(N(0,1), 0),
                            labels U{0..999}, W He-initialised, b = 0, eta = 0.01.
* ``alexnet_fc_local_4x16`` one process's blocks of the same stack on a
                            P_r x P_c = 4 x 16 grid at global B = 1024 (local B = 64).
* ``vgg_fc_b512``          25088-4096-4096-1000, B=512, bf16, x = |N(0,1)|.
* ``conv3x3_tile``         3x3 stride-1 conv, 256 -> 256 channels, a 56x56 tile of a
                            224x224 image split 4x4, 1-pixel halo supplied, B = 32.

Every tensor gets its own stream from ``numpy.random.SeedSequence(seed).spawn``
in a fixed, recorded order, so the device path and the oracle see identical bits.
Real ImageNet features are not available; these distributions stand in for them.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "MLPConfig", "ConvTileConfig", "CONFIGS", "get_config",
    "make_mlp_inputs", "make_local_inputs", "make_conv_inputs", "to_bf16_bits",
    "bf16_bits_to_f32", "scaled_mlp",
]


@dataclass(frozen=True)
class MLPConfig:
    name: str
    dims: tuple            # d_0 .. d_L
    batch: int             # global mini-batch B
    dtype: str             # "f32" or "bf16" (operand type; accumulation is fp32)
    lr: float = 0.01
    steps: int = 1
    x_dist: str = "relu_normal"   # "uniform01" | "relu_normal" | "abs_normal" | "normal"
    grid: tuple = (1, 1)   # (P_r, P_c) for the local-block workload
    note: str = ""

    @property
    def n_layers(self) -> int:
        return len(self.dims) - 1

    @property
    def local_batch(self) -> int:
        return self.batch // self.grid[1]

    def gemm_flops(self, batch: int | None = None, with_dx1: bool = False) -> int:
        """Algorithmic flops of one fwd+bwd: forward and dW for every layer, dX from layer 2."""
        B = self.batch if batch is None else batch
        f = 0
        for i in range(1, self.n_layers + 1):
            mk = self.dims[i] * self.dims[i - 1]
            f += 2 * mk * B          # forward
            f += 2 * mk * B          # weight gradient
            if i >= 2 or with_dx1:
                f += 2 * mk * B      # activation gradient
        return f

    @property
    def n_params(self) -> int:
        return sum(self.dims[i] * self.dims[i - 1] for i in range(1, len(self.dims)))


@dataclass(frozen=True)
class ConvTileConfig:
    name: str
    batch: int = 32
    tile_h: int = 56
    tile_w: int = 56
    c_in: int = 256
    c_out: int = 256
    image: int = 224
    grid: tuple = (4, 4)
    note: str = field(default="")

    def flops_per_pass(self) -> int:
        return 2 * self.batch * self.tile_h * self.tile_w * self.c_out * 9 * self.c_in


CONFIGS = {
    "mlp784_b64_f32": MLPConfig("mlp784_b64_f32", (784, 256, 128, 10), 64, "f32",
                                steps=1, x_dist="uniform01"),
    "alexnet_fc_b256": MLPConfig("alexnet_fc_b256", (9216, 4096, 4096, 1000), 256, "bf16",
                                 steps=10, x_dist="relu_normal"),
    "alexnet_fc_local_4x16": MLPConfig("alexnet_fc_local_4x16", (9216, 4096, 4096, 1000), 1024,
                                       "bf16", steps=1, x_dist="normal", grid=(4, 16)),
    "vgg_fc_b512": MLPConfig("vgg_fc_b512", (25088, 4096, 4096, 1000), 512, "bf16",
                             steps=10, x_dist="abs_normal"),
    "conv3x3_tile": ConvTileConfig("conv3x3_tile"),
}


def get_config(name: str):
    return CONFIGS[name]


def scaled_mlp(dims, batch, dtype="bf16", x_dist="relu_normal", lr=0.01, steps=1, name="custom"):
    """A workload of the same structure at another size (parity tests at oracle-friendly sizes)."""
    return MLPConfig(name, tuple(int(d) for d in dims), int(batch), dtype, lr=lr, steps=steps,
                     x_dist=x_dist)


# ----------------------------------------------------------------------------------------
# bf16 bit patterns. The conversion is torch's CPU cast (round to nearest even); it is used
# only to hand bf16 *inputs* to both sides, never to produce expected values.
# ----------------------------------------------------------------------------------------
def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32)


def _streams(seed: int, n: int):
    return [np.random.default_rng(s) for s in np.random.SeedSequence(seed).spawn(n)]


def _draw_x(rng, shape, dist):
    if dist == "uniform01":
        return rng.random(shape, dtype=np.float64).astype(np.float32)
    z = rng.standard_normal(shape, dtype=np.float64)
    if dist == "relu_normal":
        z = np.maximum(z, 0.0)
    elif dist == "abs_normal":
        z = np.abs(z)
    elif dist != "normal":
        raise ValueError(dist)
    return z.astype(np.float32)


def make_mlp_inputs(cfg: MLPConfig, seed: int = 0, batch: int | None = None):
    """Weights, biases, input batch and labels for a full-network step.

    Stream order: x, labels, then (W_i, b_i) for i = 1..L. Weights are fp32 masters
    drawn N(0, 2/fan_in); biases are zero. For bf16 workloads ``x_bits`` holds the
    bf16 input batch (the device consumes it directly); the weight copies are left
    to each side to derive from the masters.
    Layout: W_i is [d_i][d_{i-1}] row-major, x is [B][d_0] (one sample per row).
    """
    B = cfg.batch if batch is None else batch
    L = cfg.n_layers
    rs = _streams(seed, 2 + 2 * L)
    x = _draw_x(rs[0], (B, cfg.dims[0]), cfg.x_dist)
    labels = rs[1].integers(0, cfg.dims[-1], size=B, dtype=np.int64).astype(np.int32)
    ws, bs = [], []
    for i in range(1, L + 1):
        fan_in = cfg.dims[i - 1]
        w = rs[2 * i].standard_normal((cfg.dims[i], fan_in), dtype=np.float64)
        ws.append((w * np.sqrt(2.0 / fan_in)).astype(np.float32))
        bs.append(np.zeros(cfg.dims[i], dtype=np.float32))
    out = {"x": x, "labels": labels, "w": ws, "b": bs, "batch": B}
    if cfg.dtype == "bf16":
        out["x_bits"] = to_bf16_bits(x)
    return out


def make_local_inputs(d_out_blk: int, d_in: int, b_blk: int, seed: int = 0, dtype: str = "bf16",
                      bias: bool = True):
    """One layer's local blocks: W_blk [d_out_blk][d_in], X_blk [b_blk][d_in],
    dY_blk [b_blk][d_out_blk], bias block; X and dY ~ N(0,1), W He-initialised.
    Stream order: W, X, dY, bias, SGD master copy perturbation (unused by default).
    """
    rs = _streams(seed, 4)
    w = (rs[0].standard_normal((d_out_blk, d_in)) * np.sqrt(2.0 / d_in)).astype(np.float32)
    x = rs[1].standard_normal((b_blk, d_in)).astype(np.float32)
    dy = rs[2].standard_normal((b_blk, d_out_blk)).astype(np.float32)
    b = (rs[3].standard_normal(d_out_blk) * 0.1).astype(np.float32) if bias else \
        np.zeros(d_out_blk, np.float32)
    out = {"w": w, "x": x, "dy": dy, "b": b}
    if dtype == "bf16":
        out["w_bits"] = to_bf16_bits(w)
        out["x_bits"] = to_bf16_bits(x)
        out["dy_bits"] = to_bf16_bits(dy)
    return out


def make_conv_inputs(batch: int, h: int, w: int, c_in: int, c_out: int, seed: int = 0,
                     border: tuple = (False, False, False, False)):
    """A conv tile with its 1-pixel halo already in place.

    x_pad [B][h+2][w+2][c_in] and dy_pad [B][h+2][w+2][c_out] are N(0,1); the weights
    [c_out][3][3][c_in] are N(0, 2/(9 c_in)). ``border`` = (top, bottom, left, right)
    marks halo sides that lie on the global image border; those halo rows/columns are
    zero (the image is zero-padded). Returned as fp32 values and bf16 bit patterns.
    Stream order: x_pad, w, dy_pad.
    """
    rs = _streams(seed, 3)
    x = rs[0].standard_normal((batch, h + 2, w + 2, c_in)).astype(np.float32)
    wt = (rs[1].standard_normal((c_out, 3, 3, c_in)) * np.sqrt(2.0 / (9 * c_in))).astype(np.float32)
    dy = rs[2].standard_normal((batch, h + 2, w + 2, c_out)).astype(np.float32)
    top, bottom, left, right = border
    for a in (x, dy):
        if top:
            a[:, 0] = 0
        if bottom:
            a[:, -1] = 0
        if left:
            a[:, :, 0] = 0
        if right:
            a[:, :, -1] = 0
    return {"x_pad": x, "w": wt, "dy_pad": dy,
            "x_bits": to_bf16_bits(x), "w_bits": to_bf16_bits(wt), "dy_bits": to_bf16_bits(dy)}
