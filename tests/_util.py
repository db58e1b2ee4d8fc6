"""Helpers shared by the GPU tests: device copies of seeded inputs and error metrics."""
from __future__ import annotations

import numpy as np

# Parity bars. Inputs are identical bits on both sides, so an fp32-output product differs
# from the fp64 oracle only by fp32 accumulation; bf16 outputs add one rounding.
TOL_F32 = 1e-4      # max normwise relative error, fp32 path
TOL_BF16 = 2e-2     # max normwise relative error, bf16 operands with fp32 accumulation


def nrm_err(got, ref) -> float:
    """max_j |g_j - o_j| / max_j |o_j| (normwise infinity-norm relative error)."""
    g = np.asarray(got, dtype=np.float64)
    o = np.asarray(ref, dtype=np.float64)
    assert g.shape == o.shape, (g.shape, o.shape)
    if o.size == 0:
        return 0.0
    den = np.max(np.abs(o))
    num = np.max(np.abs(g - o))
    if den == 0:
        return float(num)
    return float(num / den)


def host(t) -> np.ndarray:
    import torch
    if t.dtype == torch.bfloat16:
        return t.float().cpu().numpy().astype(np.float64)
    return t.cpu().numpy().astype(np.float64)


def dev_f32(a, dev):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)


def dev_bf16_bits(bits, dev):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)


def bf16_values(bits) -> np.ndarray:
    from synthdata import bf16_bits_to_f32
    return bf16_bits_to_f32(bits).astype(np.float64)


def make_layers(imbd, d, dev, dtype: str, grads: bool = False):
    """Device parameters from seeded fp32 masters; the bf16 copies come from the
    library's own cast kernel (the path under test)."""
    import torch
    layers = []
    for w, b in zip(d["w"], d["b"]):
        w32 = dev_f32(w, dev)
        b32 = dev_f32(b, dev)
        if dtype == "bf16":
            wlp = torch.empty(w.shape, dtype=torch.bfloat16, device=dev)
            imbd.cast_f32_bf16(w32, wlp)
        else:
            wlp = w32
        l = {"w": w32, "w_lp": wlp, "b": b32}
        if grads:
            l["dw"] = torch.empty_like(w32)
            l["db"] = torch.empty_like(b32)
        layers.append(l)
    return layers


def input_on_device(d, dev, dtype: str):
    if dtype == "bf16":
        return dev_bf16_bits(d["x_bits"], dev), bf16_values(d["x_bits"])
    return dev_f32(d["x"], dev), np.asarray(d["x"], np.float64)


def workspace(imbd, net, dev):
    import torch
    n = imbd.mlp_workspace_bytes(net)
    return torch.zeros(n, dtype=torch.uint8, device=dev)
