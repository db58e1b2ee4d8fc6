"""Parity of the wide-batch forward / Delta_X kernel and the large-tile weight-gradient
kernel at their edges, through the local-block entry points: ragged batch tails (a last
sample tile of one sample), ragged row tiles, K tails of 8, both operand layouts (W rows
for the forward, W k-rows for Delta_X), the bias / ReLU / ReLU' mask epilogues, bf16 and
fp32 outputs, and forced K splits (the workspace is sized under the same setting). The weight-gradient kernel's fp32 store runs
at any batch: a single sample, a ragged 65, and output rows fewer than one tile."""
import numpy as np
import pytest

import oracle
from synthdata import make_local_inputs
from tests._util import bf16_values, dev_bf16_bits, host, nrm_err

pytestmark = pytest.mark.gpu

TOL_F32_OUT = 1e-5     # fp32 outputs of exact bf16 products, fp32 accumulation
TOL_BF16_OUT = 2.0 ** -8 + 1e-5   # one bf16 rounding of the largest value plus fp32 accumulation


def _splits(n):
    """Force the wide kernel's K split for the duration of a block (None: planned)."""
    import paper_1712_04432_amd as m
    return m.options(wide_splits=n)


def _blocks(dout, din, b, seed, dev):
    d = make_local_inputs(dout, din, b, seed=seed, dtype="bf16")
    W, X, DY = bf16_values(d["w_bits"]), bf16_values(d["x_bits"]), bf16_values(d["dy_bits"])
    return d, W, X, DY, dev_bf16_bits(d["w_bits"], dev), dev_bf16_bits(d["x_bits"], dev), \
        dev_bf16_bits(d["dy_bits"], dev)


@pytest.mark.parametrize("dout,din,b", [(136, 72, 257), (264, 1032, 300), (256, 64, 384), (520, 200, 641)])
@pytest.mark.parametrize("out_bf16", [False, True])
def test_wide_forward_bias_relu(imbd, dev, dout, din, b, out_bf16):
    import torch
    d, W, X, _, wd, xd, _ = _blocks(dout, din, b, 21, dev)
    bias = torch.from_numpy(d["b"]).to(dev)
    ref = oracle.relu(oracle.affine_fwd(W, X, d["b"].astype(np.float64)))
    if out_bf16:
        ref = oracle.round_bf16(ref)
    for s in (None, 1, 2, 3):
        with _splits(s):
            y = torch.empty((b, dout), dtype=torch.bfloat16 if out_bf16 else torch.float32, device=dev)
            ws = torch.zeros(max(imbd.mlp_local_workspace_bytes(0, imbd.IMBD_BF16, dout, din, b), 16),
                             dtype=torch.uint8, device=dev)
            imbd.mlp_local_fwd(wd, xd, y, 1, 1, bias=bias, relu=True, ws=ws)
            torch.cuda.synchronize()
        got = host(y)
        assert nrm_err(got, ref) < (TOL_BF16_OUT if out_bf16 else TOL_F32_OUT), s
        if out_bf16:
            # bf16 outputs: the rounding of a value within the fp32 bar of the exact one
            assert np.max(np.abs(got - ref)) <= 2.0 ** -7 * np.max(np.abs(ref)), s


@pytest.mark.parametrize("dout,din,b", [(72, 136, 257), (200, 264, 300), (64, 520, 513)])
def test_wide_delta_x_masked_and_weight_gradient(imbd, dev, dout, din, b):
    import torch
    P_c = 4
    d, W, X, DY, wd, xd, dyd = _blocks(dout, din, b, 22, dev)
    rdw, rdb, rdx = oracle.local_bwd(W, DY, X, 1.0 / (b * P_c), mask_src=X)
    for s in (None, 1, 2):
        with _splits(s):
            dw = torch.empty((dout, din), device=dev)
            db = torch.empty(dout, device=dev)
            dx = torch.empty((b, din), device=dev)
            ws = torch.zeros(max(imbd.mlp_local_workspace_bytes(1, imbd.IMBD_BF16, dout, din, b), 16),
                             dtype=torch.uint8, device=dev)
            imbd.mlp_local_bwd(wd, dyd, xd, dw, 1, P_c, db_part=db, dx_part=dx, mask_relu=True, ws=ws)
            torch.cuda.synchronize()
        assert nrm_err(host(dx), rdx) < TOL_F32_OUT, s
        assert nrm_err(host(dw), rdw) < TOL_F32_OUT, s
        assert nrm_err(host(db), rdb) < TOL_F32_OUT, s
    # masked entries are exact zeros where the layer input is not positive
    assert np.all(host(dx)[X <= 0] == 0.0)


@pytest.mark.parametrize("dout,din,b", [(10, 128, 1), (10, 128, 65), (300, 264, 1), (300, 264, 65), (8, 8, 3)])
def test_weight_gradient_store_small_batches(imbd, dev, dout, din, b):
    import torch
    d, W, X, DY, wd, xd, dyd = _blocks(dout, din, b, 23, dev)
    rdw, rdb, _ = oracle.local_bwd(W, DY, X, 1.0 / b, want_dx=False)
    dw = torch.full((dout, din), 7.0, device=dev)
    db = torch.empty(dout, device=dev)
    ws = torch.zeros(max(imbd.mlp_local_workspace_bytes(1, imbd.IMBD_BF16, dout, din, b), 16),
                     dtype=torch.uint8, device=dev)
    imbd.mlp_local_bwd(wd, dyd, xd, dw, 1, 1, db_part=db, ws=ws)
    torch.cuda.synchronize()
    assert nrm_err(host(dw), rdw) < TOL_F32_OUT
    assert nrm_err(host(db), rdb) < TOL_F32_OUT


def test_wide_products_are_deterministic(imbd, dev):
    """Split partials are added in split order: identical inputs give identical bits."""
    import torch
    dout, din, b = 264, 1032, 641
    d, W, X, DY, wd, xd, dyd = _blocks(dout, din, b, 24, dev)
    outs = []
    for _ in range(2):
        y = torch.empty((b, dout), device=dev)
        dx = torch.empty((b, din), device=dev)
        dw = torch.empty((dout, din), device=dev)
        ws = torch.zeros(max(imbd.mlp_local_workspace_bytes(0, imbd.IMBD_BF16, dout, din, b),
                             imbd.mlp_local_workspace_bytes(1, imbd.IMBD_BF16, dout, din, b), 16),
                         dtype=torch.uint8, device=dev)
        imbd.mlp_local_fwd(wd, xd, y, 1, 1, ws=ws)
        imbd.mlp_local_bwd(wd, dyd, xd, dw, 1, 1, dx_part=dx, ws=ws)
        torch.cuda.synchronize()
        outs.append((y.clone(), dx.clone(), dw.clone()))
    for a, c in zip(*outs):
        assert torch.equal(a, c)
