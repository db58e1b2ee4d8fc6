"""Whole-iteration parity of mlp_fwd / mlp_bwd / mlp_train_step against the oracle.

* fp32 784-256-128-10, B=64: every intermediate at 1e-4 (normwise).
* bf16 networks at oracle-friendly sizes: one step and ten steps against the oracle's
  bf16-mirrored mode at 2e-2.
* Full AlexNet (9216-4096-4096-1000, B=256) and VGG (25088-4096-4096-1000, B=512) FC
  stacks: one step in the launch configuration the benchmark times, checked on sampled
  outputs that the oracle recomputes from the device's own layer inputs.
"""
import numpy as np
import pytest

import oracle
from synthdata import get_config, make_mlp_inputs, scaled_mlp
from tests._util import (TOL_BF16, TOL_F32, host, input_on_device, make_layers, nrm_err,
                         workspace)

pytestmark = pytest.mark.gpu


def _flush(msg):
    print(msg, flush=True)


def _setup(imbd, cfg, dev, seed=0, grads=False):
    import torch
    d = make_mlp_inputs(cfg, seed=seed)
    net = imbd.MLP(cfg.dims, cfg.batch, cfg.dtype)
    layers = make_layers(imbd, d, dev, cfg.dtype, grads=grads)
    x, xv = input_on_device(d, dev, cfg.dtype)
    lab = torch.from_numpy(d["labels"]).to(dev)
    ws = workspace(imbd, net, dev)
    loss = torch.zeros(1, device=dev)
    return d, net, layers, x, xv, lab, ws, loss


def test_fp32_mlp784_one_step_every_intermediate(imbd, dev):
    import torch
    cfg = get_config("mlp784_b64_f32")
    _flush(f"step {cfg.name}")
    d, net, layers, x, xv, lab, ws, loss = _setup(imbd, cfg, dev, grads=True)
    dx1 = torch.empty((cfg.batch, cfg.dims[0]), device=dev)
    imbd.mlp_fwd(net, layers, x, lab, ws, loss)
    imbd.mlp_bwd(net, layers, x, ws, False, cfg.lr, dx1=dx1)
    torch.cuda.synchronize()
    ref = oracle.train_step(d["w"], d["b"], xv, d["labels"], cfg.lr, "f32", want_dx1=True)
    assert abs(loss.item() - ref["loss"]) < TOL_F32 * abs(ref["loss"])
    for i in (1, 2):
        assert nrm_err(host(imbd.ws_view(net, ws, imbd.IMBD_WS_ACT, i)), ref["acts"][i]) < TOL_F32
    assert nrm_err(host(imbd.ws_view(net, ws, imbd.IMBD_WS_LOGITS)), ref["logits"]) < TOL_F32
    for i in (1, 2, 3):
        assert nrm_err(host(imbd.ws_view(net, ws, imbd.IMBD_WS_DY, i)), ref["dY"][i - 1]) < TOL_F32
    for i in range(3):
        assert nrm_err(host(layers[i]["dw"]), ref["dW"][i]) < TOL_F32, i
        assert nrm_err(host(layers[i]["db"]), ref["db"][i]) < TOL_F32, i
    assert nrm_err(host(dx1), ref["dx1"]) < TOL_F32
    # parameters untouched without the fused update
    for i in range(3):
        assert np.array_equal(host(layers[i]["w"]), d["w"][i].astype(np.float64))


def test_fp32_mlp784_fused_update(imbd, dev):
    """The fused update is compared as W' - W (Eq. (1) step), allowing the one fp32
    rounding of W' on top of the 1e-4 gradient bar."""
    import torch
    cfg = get_config("mlp784_b64_f32")
    d, net, layers, x, xv, lab, ws, loss = _setup(imbd, cfg, dev)
    imbd.mlp_train_step(net, layers, x, lab, ws, cfg.lr, loss)
    torch.cuda.synchronize()
    ref = oracle.train_step(d["w"], d["b"], xv, d["labels"], cfg.lr, "f32")
    for i in range(3):
        w0 = d["w"][i].astype(np.float64)
        delta_g = host(layers[i]["w"]) - w0
        delta_o = ref["w"][i] - w0
        ulp = np.spacing(np.abs(w0).max().astype(np.float32))
        assert np.max(np.abs(delta_g - delta_o)) <= TOL_F32 * np.max(np.abs(delta_o)) + ulp, i
        assert nrm_err(host(layers[i]["b"]) - d["b"][i], ref["b"][i] - d["b"][i]) < TOL_F32


@pytest.mark.parametrize("dims,B", [((576, 320, 256, 100), 64), ((33, 17, 5), 3), ((8, 1, 2), 1),
                                    ((1000, 300, 200, 10), 96), ((4096, 1000, 128), 32),
                                    # past 256 samples (the wide-batch products): ragged
                                    # batch, rows and K, split and whole, fp32 logits
                                    ((1032, 264, 136), 777), ((1032, 520, 264, 136), 300)])
def test_bf16_one_step_matches_mirrored_oracle(imbd, dev, dims, B):
    import torch
    cfg = scaled_mlp(dims, B, "bf16")
    _flush(f"bf16 step {dims} B={B}")
    d, net, layers, x, xv, lab, ws, loss = _setup(imbd, cfg, dev, seed=3, grads=True)
    imbd.mlp_fwd(net, layers, x, lab, ws, loss)
    imbd.mlp_bwd(net, layers, x, ws, False, cfg.lr)
    torch.cuda.synchronize()
    ref = oracle.train_step(d["w"], d["b"], xv, d["labels"], cfg.lr, "bf16")
    L = len(dims) - 1
    assert abs(loss.item() - ref["loss"]) < TOL_BF16 * abs(ref["loss"])
    for i in range(1, L):
        assert nrm_err(host(imbd.ws_view(net, ws, imbd.IMBD_WS_ACT, i)), ref["acts"][i]) < TOL_BF16
    assert nrm_err(host(imbd.ws_view(net, ws, imbd.IMBD_WS_LOGITS)), ref["logits"]) < TOL_BF16
    for i in range(L):
        assert nrm_err(host(layers[i]["dw"]), ref["dW"][i]) < TOL_BF16, i
        assert nrm_err(host(layers[i]["db"]), ref["db"][i]) < TOL_BF16, i


@pytest.mark.parametrize("dims,B", [((2056, 2104, 24), 72), ((136, 8, 16), 8), ((4096, 1000, 128), 256),
                                    ((136, 8, 16), 1), ((264, 128, 24), 5),
                                    # 16 KB master pitch, two tiles per workgroup: the spread row-block order
                                    ((4096, 2048, 16), 72),
                                    # past 256 samples: Delta_Y streamed (300), large tiles (777)
                                    ((264, 128, 24), 300), ((1032, 264, 16), 777)])
def test_bf16_fused_update_matches_oracle(imbd, dev, dims, B):
    """The fused weight update (Eq. (1) applied inside the weight-gradient product) on
    shapes that give the persistent update kernel several tiles per workgroup (17 x 17
    tiles of the first layer), ragged tile edges and a batch that is not a multiple of
    the 64-sample K tile; the bf16 copy must be the rounding of every new master."""
    _check_fused_update(imbd, dev, dims, B)


# the options that route the fused update past 256 samples
_UPDATE_ROUTES = {"streamed": {"dw_wide_min_k": 100000},
                  "reload": {"dw_wide_min_k": 100000, "dw_stream": 0},
                  "wide": {"dw_wide_min_k": 257},
                  "wide_dual": {"dw_wide_min_k": 257, "dw_wide_dual": 1}}


@pytest.mark.parametrize("route", sorted(_UPDATE_ROUTES))
@pytest.mark.parametrize("dims,B", [((264, 128, 24), 300), ((1032, 264, 16), 777), ((2056, 520, 16), 2048)])
def test_bf16_fused_update_every_kernel_past_256_samples(imbd, dev, dims, B, route):
    """Past 256 samples three kernels can apply the fused update: the persistent one with
    Delta_Y streamed in slabs, the persistent one with its resident Delta_Y block reloaded
    per 256-sample chunk, and the large-tile one (the default) with one or two workgroups
    per CU. Each is forced in turn, up to the persistent kernel's 2048 samples."""
    with imbd.options(**_UPDATE_ROUTES[route]):
        _check_fused_update(imbd, dev, dims, B)


def _check_fused_update(imbd, dev, dims, B):
    import torch
    cfg = scaled_mlp(dims, B, "bf16")
    _flush(f"bf16 fused update {dims} B={B}")
    d, net, layers, x, xv, lab, ws, loss = _setup(imbd, cfg, dev, seed=11)
    w0 = [host(l["w"]) for l in layers]
    b0 = [host(l["b"]) for l in layers]
    imbd.mlp_train_step(net, layers, x, lab, ws, cfg.lr, loss)
    torch.cuda.synchronize()
    ref = oracle.train_step(w0, b0, xv, d["labels"], cfg.lr, "bf16")
    # the batch mean of the losses (carried by a product launch's extra workgroup)
    assert abs(loss.item() - ref["loss"]) < TOL_BF16 * abs(ref["loss"])
    for i in range(len(dims) - 1):
        wn = host(layers[i]["w"])
        assert nrm_err(wn - w0[i], ref["w"][i] - w0[i]) < TOL_BF16, i
        assert nrm_err(host(layers[i]["b"]) - b0[i], ref["b"][i] - b0[i]) < TOL_BF16, i
        assert np.array_equal(host(layers[i]["w_lp"]), oracle.round_bf16(wn)), i


def test_bf16_ten_steps_match_mirrored_oracle(imbd, dev):
    """Ten fused steps on one fixed batch. Every step is compared with the oracle's step
    taken from the device's own state (masters and biases read back), at the bf16 bar,
    so each of the ten updates is checked without the trajectory noise of bf16: two
    valid bf16 implementations drift apart by ~2-3% in their weight deltas after ten
    steps (cascading rounding flips of Delta_Y, measured by emulating fp32 accumulation
    in the oracle). The free-running loss curve is compared as well."""
    import torch
    cfg = scaled_mlp((576, 320, 256, 100), 64, "bf16", steps=10)
    _flush("bf16 ten steps")
    d, net, layers, x, xv, lab, ws, loss = _setup(imbd, cfg, dev, seed=4)
    ws_o, bs_o = [w.astype(np.float64) for w in d["w"]], [b.astype(np.float64) for b in d["b"]]
    losses_g, losses_o, worst = [], [], 0.0
    for t in range(10):
        w_dev = [host(l["w"]) for l in layers]
        b_dev = [host(l["b"]) for l in layers]
        imbd.mlp_train_step(net, layers, x, lab, ws, cfg.lr, loss)
        torch.cuda.synchronize()
        losses_g.append(loss.item())
        forced = oracle.train_step(w_dev, b_dev, xv, d["labels"], cfg.lr, "bf16")
        for i in range(3):
            e = nrm_err(host(layers[i]["w"]) - w_dev[i], forced["w"][i] - w_dev[i])
            worst = max(worst, e)
            assert e < TOL_BF16, (t, i, e)
            assert nrm_err(host(layers[i]["b"]) - b_dev[i], forced["b"][i] - b_dev[i]) < TOL_BF16, (t, i)
            # the bf16 copy is the rounding of the updated master
            assert np.array_equal(host(layers[i]["w_lp"]), oracle.round_bf16(host(layers[i]["w"])))
        free = oracle.train_step(ws_o, bs_o, xv, d["labels"], cfg.lr, "bf16")
        losses_o.append(free["loss"])
        ws_o, bs_o = free["w"], free["b"]
    print(f"ten steps: worst per-step update error {worst:.2e}, loss curves {nrm_err(losses_g, losses_o):.2e}")
    assert losses_o[-1] < losses_o[0]                      # the same batch every step: loss falls
    assert nrm_err(losses_g, losses_o) < TOL_BF16


@pytest.mark.parametrize("dims,B", [((576, 320, 256, 100), 64), ((64, 32, 10), 16), ((256, 100), 32)])
def test_train_step_loss_equals_forward_loss(imbd, dev, dims, B):
    """mlp_train_step computes the loss mean inside a later launch of the iteration (the
    top layer's Delta_X reduce) when it can, else in a launch of its own (a Delta_X
    product off the skinny path; a one-layer network, which has no Delta_X product):
    every route gives the bits of mlp_fwd's loss, and the oracle's loss."""
    import torch
    cfg = scaled_mlp(dims, B, "bf16")
    _flush(f"train-step loss {dims} B={B}")
    d, net, layers, x, xv, lab, ws, loss = _setup(imbd, cfg, dev, seed=6)
    imbd.mlp_fwd(net, layers, x, lab, ws, loss)
    torch.cuda.synchronize()
    fwd_loss = loss.clone()
    d, net, layers, x, xv, lab, ws, loss = _setup(imbd, cfg, dev, seed=6)
    loss.fill_(float("nan"))
    imbd.mlp_train_step(net, layers, x, lab, ws, cfg.lr, loss)
    torch.cuda.synchronize()
    assert torch.equal(loss, fwd_loss)
    ref = oracle.train_step(d["w"], d["b"], xv, d["labels"], cfg.lr, "bf16")
    assert abs(loss.item() - ref["loss"]) < TOL_BF16 * abs(ref["loss"])


@pytest.mark.parametrize("B", [128, 300, 600])
def test_step_is_deterministic(imbd, dev, B):
    """Two identical steps give identical bits (fixed split order in every reduction),
    also past 256 samples: Delta_Y streamed through the update kernel (300), the large-tile
    products (600)."""
    import torch
    cfg = scaled_mlp((2048, 512, 256, 100), B, "bf16")
    outs = []
    for _ in range(2):
        d, net, layers, x, xv, lab, ws, loss = _setup(imbd, cfg, dev, seed=5)
        imbd.mlp_train_step(net, layers, x, lab, ws, cfg.lr, loss)
        torch.cuda.synchronize()
        outs.append([l["w"].clone() for l in layers] + [loss.clone()])
    for a, b in zip(*outs):
        assert torch.equal(a, b)


# ------------------------------------------------------------------ full-size stacks
def _sampled_full_step(imbd, dev, name, n_rows=24, n_cols=32, seed=0):
    """One fused step at full size; per layer, sampled outputs recomputed by the oracle from
    the device's own inputs to that layer (bf16 bits read back). name: a configuration
    name or a configuration."""
    import torch
    cfg = get_config(name) if isinstance(name, str) else name
    _flush(f"full step {cfg.name} B={cfg.batch}")
    d, net, layers, x, xv, lab, ws, loss = _setup(imbd, cfg, dev, seed=seed)
    L = cfg.n_layers
    B = cfg.batch
    rng = np.random.default_rng(99)
    rows = [rng.choice(B, min(n_rows, B), replace=False) for _ in range(L + 1)]
    cols = [None] + [np.sort(rng.choice(cfg.dims[i], min(n_cols, cfg.dims[i]), replace=False))
                     for i in range(1, L + 1)]
    ci = [None] + [torch.from_numpy(c).to(dev) for c in cols[1:]]
    # weights before the step: sampled rows, and all of W_i for i >= 2 (needed by W^T dY)
    w16_rows = [None] + [host(layers[i - 1]["w_lp"][ci[i]]) for i in range(1, L + 1)]
    w32_rows = [None] + [host(layers[i - 1]["w"][ci[i]]) for i in range(1, L + 1)]
    w16_full = [None, None] + [host(layers[i - 1]["w_lp"]) for i in range(2, L + 1)]
    imbd.mlp_fwd(net, layers, x, lab, ws, loss)
    torch.cuda.synchronize()
    acts = [xv] + [host(imbd.ws_view(net, ws, imbd.IMBD_WS_ACT, i)) for i in range(1, L)]
    logits = host(imbd.ws_view(net, ws, imbd.IMBD_WS_LOGITS))
    imbd.mlp_bwd(net, layers, x, ws, True, cfg.lr)
    torch.cuda.synchronize()
    # Delta_Y_L comes from the forward call, the others from the backward call
    dys = [host(imbd.ws_view(net, ws, imbd.IMBD_WS_DY, i)) for i in range(1, L + 1)]
    for i in range(1, L + 1):
        r, c = rows[i], cols[i]
        # forward: Y_i(rows, cols) from W_i (bf16 copy) and the device's X_i
        y = oracle.affine_fwd(w16_rows[i], acts[i - 1][r], d["b"][i - 1][c])
        got = (acts[i][r][:, c] if i < L else logits[r][:, c])
        ref = oracle.round_bf16(oracle.relu(y)) if i < L else y
        assert nrm_err(got, ref) < TOL_BF16, f"forward layer {i}"
        # weight update: rows `cols` of Delta_W_i from the device's Delta_Y_i and X_i
        dW, _ = oracle.weight_grad(dys[i - 1][:, c], acts[i - 1], 1.0)
        delta_g = host(layers[i - 1]["w"][ci[i]]) - w32_rows[i]
        assert nrm_err(delta_g, -cfg.lr * dW) < TOL_BF16, f"update layer {i}"
        # the bf16 copy is the rounding of the updated master
        assert np.array_equal(host(layers[i - 1]["w_lp"][ci[i]]),
                              oracle.round_bf16(host(layers[i - 1]["w"][ci[i]])))
        # activation gradient: Delta_Y_{i-1}(rows, :) = W_i^T Delta_Y_i masked by X_i
        if i >= 2:
            dx = oracle.input_grad(w16_full[i], dys[i - 1][r])
            ref = oracle.round_bf16(oracle.relu_mask(dx, acts[i - 1][r]))
            assert nrm_err(dys[i - 2][r], ref) < TOL_BF16, f"dX layer {i}"
    # the loss and the top gradient from the device's logits
    r = rows[0]
    l_ref, dz, _ = oracle.softmax_xent(logits, d["labels"], 1.0 / B)
    assert abs(loss.item() - l_ref) < 1e-5 * abs(l_ref)
    assert nrm_err(dys[L - 1][r], oracle.round_bf16(dz[r])) < TOL_BF16


def test_alexnet_fc_b256_full_size_sampled(imbd, dev):
    _sampled_full_step(imbd, dev, "alexnet_fc_b256")


def test_vgg_fc_b512_full_size_sampled(imbd, dev):
    _sampled_full_step(imbd, dev, "vgg_fc_b512", n_rows=16, n_cols=16)


@pytest.mark.parametrize("B", [1, 8, 100, 257, 1024, 2048])
def test_alexnet_fc_batch_sweep_sizes_sampled(imbd, dev, B):
    """The batch sizes of the batch sweep (bench.py --workload batch_sweep) beyond the
    benchmark's 256: one sample (B = 1), ragged batches on the skinny path (100) and past
    it (257), and the large batches on the tiled products (1024, 2048)."""
    cfg = scaled_mlp((9216, 4096, 4096, 1000), B, "bf16", name="alexnet_fc")
    _sampled_full_step(imbd, dev, cfg, n_rows=16, n_cols=16)


def test_workspace_too_small_on_device(imbd, dev):
    import torch
    cfg = scaled_mlp((64, 32, 10), 8, "bf16")
    d, net, layers, x, xv, lab, ws, loss = _setup(imbd, cfg, dev)
    with pytest.raises(imbd.ImbdError) as e:
        imbd.mlp_fwd(net, layers, x, lab, ws[:128], loss)
    assert e.value.status == imbd.IMBD_EWORKSPACE
    torch.cuda.synchronize()


# --------------------------------------------------------------- software 1.5D grid
@pytest.mark.parametrize("P_r,P_c", [(2, 4), (4, 1), (1, 4)])
def test_grid_of_local_blocks_reproduces_the_step(imbd, dev, P_r, P_c):
    """Every process (r, c) of a P_r x P_c grid runs the local kernels on its blocks; the
    collectives of Sec. 2.3 are done in software here (concatenate / sum in fp64) and the
    result must equal the oracle's unpartitioned iteration."""
    import torch
    from tests._util import dev_f32
    cfg = scaled_mlp((256, 128, 64, 16), 32, "f32", x_dist="normal")
    d = make_mlp_inputs(cfg, seed=6)
    ref = oracle.train_step(d["w"], d["b"], d["x"], d["labels"], 0.01, "f64")
    B = cfg.batch
    acts = [np.asarray(d["x"], np.float64)]
    for i in range(3):
        W, b = d["w"][i], d["b"][i]
        dout = W.shape[0]
        Y = np.zeros((B, dout))
        for r in range(P_r):
            rs = oracle.block_rows(dout, P_r, r)
            for c in range(P_c):
                cs = oracle.block_rows(B, P_c, c)
                y = torch.empty((B // P_c, dout // P_r), device=dev)
                wsz = imbd.mlp_local_workspace_bytes(0, imbd.IMBD_F32, dout // P_r, W.shape[1], B // P_c)
                wsb = torch.zeros(max(wsz, 16), dtype=torch.uint8, device=dev)
                imbd.mlp_local_fwd(dev_f32(W[rs], dev), dev_f32(acts[i][cs], dev), y, P_r, P_c,
                                   bias=dev_f32(b[rs], dev), relu=i < 2, ws=wsb)
                Y[cs, rs] = host(y)                   # all-gather over r
        acts.append(Y)
    assert nrm_err(acts[3], ref["logits"]) < TOL_F32
    loss, dz, _ = oracle.softmax_xent(acts[3], d["labels"], 1.0 / B)   # on the gathered logits
    dY = dz * B                                      # raw per-sample gradient
    for i in range(2, -1, -1):
        W = d["w"][i]
        dout, din = W.shape
        dW = np.zeros((dout, din))
        db = np.zeros(dout)
        dX = np.zeros((B, din))
        for r in range(P_r):
            rs = oracle.block_rows(dout, P_r, r)
            for c in range(P_c):
                cs = oracle.block_rows(B, P_c, c)
                dwp = torch.empty((dout // P_r, din), device=dev)
                dbp = torch.empty(dout // P_r, device=dev)
                dxp = torch.empty((B // P_c, din), device=dev)
                wsz = imbd.mlp_local_workspace_bytes(1, imbd.IMBD_F32, dout // P_r, din, B // P_c)
                wsb = torch.zeros(max(wsz, 16), dtype=torch.uint8, device=dev)
                imbd.mlp_local_bwd(dev_f32(W[rs], dev), dev_f32(dY[cs][:, rs], dev), dev_f32(acts[i][cs], dev),
                                   dwp, P_r, P_c, db_part=dbp, dx_part=dxp if i > 0 else None,
                                   mask_relu=i > 0, ws=wsb)
                dW[rs] += host(dwp)                  # all-reduce over P_c
                db[rs] += host(dbp)
                if i > 0:
                    dX[cs] += host(dxp)              # all-reduce over P_r
        assert nrm_err(dW, ref["dW"][i]) < TOL_F32, i
        assert nrm_err(db, ref["db"][i]) < TOL_F32, i
        if i > 0:
            assert nrm_err(dX / B, ref["dY"][i - 1]) < TOL_F32, i
        dY = dX


def test_alexnet_local_4x16_blocks_full_size(imbd, dev):
    """One process's blocks of the 9216-4096-4096-1000 stack on a 4 x 16 grid at global
    B = 1024 (local B = 64), bf16 operands, partials left unreduced; sampled checks."""
    import torch
    from synthdata import make_local_inputs
    from tests._util import bf16_values, dev_bf16_bits
    cfg = get_config("alexnet_fc_local_4x16")
    P_r, P_c = cfg.grid
    b = cfg.local_batch
    rng = np.random.default_rng(7)
    for i in range(1, 4):
        dout, din = cfg.dims[i] // P_r, cfg.dims[i - 1]
        _flush(f"local 4x16 layer {i}: {dout}x{din}, b={b}")
        d = make_local_inputs(dout, din, b, seed=10 + i)
        W, X, DY = bf16_values(d["w_bits"]), bf16_values(d["x_bits"]), bf16_values(d["dy_bits"])
        wd, xd, dyd = dev_bf16_bits(d["w_bits"], dev), dev_bf16_bits(d["x_bits"], dev), dev_bf16_bits(d["dy_bits"], dev)
        wsn = max(imbd.mlp_local_workspace_bytes(0, 1, dout, din, b), imbd.mlp_local_workspace_bytes(1, 1, dout, din, b), 16)
        ws = torch.zeros(wsn, dtype=torch.uint8, device=dev)
        y = torch.empty((b, dout), device=dev, dtype=torch.bfloat16)
        imbd.mlp_local_fwd(wd, xd, y, P_r, P_c, bias=torch.zeros(dout, device=dev), relu=i < 3, ws=ws)
        dw = torch.empty((dout, din), device=dev)
        db = torch.empty(dout, device=dev)
        dx = torch.empty((b, din), device=dev) if i >= 2 else None
        imbd.mlp_local_bwd(wd, dyd, xd, dw, P_r, P_c, db_part=db, dx_part=dx, mask_relu=i >= 2, ws=ws)
        torch.cuda.synchronize()
        cols = rng.choice(dout, 48, replace=False)
        yref = oracle.affine_fwd(W[cols], X)
        yref = oracle.round_bf16(oracle.relu(yref) if i < 3 else yref)
        assert nrm_err(host(y)[:, cols], yref) < TOL_BF16
        rdw, rdb = oracle.weight_grad(DY[:, cols], X, 1.0 / (b * P_c))
        assert nrm_err(host(dw)[cols], rdw) < 1e-4
        assert nrm_err(host(db)[cols], rdb) < 1e-4
        if dx is not None:
            rows = rng.choice(b, 8, replace=False)
            rdx = oracle.relu_mask(oracle.input_grad(W, DY[rows]), X[rows])
            assert nrm_err(host(dx)[rows], rdx) < 1e-4



def test_wide_top_layer_softmax_one_pass_matches_two(imbd, dev):
    """Past 256 samples the top layer's K-split partials go straight into the softmax pass
    (one launch for the split reduce and the softmax cross-entropy). Against the reduce and
    the row softmax as two launches (option top_unfused): the logits bit for bit (the same
    split-order sum and bias), the per-sample losses, the loss and Delta_Y of the top layer
    within fp32 rounding of the two summation orders, and both against the oracle."""
    import torch
    cfg = scaled_mlp((2048, 2048, 1000), 512, "bf16")
    _flush("wide top layer: softmax in one pass vs two")
    d, net, layers, x, xv, lab, ws, loss = _setup(imbd, cfg, dev, seed=4)
    out = {}
    for unfused in (0, 1):
        with imbd.options(top_unfused=unfused):
            imbd.timing_begin(imbd.IMBD_K_SPLITK, -1, 16)
            imbd.mlp_fwd(net, layers, x, lab, ws, loss)
            n_red, _ = imbd.timing_end()
        torch.cuda.synchronize()
        out[unfused] = (host(imbd.ws_view(net, ws, imbd.IMBD_WS_LOGITS)), loss.item(),
                        host(imbd.ws_view(net, ws, imbd.IMBD_WS_DY, 2)), n_red)
    # two K-split reduces of the hidden layers either way; the top layer's only when unfused
    assert out[1][3] == out[0][3] + 1, (out[0][3], out[1][3])
    assert np.array_equal(out[0][0], out[1][0])
    assert abs(out[0][1] - out[1][1]) <= 1e-6 * abs(out[1][1])
    assert nrm_err(out[0][2], out[1][2]) < 1e-5
    ref = oracle.train_step(d["w"], d["b"], xv, d["labels"], cfg.lr, "bf16")
    assert abs(out[0][1] - ref["loss"]) < TOL_BF16 * abs(ref["loss"])
    assert nrm_err(out[0][0], ref["logits"]) < TOL_BF16


def test_dx_reduce_carried_by_update_launch_matches_own_launch(imbd, dev):
    """At 256 samples the layer-2 Delta_X product's split-K partials are added (with the
    ReLU mask, into Delta_Y_1) by the MMA waves of layer 2's update launch instead of a
    reduce launch of its own (option reduce_tail). One full fused step of the
    9216-4096-4096-1000 stack from the same seeded state both ways: one split reduce launch
    fewer, and every output bit for bit the same (the same reduce arithmetic): fp32
    masters, bf16 copies, biases, loss, hidden activations and every Delta_Y."""
    import torch
    cfg = get_config("alexnet_fc_b256")
    _flush("Delta_X reduce carried by the update launch vs its own launch")
    out = {}
    for tail in (1, 0):
        d, net, layers, x, xv, lab, ws, loss = _setup(imbd, cfg, dev, seed=6)
        with imbd.options(reduce_tail=tail):
            imbd.timing_begin(imbd.IMBD_K_SPLITK, -1, 64)
            imbd.mlp_train_step(net, layers, x, lab, ws, cfg.lr, loss)
            n_red, _ = imbd.timing_end()
        torch.cuda.synchronize()
        out[tail] = {"n_red": n_red, "loss": loss.item(),
                     "w": [host(l["w"]) for l in layers], "b": [host(l["b"]) for l in layers],
                     "w16": [l["w_lp"].view(torch.int16).cpu().numpy() for l in layers],
                     "act": [imbd.ws_view(net, ws, imbd.IMBD_WS_ACT, i).view(torch.int16).cpu().numpy() for i in (1, 2)],
                     "dy": [imbd.ws_view(net, ws, imbd.IMBD_WS_DY, i).view(torch.int16).cpu().numpy() for i in (1, 2)]}
    assert out[0]["n_red"] == out[1]["n_red"] + 1, (out[0]["n_red"], out[1]["n_red"])
    assert out[0]["loss"] == out[1]["loss"]
    for k in ("w", "b", "w16", "act", "dy"):
        for i, (a, b) in enumerate(zip(out[0][k], out[1][k])):
            assert np.array_equal(a, b), (k, i)


@pytest.mark.parametrize("update", ["large_tile", "persistent"])
def test_wide_dx_reduce_carried_by_update_launch_matches_own_launch(imbd, dev, update):
    """Past 256 samples a layer's Delta_X split-K partials are added (with the ReLU mask,
    into the Delta_Y of the layer below) by the workgroups of that layer's large-tile update
    launch after their tiles, instead of a reduce launch of its own (option reduce_tail). A
    2048-2048-2048-1000 stack at 512 samples, the wide-batch products split in K two ways:
    two split reduce launches fewer (layers 3 and 2), and every output bit for bit the
    same: fp32 masters, bf16 copies, biases, loss, hidden activations and every Delta_Y.
    With the update forced onto the persistent kernel (which carries only the skinny
    kernel's reduce) the deferred reduce gets its own launch before the update: the same
    launch count and bits."""
    import torch
    cfg = scaled_mlp((2048, 2048, 2048, 1000), 512, "bf16")
    _flush(f"wide Delta_X reduce carried by the update launch vs its own launch ({update} update)")
    route = {} if update == "large_tile" else {"dw_wide_min_k": 100000}
    out = {}
    for tail in (1, 0):
        d, net, layers, x, xv, lab, ws, loss = _setup(imbd, cfg, dev, seed=8)
        with imbd.options(reduce_tail=tail, wide_splits=2, **route):
            imbd.timing_begin(imbd.IMBD_K_SPLITK, -1, 64)
            imbd.mlp_train_step(net, layers, x, lab, ws, cfg.lr, loss)
            n_red, _ = imbd.timing_end()
        torch.cuda.synchronize()
        out[tail] = {"n_red": n_red, "loss": loss.item(),
                     "w": [host(l["w"]) for l in layers], "b": [host(l["b"]) for l in layers],
                     "w16": [l["w_lp"].view(torch.int16).cpu().numpy() for l in layers],
                     "act": [imbd.ws_view(net, ws, imbd.IMBD_WS_ACT, i).view(torch.int16).cpu().numpy() for i in (1, 2)],
                     "dy": [imbd.ws_view(net, ws, imbd.IMBD_WS_DY, i).view(torch.int16).cpu().numpy() for i in (1, 2, 3)]}
    carried = 2 if update == "large_tile" else 0
    assert out[0]["n_red"] == out[1]["n_red"] + carried, (out[0]["n_red"], out[1]["n_red"])
    assert out[0]["loss"] == out[1]["loss"]
    for k in ("w", "b", "w16", "act", "dy"):
        for i, (a, b) in enumerate(zip(out[0][k], out[1][k])):
            assert np.array_equal(a, b), (k, i)
