"""Parity of the domain-parallel 3x3 conv tile (Sec. 2.2 of the paper) against the oracle.

bf16 operands with the halo in place; outputs compared normwise: fp32 outputs at 1e-5
(identical operand bits, only fp32 accumulation differs), bf16 outputs at the 2e-2 bar
(and one bf16 rounding, 2^-8). The full-size interior tile (32 x 56 x 56, 256 -> 256) is
checked on every element of all three passes; the corner tile and other full-size shapes
on sampled outputs that the oracle computes one by one."""
import numpy as np
import pytest

import oracle
from synthdata import make_conv_inputs
from tests._util import TOL_BF16, bf16_values, dev_bf16_bits, host, nrm_err

pytestmark = pytest.mark.gpu


def _flush(msg):
    print(msg, flush=True)


def _run(imbd, dev, d, out_bf16=False):
    import torch
    x = dev_bf16_bits(d["x_bits"], dev)
    w = dev_bf16_bits(d["w_bits"], dev)
    dy = dev_bf16_bits(d["dy_bits"], dev)
    N, Hp, Wp, Ci = x.shape
    Co = w.shape[0]
    H, W = Hp - 2, Wp - 2
    odt = torch.bfloat16 if out_bf16 else torch.float32
    y = torch.full((N, H, W, Co), float("nan"), dtype=odt, device=dev)
    dx = torch.full((N, H, W, Ci), float("nan"), dtype=odt, device=dev)
    dw = torch.full((Co, 3, 3, Ci), float("nan"), device=dev)
    nws = imbd.conv3x3_wgrad_workspace_bytes(N, H, W, Ci, Co)
    ws = torch.zeros(max(nws, 16), dtype=torch.uint8, device=dev)
    imbd.conv3x3_tile_fwd(x, w, y)
    imbd.conv3x3_tile_dgrad(dy, w, dx)
    imbd.conv3x3_tile_wgrad(x, dy, dw, ws=ws)
    torch.cuda.synchronize()
    return y, dx, dw


@pytest.mark.parametrize("N,H,W,Ci,Co", [(2, 5, 7, 64, 128), (1, 9, 4, 128, 64), (2, 6, 6, 128, 128),
                                         (1, 1, 1, 64, 64), (3, 11, 13, 64, 64),
                                         # 256 output channels: the large-tile forward / input-gradient
                                         # kernel (one tile; ragged last tile; idle workgroups of the
                                         # padded grid; 256 input channels), and for C_in = 256 the
                                         # weight-gradient kernel
                                         (1, 2, 3, 256, 256), (2, 5, 7, 64, 256), (3, 20, 20, 64, 256),
                                         (1, 6, 11, 256, 64), (2, 7, 9, 256, 128),
                                         # C_in a multiple of 128 as well: the split-K weight-gradient
                                         # kernel (two splits, the last of 6 positions; 19 splits)
                                         (2, 5, 7, 128, 256), (3, 20, 20, 128, 256)])
@pytest.mark.parametrize("border", [(False, False, False, False), (True, False, True, False),
                                    (True, True, True, True)])
def test_conv_tile_small(imbd, dev, N, H, W, Ci, Co, border):
    _flush(f"conv small {(N, H, W, Ci, Co)} border={border}")
    d = make_conv_inputs(N, H, W, Ci, Co, seed=H * 100 + W, border=border)
    xv, wv, dyv = bf16_values(d["x_bits"]), bf16_values(d["w_bits"]), bf16_values(d["dy_bits"])
    y, dx, dw = _run(imbd, dev, d)
    assert nrm_err(host(y), oracle.conv3x3_fwd(xv, wv)) < 1e-5
    assert nrm_err(host(dx), oracle.conv3x3_dgrad(dyv, wv)) < 1e-5
    assert nrm_err(host(dw), oracle.conv3x3_wgrad(xv, dyv)) < 1e-5
    y16, dx16, _ = _run(imbd, dev, d, out_bf16=True)
    assert nrm_err(host(y16), oracle.conv3x3_fwd(xv, wv)) < 2.0 ** -8 + 1e-5
    assert nrm_err(host(dx16), oracle.conv3x3_dgrad(dyv, wv)) < 2.0 ** -8 + 1e-5


@pytest.mark.parametrize("border", [(False, False, False, False), (True, False, True, False)])
def test_conv_tile_full_size_sampled(imbd, dev, border):
    """The 56x56 tile of a 224x224 image split 4x4, batch 32, 256 -> 256 channels:
    an interior tile and a corner tile (zero halo on two sides)."""
    _flush(f"conv full size border={border}")
    N, H, W, C = 32, 56, 56, 256
    d = make_conv_inputs(N, H, W, C, C, seed=5, border=border)
    xv, wv, dyv = bf16_values(d["x_bits"]), bf16_values(d["w_bits"]), bf16_values(d["dy_bits"])
    y, dx, dw = _run(imbd, dev, d)
    rng = np.random.default_rng(1)
    # include the tile's corners and edges among the samples
    yi = np.concatenate([rng.choice(y.numel(), 200, replace=False),
                         [0, C - 1, (W - 1) * C, ((H - 1) * W) * C + 3, y.numel() - 1]])
    assert nrm_err(host(y).reshape(-1)[yi], oracle.conv3x3_fwd_at(xv, wv, yi)) < 1e-5
    xi = np.concatenate([rng.choice(dx.numel(), 200, replace=False), [0, dx.numel() - 1]])
    assert nrm_err(host(dx).reshape(-1)[xi], oracle.conv3x3_dgrad_at(dyv, wv, xi)) < 1e-5
    wi = rng.choice(dw.numel(), 24, replace=False)
    assert nrm_err(host(dw).reshape(-1)[wi], oracle.conv3x3_wgrad_at(xv, dyv, wi)) < 1e-5
    # every output written (no NaN left from the fill) and finite
    import torch
    assert torch.isfinite(y).all().item() and torch.isfinite(dx).all().item() and torch.isfinite(dw).all().item()


@pytest.mark.timeout(600)
def test_conv_tile_full_size_every_element(imbd, dev):
    """The interior 56x56 tile, batch 32, 256 -> 256 channels: every element of the
    forward output, of the input gradient and of the tile's partial weight gradient (the
    tile's share of the all-reduce of Eq. (7)) against the oracle's direct convolution;
    and conv3x3_tile_bwd (both backward passes in one call) gives the bits of the two
    separate calls."""
    import torch
    _flush("conv full size, every element")
    N, H, W, C = 32, 56, 56, 256
    d = make_conv_inputs(N, H, W, C, C, seed=5)
    xv, wv, dyv = bf16_values(d["x_bits"]), bf16_values(d["w_bits"]), bf16_values(d["dy_bits"])
    y, dx, dw = _run(imbd, dev, d)
    ey = nrm_err(host(y), oracle.conv3x3_fwd(xv, wv))
    ew = nrm_err(host(dw), oracle.conv3x3_wgrad(xv, dyv))
    ex = nrm_err(host(dx), oracle.conv3x3_dgrad(dyv, wv))
    _flush(f"conv full size: y {ey:.1e} dx {ex:.1e} dw {ew:.1e}")
    assert ey < 1e-5 and ex < 1e-5 and ew < 1e-5
    xd, wd, dyd = dev_bf16_bits(d["x_bits"], dev), dev_bf16_bits(d["w_bits"], dev), dev_bf16_bits(d["dy_bits"], dev)
    dx2 = torch.full_like(dx, float("nan"))
    dw2 = torch.full_like(dw, float("nan"))
    ws = torch.zeros(max(imbd.conv3x3_wgrad_workspace_bytes(N, H, W, C, C), 16), dtype=torch.uint8, device=dev)
    imbd.conv3x3_tile_bwd(xd, wd, dyd, dw2, dx=dx2, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(dx2, dx) and torch.equal(dw2, dw)


def test_conv_tile_128_position_tiles_sampled(imbd, dev):
    """A tile size for which the forward kernel plans 128-position tiles (225 tiles fill
    one round of workgroups; 258 tiles of 112 positions would need a second, short one):
    sampled outputs of the three passes."""
    _flush("conv 8x60x60 128->256")
    N, H, W, Ci, Co = 8, 60, 60, 128, 256
    d = make_conv_inputs(N, H, W, Ci, Co, seed=9, border=(True, False, False, True))
    xv, wv, dyv = bf16_values(d["x_bits"]), bf16_values(d["w_bits"]), bf16_values(d["dy_bits"])
    y, dx, dw = _run(imbd, dev, d)
    rng = np.random.default_rng(3)
    yi = np.concatenate([rng.choice(y.numel(), 300, replace=False), [0, y.numel() - 1]])
    assert nrm_err(host(y).reshape(-1)[yi], oracle.conv3x3_fwd_at(xv, wv, yi)) < 1e-5
    xi = rng.choice(dx.numel(), 200, replace=False)
    assert nrm_err(host(dx).reshape(-1)[xi], oracle.conv3x3_dgrad_at(dyv, wv, xi)) < 1e-5
    wi = rng.choice(dw.numel(), 24, replace=False)
    assert nrm_err(host(dw).reshape(-1)[wi], oracle.conv3x3_wgrad_at(xv, dyv, wi)) < 1e-5
    import torch
    assert torch.isfinite(y).all().item() and torch.isfinite(dx).all().item() and torch.isfinite(dw).all().item()


@pytest.mark.parametrize("N,H,W", [(4, 92, 92), (4, 113, 113)])
@pytest.mark.parametrize("tile", [128, 112])
def test_conv_tile_last_round_sampled(imbd, dev, N, H, W, tile):
    """More tiles than one round of workgroups on 256 CUs, both tile heights forced:
    4 x 92 x 92 has 265 tiles of 128 positions, whose last 9 run as 128-channel halves (18
    workgroups), or 303 of 112, whose last 47 run as halves; 4 x 113 x 113 has 400 of 128
    (457 of 112), whose last 144 (201) run whole. Every channel of rows in the last round's
    tiles and random outputs elsewhere, fp32 and bf16 outputs, forward and input
    gradient."""
    _flush(f"conv last round {(N, H, W)} tile {tile}")
    C = 256
    d = make_conv_inputs(N, H, W, C, C, seed=H, border=(True, True, False, False))
    xv, wv, dyv = bf16_values(d["x_bits"]), bf16_values(d["w_bits"]), bf16_values(d["dy_bits"])
    M = N * H * W
    rng = np.random.default_rng(H)
    rows = np.array([256 * 128, 256 * 128 + 1, (M + 256 * 128) // 2, M - 129, M - 1])
    full = (rows[:, None] * C + np.arange(C)[None, :]).reshape(-1)
    idx = np.concatenate([full, rng.choice(M * C, 300, replace=False)])
    ry = oracle.conv3x3_fwd_at(xv, wv, idx)
    rx = oracle.conv3x3_dgrad_at(dyv, wv, idx)
    for out_bf16 in (False, True):
        with imbd.options(conv_nt=2 if tile == 128 else 3):
            y, dx, _ = _run(imbd, dev, d, out_bf16=out_bf16)
        tol = 2.0 ** -8 + 1e-5 if out_bf16 else 1e-5
        assert nrm_err(host(y).reshape(-1)[idx], ry) < tol
        assert nrm_err(host(dx).reshape(-1)[idx], rx) < tol
        import torch
        assert torch.isfinite(y).all().item() and torch.isfinite(dx).all().item()


def test_conv_tile_heights_agree_bitwise(imbd, dev):
    """The 32 x 56 x 56 tile, 256 -> 256 channels, forward and input gradient with tiles of
    128 positions (784 tiles: three rounds and a short one of 128-channel halves) and of
    112 (896: three rounds and a full round of halves): every output is the same sum in
    the same slab and MFMA order, so the two give identical bits, fp32 and bf16."""
    import torch
    _flush("conv tile heights 128 / 112, full size")
    N, H, W, C = 32, 56, 56, 256
    d = make_conv_inputs(N, H, W, C, C, seed=11, border=(False, True, False, True))
    x = dev_bf16_bits(d["x_bits"], dev)
    w = dev_bf16_bits(d["w_bits"], dev)
    dy = dev_bf16_bits(d["dy_bits"], dev)
    for odt in (torch.float32, torch.bfloat16):
        outs = []
        for o in (2, 3):
            y = torch.full((N, H, W, C), float("nan"), dtype=odt, device=dev)
            dx = torch.full((N, H, W, C), float("nan"), dtype=odt, device=dev)
            with imbd.options(conv_nt=o):
                imbd.conv3x3_tile_fwd(x, w, y)
                imbd.conv3x3_tile_dgrad(dy, w, dx)
            torch.cuda.synchronize()
            outs.append((y, dx))
        assert torch.isfinite(outs[0][0]).all().item() and torch.isfinite(outs[0][1]).all().item()
        assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


def test_conv_stitched_domain_split(imbd, dev):
    """Domain parallelism on one GPU: a 2x2 split of a zero-padded image with exchanged
    halos (cut from the full padded tensor) reproduces the full-image conv, the summed
    weight gradient and the full input gradient (the halo exchange and the all-reduce of
    Eq. (7) done in software)."""
    import torch
    from synthdata import to_bf16_bits
    rng = np.random.default_rng(2)
    N, H, W, Ci, Co = 2, 12, 10, 64, 64
    x = to_bf16_bits(rng.standard_normal((N, H, W, Ci)).astype(np.float32))
    dy = to_bf16_bits(rng.standard_normal((N, H, W, Co)).astype(np.float32))
    wt = to_bf16_bits((rng.standard_normal((Co, 3, 3, Ci)) * 0.05).astype(np.float32))
    xp = np.pad(bf16_values(x), ((0, 0), (1, 1), (1, 1), (0, 0)))
    dyp = np.pad(bf16_values(dy), ((0, 0), (1, 1), (1, 1), (0, 0)))
    wv = bf16_values(wt)
    y_full, dx_full, dw_full = oracle.conv3x3_fwd(xp, wv), oracle.conv3x3_dgrad(dyp, wv), oracle.conv3x3_wgrad(xp, dyp)
    wd = dev_bf16_bits(wt, dev)
    th, tw = H // 2, W // 2
    y = np.zeros_like(y_full)
    dx = np.zeros_like(dx_full)
    dw = np.zeros_like(dw_full)
    for ti in range(2):
        for tj in range(2):
            hs, ws_ = ti * th, tj * tw
            xt = to_bf16_bits(xp[:, hs:hs + th + 2, ws_:ws_ + tw + 2].astype(np.float32))
            dyt = to_bf16_bits(dyp[:, hs:hs + th + 2, ws_:ws_ + tw + 2].astype(np.float32))
            xd, dyd = dev_bf16_bits(xt, dev), dev_bf16_bits(dyt, dev)
            yt = torch.empty((N, th, tw, Co), device=dev)
            dxt = torch.empty((N, th, tw, Ci), device=dev)
            dwt = torch.empty((Co, 3, 3, Ci), device=dev)
            nws = imbd.conv3x3_wgrad_workspace_bytes(N, th, tw, Ci, Co)
            wsb = torch.zeros(max(nws, 16), dtype=torch.uint8, device=dev)
            imbd.conv3x3_tile_fwd(xd, wd, yt)
            imbd.conv3x3_tile_dgrad(dyd, wd, dxt)
            imbd.conv3x3_tile_wgrad(xd, dyd, dwt, ws=wsb)
            torch.cuda.synchronize()
            y[:, hs:hs + th, ws_:ws_ + tw] = host(yt)
            dx[:, hs:hs + th, ws_:ws_ + tw] = host(dxt)
            dw += host(dwt)
    assert nrm_err(y, y_full) < 1e-5
    assert nrm_err(dx, dx_full) < 1e-5
    assert nrm_err(dw, dw_full) < 1e-5


def test_conv_tile_is_deterministic(imbd, dev):
    """The three passes of the 256-channel kernels twice on the same inputs: identical bits
    (the weight gradient's split partials are added in split order)."""
    d = make_conv_inputs(2, 9, 10, 128, 256, seed=4)
    a = _run(imbd, dev, d)
    b = _run(imbd, dev, d)
    import torch
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_conv_errors(imbd, dev):
    import torch
    x = torch.zeros((1, 4, 4, 48), dtype=torch.bfloat16, device=dev)
    w = torch.zeros((64, 3, 3, 48), dtype=torch.bfloat16, device=dev)
    y = torch.zeros((1, 2, 2, 64), device=dev)
    with pytest.raises(imbd.ImbdError) as e:
        imbd.conv3x3_tile_fwd(x, w, y)               # C_in not a multiple of 64
    assert e.value.status == imbd.IMBD_EUNSUPPORTED
    d = make_conv_inputs(32, 56, 56, 256, 256, seed=0)
    xd, dyd = dev_bf16_bits(d["x_bits"], dev), dev_bf16_bits(d["dy_bits"], dev)
    dw = torch.zeros((256, 3, 3, 256), device=dev)
    assert imbd.conv3x3_wgrad_workspace_bytes(32, 56, 56, 256, 256) > 0
    with pytest.raises(imbd.ImbdError) as e:
        imbd.conv3x3_tile_wgrad(xd, dyd, dw, ws=torch.zeros(64, dtype=torch.uint8, device=dev))
    assert e.value.status == imbd.IMBD_EWORKSPACE
    torch.cuda.synchronize()
