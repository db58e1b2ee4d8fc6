"""Per-kernel parity of the HIP path against the oracle, through the C ABI.

Shapes span several tiles and ragged tails (M, N, K not multiples of the 64/128 tiles,
K not a multiple of the 8-element vector, single rows/columns)."""
import numpy as np
import pytest

import oracle
from synthdata import make_local_inputs, to_bf16_bits
from tests._util import TOL_BF16, TOL_F32, bf16_values, dev_bf16_bits, dev_f32, host, nrm_err

pytestmark = pytest.mark.gpu


def _flush(msg):
    print(msg, flush=True)


# ------------------------------------------------------------------------------ cast
def test_cast_f32_bf16_bit_exact(imbd, dev):
    import torch
    rng = np.random.default_rng(0)
    f = np.concatenate([
        (rng.standard_normal(100003) * 10.0 ** rng.integers(-38, 38, 100003)).astype(np.float32),
        (np.arange(1, 5000, dtype=np.uint32) << 16 | np.uint32(0x8000)).view(np.float32),   # ties
        np.array([0.0, -0.0, 1e-45, -1e-45, 3.39e38, 3.4e38, -3.4e38, np.inf, -np.inf], np.float32),
    ]).astype(np.float32)
    src = dev_f32(f, dev)
    dst = torch.empty(f.size, dtype=torch.bfloat16, device=dev)
    imbd.cast_f32_bf16(src, dst)
    got = dst.view(torch.int16).cpu().numpy().view(np.uint16)
    ref = oracle.bf16_bits_of(oracle.round_bf16(f.astype(np.float64)))
    assert np.array_equal(got, ref)
    # NaN stays NaN
    nan = dev_f32(np.array([np.nan], np.float32), dev)
    out = torch.empty(1, dtype=torch.bfloat16, device=dev)
    imbd.cast_f32_bf16(nan, out)
    assert torch.isnan(out.float()).item()


# ------------------------------------------------------------------------------- SGD
@pytest.mark.parametrize("n", [1, 3, 4, 1000, 1 << 20, (1 << 20) + 7])
def test_sgd_step_bit_exact(imbd, dev, n):
    """Eq. (1): w - lr*g with one fp32 rounding; lr given as the fp32 value both sides use."""
    import torch
    rng = np.random.default_rng(n)
    w = rng.standard_normal(n).astype(np.float32)
    g = rng.standard_normal(n).astype(np.float32)
    lr = float(np.float32(0.01))
    wd, gd = dev_f32(w, dev), dev_f32(g, dev)
    w16 = torch.empty(n, dtype=torch.bfloat16, device=dev)
    imbd.sgd_step(wd, gd, lr, 1.0, w_lp=w16)
    ref = oracle.round_to(oracle.sgd(w, g, lr), "f32")
    assert np.array_equal(wd.cpu().numpy().astype(np.float64), ref)
    assert np.array_equal(w16.view(torch.int16).cpu().numpy().view(np.uint16),
                          oracle.bf16_bits_of(oracle.round_bf16(ref)))


def test_sgd_step_unaligned_and_scaled(imbd, dev):
    rng = np.random.default_rng(5)
    w = rng.standard_normal(1001).astype(np.float32)
    g = rng.standard_normal(1001).astype(np.float32)
    base = dev_f32(np.concatenate([[0], w]), dev)
    gb = dev_f32(np.concatenate([[0], g]), dev)
    wd, gd = base[1:], gb[1:]                       # 4-byte offset: scalar kernel
    imbd.sgd_step(wd, gd, 0.5, 0.25)
    step = float(np.float32(np.float32(0.5) * np.float32(0.25)))
    ref = oracle.round_to(oracle.sgd(w, g, step), "f32")
    assert np.array_equal(wd.cpu().numpy().astype(np.float64), ref)


# --------------------------------------------------------------------------- softmax
@pytest.mark.parametrize("B,C,dz_dtype", [(64, 10, "f32"), (256, 1000, "bf16"), (256, 1000, "f32"),
                                          (5, 3, "f32"), (1, 1, "f32"), (33, 129, "bf16")])
def test_softmax_xent(imbd, dev, B, C, dz_dtype):
    import torch
    rng = np.random.default_rng(B * 1000 + C)
    z = (rng.standard_normal((B, C)) * 4).astype(np.float32)
    lab = rng.integers(0, C, B).astype(np.int32)
    zd = dev_f32(z, dev)
    ld = torch.from_numpy(lab).to(dev)
    loss = torch.zeros(1, device=dev)
    rows = torch.zeros(B, device=dev)
    dz = torch.empty((B, C), device=dev, dtype=torch.bfloat16 if dz_dtype == "bf16" else torch.float32)
    imbd.softmax_xent(zd, ld, 1.0 / B, loss, rows, dz)
    rl, rdz, rrows = oracle.softmax_xent(z, lab, 1.0 / B)
    assert abs(loss.item() - rl) <= 1e-5 * max(1.0, abs(rl))
    assert nrm_err(host(rows), rrows) < 1e-5
    tol = TOL_BF16 if dz_dtype == "bf16" else TOL_F32
    assert nrm_err(host(dz), rdz) < tol
    if dz_dtype == "bf16":
        assert nrm_err(host(dz), rdz) < 2.0 ** -8 + 1e-5
    else:
        assert nrm_err(host(dz), rdz) < 1e-6


@pytest.mark.parametrize("dz_dtype", ["f32", "bf16"])
def test_softmax_bad_label_gives_nan_not_a_fault(imbd, dev, dz_dtype):
    """A label outside [0, C) makes its sample's loss and its whole gradient row NaN (there
    is no one-hot to subtract), so the corruption cannot reach an update unseen; the other
    rows are untouched."""
    import torch
    z = dev_f32(np.zeros((4, 10), np.float32), dev)
    lab = torch.tensor([0, 10, -1, 9], dtype=torch.int32, device=dev)
    loss = torch.zeros(1, device=dev)
    rows = torch.zeros(4, device=dev)
    dz = torch.zeros((4, 10), device=dev, dtype=torch.float32 if dz_dtype == "f32" else torch.bfloat16)
    imbd.softmax_xent(z, lab, 0.25, loss, rows, dz)
    r = rows.cpu().numpy()
    g = host(dz)
    assert np.isnan(r[1]) and np.isnan(r[2]) and np.isnan(loss.item())
    assert r[0] == pytest.approx(np.log(10), rel=1e-6) and r[3] == pytest.approx(np.log(10), rel=1e-6)
    assert np.isnan(g[1]).all() and np.isnan(g[2]).all()
    for i in (0, 3):
        _, ref, _ = oracle.softmax_xent(np.zeros((1, 10)), [int(lab[i])], 0.25)
        assert np.isfinite(g[i]).all() and nrm_err(g[i], ref[0]) < 1e-2


def test_fused_top_layer_bad_label_gives_nan_row(imbd, dev):
    """The same through the top layer's fused split reduce + softmax (mlp_fwd at a shape
    whose top product runs on the B <= 256 product kernel)."""
    import torch
    from synthdata import make_mlp_inputs, scaled_mlp
    from tests._util import input_on_device, make_layers, workspace
    cfg = scaled_mlp((576, 320, 256, 100), 64, "bf16")
    d = make_mlp_inputs(cfg, seed=2)
    net = imbd.MLP(cfg.dims, cfg.batch, "bf16")
    layers = make_layers(imbd, d, dev, "bf16")
    x, _ = input_on_device(d, dev, "bf16")
    lab_h = d["labels"].copy()
    lab_h[5], lab_h[17] = 100, -3
    lab = torch.from_numpy(lab_h).to(dev)
    ws = workspace(imbd, net, dev)
    loss = torch.zeros(1, device=dev)
    imbd.mlp_fwd(net, layers, x, lab, ws, loss)
    torch.cuda.synchronize()
    rl = host(imbd.ws_view(net, ws, imbd.IMBD_WS_ROWLOSS))
    dy = host(imbd.ws_view(net, ws, imbd.IMBD_WS_DY, 3))
    bad = np.zeros(64, bool)
    bad[[5, 17]] = True
    assert np.isnan(loss.item())
    assert np.isnan(rl[bad]).all() and np.isfinite(rl[~bad]).all()
    assert np.isnan(dy[bad]).all() and np.isfinite(dy[~bad]).all()


# ------------------------------------------------------------------ local products
LOCAL_SHAPES = [
    # d_out_blk, d_in, b_blk
    (256, 784, 64), (128, 256, 64), (10, 128, 64),             # the 784-256-128-10 layers
    (1024, 4096, 64), (250, 4096, 64),                          # 4 x 16 grid blocks
    (130, 200, 70), (37, 100, 13), (1, 1, 1), (64, 64, 64), (129, 65, 257), (3, 8, 5),
    # past 256 samples, bf16: the wide-batch product kernel, ragged in every dimension
    # (forward split over K; Delta_X whole), and a forward split 8 ways
    (264, 1032, 777), (512, 4096, 300),
    (200, 1000, 128),
    # 9 x 33 tiles of 128 x 128, ragged: the fp32 weight-gradient store on two workgroups per CU
    (1032, 4104, 72),
    # a 500-byte Delta_Y pitch with more than 128 samples: not read in place (the paired launch
    # takes 4-byte pieces up to 128 samples), so the block is copied into 16-byte rows first
    (250, 512, 200),
]


def _local_inputs(dout, din, b, dtype, seed=0):
    d = make_local_inputs(dout, din, b, seed=seed, dtype=dtype)
    if dtype == "bf16":
        return d, bf16_values(d["w_bits"]), bf16_values(d["x_bits"]), bf16_values(d["dy_bits"])
    return d, d["w"].astype(np.float64), d["x"].astype(np.float64), d["dy"].astype(np.float64)


def _to_dev(d, key, dtype, dev):
    return dev_bf16_bits(d[key + "_bits"], dev) if dtype == "bf16" else dev_f32(d[key], dev)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", LOCAL_SHAPES)
def test_local_fwd_parity(imbd, dev, dtype, shape):
    import torch
    dout, din, b = shape
    _flush(f"local_fwd {dtype} {shape}")
    d, W, X, _ = _local_inputs(dout, din, b, dtype)
    wd, xd = _to_dev(d, "w", dtype, dev), _to_dev(d, "x", dtype, dev)
    bias = dev_f32(d["b"], dev)
    ws = torch.zeros(max(imbd.mlp_local_workspace_bytes(0, imbd.dtype_code(wd), dout, din, b), 16),
                     dtype=torch.uint8, device=dev)
    ref = oracle.local_fwd(W, X, d["b"].astype(np.float64), apply_relu=False)
    y32 = torch.empty((b, dout), device=dev)
    imbd.mlp_local_fwd(wd, xd, y32, 4, 16, bias=bias, relu=False, ws=ws)
    assert nrm_err(host(y32), ref) < 1e-5          # only fp32 accumulation differs
    yr = torch.empty((b, dout), device=dev, dtype=torch.bfloat16 if dtype == "bf16" else torch.float32)
    imbd.mlp_local_fwd(wd, xd, yr, 4, 16, bias=bias, relu=True, ws=ws)
    rr = oracle.relu(ref)
    tol = TOL_BF16 if dtype == "bf16" else TOL_F32
    assert nrm_err(host(yr), oracle.round_to(rr, dtype)) < tol
    if dtype == "bf16":
        assert nrm_err(host(yr), rr) < 2.0 ** -8 + 1e-5


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", LOCAL_SHAPES)
def test_local_bwd_parity(imbd, dev, dtype, shape):
    import torch
    dout, din, b = shape
    _flush(f"local_bwd {dtype} {shape}")
    P_r, P_c = 4, 16
    d, W, X, DY = _local_inputs(dout, din, b, dtype, seed=1)
    wd, xd, dyd = _to_dev(d, "w", dtype, dev), _to_dev(d, "x", dtype, dev), _to_dev(d, "dy", dtype, dev)
    ws = torch.zeros(max(imbd.mlp_local_workspace_bytes(1, imbd.dtype_code(wd), dout, din, b), 16),
                     dtype=torch.uint8, device=dev)
    dw = torch.empty((dout, din), device=dev)
    db = torch.empty(dout, device=dev)
    dx = torch.empty((b, din), device=dev)
    imbd.mlp_local_bwd(wd, dyd, xd, dw, P_r, P_c, db_part=db, dx_part=dx, mask_relu=True, ws=ws)
    scale = 1.0 / (b * P_c)
    rdw, rdb, rdx = oracle.local_bwd(W, DY, X, scale, mask_src=X)
    assert nrm_err(host(dw), rdw) < 1e-5
    assert nrm_err(host(db), rdb) < 1e-5
    assert nrm_err(host(dx), rdx) < 1e-5
    # unmasked partial
    imbd.mlp_local_bwd(wd, dyd, xd, dw, P_r, P_c, dx_part=dx, mask_relu=False, ws=ws)
    assert nrm_err(host(dx), oracle.input_grad(W, DY)) < 1e-5


# (d_out block, d_in, samples): the 4 x 16 grid's layer-3 and layer-2 blocks, ragged ones, one
# with 200 samples (128-sample workgroups), and ones whose Delta_W cannot take the large-tile
# kernel (d_in not a multiple of 8), which keep two launches
PAIR_SHAPES = [(250, 4096, 64), (1024, 4096, 64), (130, 200, 70), (264, 1032, 200), (3, 8, 5), (37, 100, 13)]


@pytest.mark.parametrize("shape", PAIR_SHAPES)
def test_local_bwd_one_launch_matches_two(imbd, dev, shape):
    """The local backward pass's Delta_X and Delta_W partials are independent products; when
    both run on the large-tile kernels without partial sums they share one launch, each
    workgroup running one kernel's body, so every bit equals what two launches give. The
    launch count of the Delta_X kernel class shows which route ran."""
    import torch
    dout, din, b = shape
    _flush(f"local_bwd one launch vs two {shape}")
    d, W, X, DY = _local_inputs(dout, din, b, "bf16", seed=5)
    wd, xd, dyd = _to_dev(d, "w", "bf16", dev), _to_dev(d, "x", "bf16", dev), _to_dev(d, "dy", "bf16", dev)
    ws = torch.zeros(max(imbd.mlp_local_workspace_bytes(1, imbd.IMBD_BF16, dout, din, b), 16),
                     dtype=torch.uint8, device=dev)
    out = {}
    for pair in (1, 0):
        dw = torch.full((dout, din), 7.0, device=dev)
        db = torch.full((dout,), 7.0, device=dev)
        dx = torch.full((b, din), 7.0, device=dev)
        with imbd.options(local_pair=pair):
            imbd.timing_begin(imbd.IMBD_K_GEMM_DX, -1, 16)
            imbd.mlp_local_bwd(wd, dyd, xd, dw, 4, 16, db_part=db, dx_part=dx, mask_relu=True, ws=ws)
            n_dx, _ = imbd.timing_end()
        torch.cuda.synchronize()
        out[pair] = (host(dw), host(db), host(dx), n_dx)
    paired = din % 8 == 0
    assert out[1][3] == (0 if paired else 1) and out[0][3] == 1, (out[1][3], out[0][3])
    for a, c in zip(out[1][:3], out[0][:3]):
        assert np.array_equal(a, c)
    rdw, rdb, rdx = oracle.local_bwd(W, DY, X, 1.0 / (b * 16), mask_src=X)
    assert nrm_err(out[1][0], rdw) < 1e-5 and nrm_err(out[1][1], rdb) < 1e-5 and nrm_err(out[1][2], rdx) < 1e-5


@pytest.mark.parametrize("col0", [250, 2])
def test_local_bwd_dy_block_of_wider_rows(imbd, dev, col0):
    """The Delta_Y block as a view of the full top-layer gradient (64 x 1000, 2000-byte
    rows): a process's 250 columns from col0 on, rows 4-byte aligned but not 16-byte
    aligned. The paired launch reads them in place in 4-byte pieces; every bit equals the
    two-launch route (which copies the block into aligned rows) and the oracle agrees."""
    import torch
    _flush(f"local_bwd Delta_Y view at column {col0}")
    dout, din, b = 250, 1024, 64
    d, W, X, _ = _local_inputs(dout, din, b, "bf16", seed=7)
    rng = np.random.default_rng(col0)
    full = to_bf16_bits(rng.standard_normal((b, 1000)).astype(np.float32))
    DY = bf16_values(full)[:, col0:col0 + dout]
    wd, xd = _to_dev(d, "w", "bf16", dev), _to_dev(d, "x", "bf16", dev)
    dyd = dev_bf16_bits(full, dev)[:, col0:col0 + dout]
    ws = torch.zeros(max(imbd.mlp_local_workspace_bytes(1, imbd.IMBD_BF16, dout, din, b), 16),
                     dtype=torch.uint8, device=dev)
    out = {}
    for pair in (1, 0):
        dw = torch.full((dout, din), 7.0, device=dev)
        db = torch.full((dout,), 7.0, device=dev)
        dx = torch.full((b, din), 7.0, device=dev)
        with imbd.options(local_pair=pair):
            imbd.timing_begin(imbd.IMBD_K_GEMM_DX, -1, 16)
            imbd.mlp_local_bwd(wd, dyd, xd, dw, 4, 16, db_part=db, dx_part=dx, mask_relu=True, ws=ws)
            n_dx, _ = imbd.timing_end()
        torch.cuda.synchronize()
        out[pair] = (host(dw), host(db), host(dx), n_dx)
    assert out[1][3] == 0 and out[0][3] == 1, (out[1][3], out[0][3])
    for a, c in zip(out[1][:3], out[0][:3]):
        assert np.array_equal(a, c)
    rdw, rdb, rdx = oracle.local_bwd(W, DY, X, 1.0 / (b * 16), mask_src=X)
    assert nrm_err(out[1][0], rdw) < 1e-5 and nrm_err(out[1][1], rdb) < 1e-5 and nrm_err(out[1][2], rdx) < 1e-5


def test_local_step_graph_replay_matches_eager(imbd, dev):
    """The local forward and backward calls captured into a HIP graph (as the bench times
    them): three replays, with eager work and synchronisation between them, each give the
    bits of the eager calls (the library enqueues only kernels on the given stream)."""
    import torch
    _flush("local step graph replay")
    dout, din, b = 250, 1024, 64
    d, W, X, DY = _local_inputs(dout, din, b, "bf16", seed=11)
    wd, xd, dyd = _to_dev(d, "w", "bf16", dev), _to_dev(d, "x", "bf16", dev), _to_dev(d, "dy", "bf16", dev)
    bias = dev_f32(d["b"], dev)
    ws = torch.zeros(max(imbd.mlp_local_workspace_bytes(0, imbd.IMBD_BF16, dout, din, b),
                         imbd.mlp_local_workspace_bytes(1, imbd.IMBD_BF16, dout, din, b), 16),
                     dtype=torch.uint8, device=dev)
    y = torch.empty((b, dout), dtype=torch.bfloat16, device=dev)
    dw = torch.empty((dout, din), device=dev)
    db = torch.empty(dout, device=dev)
    dx = torch.empty((b, din), device=dev)
    outs = (y, dw, db, dx)

    def step(st):
        imbd.mlp_local_fwd(wd, xd, y, 4, 16, bias=bias, relu=True, ws=ws, stream=st)
        imbd.mlp_local_bwd(wd, dyd, xd, dw, 4, 16, db_part=db, dx_part=dx, mask_relu=True, ws=ws, stream=st)

    step(torch.cuda.current_stream())
    torch.cuda.synchronize()
    ref = [o.clone() for o in outs]
    g, cap = torch.cuda.CUDAGraph(), torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        with torch.cuda.graph(g, stream=cap):
            step(cap)
    torch.cuda.synchronize()
    for r in range(3):
        for o in outs:
            o.fill_(float("nan"))
        (wd.float() * 2.0).sum().item()   # unrelated eager work and a synchronisation
        g.replay()
        torch.cuda.synchronize()
        for o, e in zip(outs, ref):
            assert torch.equal(o, e), r


def test_local_fwd_strided_views(imbd, dev):
    """Blocks passed as views of a larger array (leading dimension > row length)."""
    import torch
    rng = np.random.default_rng(3)
    Wf = rng.standard_normal((300, 520)).astype(np.float32)
    Xf = rng.standard_normal((96, 520)).astype(np.float32)
    Wb, Xb = to_bf16_bits(Wf), to_bf16_bits(Xf)
    wd, xd = dev_bf16_bits(Wb, dev), dev_bf16_bits(Xb, dev)
    Wv, Xv = bf16_values(Wb), bf16_values(Xb)
    # process (r, c) = (1, 2) of a 3 x 4 grid over W rows and X rows, columns 8..520
    wblk, xblk = wd[100:200, 8:520], xd[48:72, 8:520]
    ybig = torch.zeros((24, 300), device=dev)
    yblk = ybig[:, 100:200]
    ws = torch.zeros(max(imbd.mlp_local_workspace_bytes(0, 1, 100, 512, 24), 16), dtype=torch.uint8, device=dev)
    imbd.mlp_local_fwd(wblk, xblk, yblk, 3, 4, ws=ws)
    ref = oracle.affine_fwd(Wv[100:200, 8:520], Xv[48:72, 8:520])
    assert nrm_err(host(yblk), ref) < 1e-5
    assert torch.count_nonzero(ybig[:, :100]).item() == 0 and torch.count_nonzero(ybig[:, 200:]).item() == 0


def test_local_wide_batch_strided_views(imbd, dev):
    """The wide-batch products on blocks passed as views (leading dimensions above the
    row lengths, output a column block of a larger array)."""
    import torch
    rng = np.random.default_rng(4)
    Wf = rng.standard_normal((300, 520)).astype(np.float32)
    Xf = rng.standard_normal((300, 520)).astype(np.float32)
    DYf = rng.standard_normal((300, 264)).astype(np.float32)
    Wb, Xb, DYb = to_bf16_bits(Wf), to_bf16_bits(Xf), to_bf16_bits(DYf)
    wd, xd, dyd = dev_bf16_bits(Wb, dev), dev_bf16_bits(Xb, dev), dev_bf16_bits(DYb, dev)
    Wv, Xv, DYv = bf16_values(Wb), bf16_values(Xb), bf16_values(DYb)
    wblk, xblk = wd[100:300, 8:520], xd[:, 8:520]
    ybig = torch.zeros((300, 400), device=dev)
    yblk = ybig[:, 100:300]
    ws = torch.zeros(max(imbd.mlp_local_workspace_bytes(0, 1, 200, 512, 300), 16), dtype=torch.uint8, device=dev)
    imbd.mlp_local_fwd(wblk, xblk, yblk, 1, 1, ws=ws)
    ref = oracle.affine_fwd(Wv[100:300, 8:520], Xv[:, 8:520])
    assert nrm_err(host(yblk), ref) < 1e-5
    assert torch.count_nonzero(ybig[:, :100]).item() == 0 and torch.count_nonzero(ybig[:, 300:]).item() == 0
    # Delta_X of a 264 x 512 block (view of rows 8..272 of a 300 x 520 array): W^T Delta_Y
    w2 = wd[8:272, 8:520]
    dx = torch.empty((300, 512), device=dev)
    dw = torch.empty((264, 512), device=dev)
    ws = torch.zeros(max(imbd.mlp_local_workspace_bytes(1, 1, 264, 512, 300), 16), dtype=torch.uint8, device=dev)
    imbd.mlp_local_bwd(w2, dyd, xblk, dw, 1, 1, dx_part=dx, mask_relu=False, ws=ws)
    assert nrm_err(host(dx), oracle.input_grad(Wv[8:272, 8:520], DYv)) < 1e-5
    # the weight-gradient partial of the same call (fp32 store, scale 1/b)
    rdw, _ = oracle.weight_grad(DYv, Xv[:, 8:520], 1.0 / 300)
    assert nrm_err(host(dw), rdw) < 1e-5


@pytest.mark.parametrize("b", [64, 300])
def test_local_fwd_misaligned_block_fits_its_workspace(imbd, dev, b):
    """A W block whose data starts 2 bytes past a 16-byte boundary fails the skinny (b = 64)
    and wide-batch (b = 300) kernels' alignment checks and runs on the tiled template; the
    workspace sized for its shapes alone must still hold that path's partials."""
    import torch
    rng = np.random.default_rng(9)
    dout, din = 264, 1032
    Wf = rng.standard_normal((dout, din + 8)).astype(np.float32)
    Xf = rng.standard_normal((b, din)).astype(np.float32)
    Wb, Xb = to_bf16_bits(Wf), to_bf16_bits(Xf)
    wd, xd = dev_bf16_bits(Wb, dev), dev_bf16_bits(Xb, dev)
    wblk = wd[:, 1:din + 1]                       # leading dimension din + 8, data 2 bytes off
    assert wblk.data_ptr() % 16 == 2
    y = torch.empty((b, dout), device=dev)
    ws = torch.zeros(max(imbd.mlp_local_workspace_bytes(0, 1, dout, din, b), 16), dtype=torch.uint8, device=dev)
    imbd.mlp_local_fwd(wblk, xd, y, 1, 1, ws=ws)
    ref = oracle.affine_fwd(bf16_values(Wb)[:, 1:din + 1], bf16_values(Xb))
    assert nrm_err(host(y), ref) < 1e-5


def test_local_bwd_empty_block_writes_zero_partials(imbd, dev):
    import torch
    dw = torch.full((5, 7), 3.0, device=dev)
    db = torch.full((5,), 3.0, device=dev)
    w = torch.zeros((5, 7), dtype=torch.bfloat16, device=dev)
    x = torch.zeros((0, 7), dtype=torch.bfloat16, device=dev)
    dy = torch.zeros((0, 5), dtype=torch.bfloat16, device=dev)
    imbd.mlp_local_bwd(w, dy, x, dw, 2, 2, db_part=db)
    torch.cuda.synchronize()
    assert torch.count_nonzero(dw).item() == 0 and torch.count_nonzero(db).item() == 0


def test_split_k_is_deterministic(imbd, dev):
    """Long-K products split K over workgroups; partial sums are added in a fixed order."""
    import torch
    d, W, X, _ = _local_inputs(512, 9216, 64, "bf16", seed=7)
    wd, xd = _to_dev(d, "w", "bf16", dev), _to_dev(d, "x", "bf16", dev)
    ws = torch.zeros(max(imbd.mlp_local_workspace_bytes(0, 1, 512, 9216, 64), 16), dtype=torch.uint8, device=dev)
    assert imbd.mlp_local_workspace_bytes(0, 1, 512, 9216, 64) > 0          # it does split
    y1 = torch.empty((64, 512), device=dev)
    y2 = torch.empty((64, 512), device=dev)
    imbd.mlp_local_fwd(wd, xd, y1, 1, 1, ws=ws)
    imbd.mlp_local_fwd(wd, xd, y2, 1, 1, ws=ws)
    assert torch.equal(y1, y2)
    assert nrm_err(host(y1), oracle.affine_fwd(W, X)) < 1e-5


SKINNY_PLAN_SHAPES = [(130, 200, 70), (64, 64, 64), (200, 1000, 256), (1000, 512, 129), (37, 104, 13),
                      (4096, 1000, 200)]


@pytest.mark.parametrize("nb", [1, 2, 4])
@pytest.mark.parametrize("splits", [1, 3])
@pytest.mark.parametrize("shape", SKINNY_PLAN_SHAPES)
def test_skinny_every_plan(imbd, dev, nb, splits, shape):
    """The B <= 256 product kernel under each forced plan: 64, 128 or 256 samples per
    workgroup (several sample tiles, a ragged last one), K whole (the epilogue applied in
    the product kernel: bias + ReLU + bf16 store, fp32 store, the ReLU mask of Delta_X) or
    split (partials and the reduce). Outputs also as column blocks of a wider array whose
    leading dimension is not a multiple of 4 (element stores instead of vector stores)."""
    import torch
    dout, din, b = shape
    _flush(f"skinny plan nb={nb} splits={splits} {shape}")
    d, W, X, DY = _local_inputs(dout, din, b, "bf16", seed=nb * 10 + splits)
    wd, xd, dyd = _to_dev(d, "w", "bf16", dev), _to_dev(d, "x", "bf16", dev), _to_dev(d, "dy", "bf16", dev)
    bias = dev_f32(d["b"], dev)
    ref = oracle.affine_fwd(W, X, d["b"].astype(np.float64))
    with imbd.options(skinny_nb=nb, skinny_splits=splits):
        nws = max(imbd.mlp_local_workspace_bytes(w, 1, dout, din, b) for w in (0, 1))
        ws = torch.zeros(max(nws, 16), dtype=torch.uint8, device=dev)
        y32 = torch.empty((b, dout), device=dev)
        imbd.mlp_local_fwd(wd, xd, y32, 1, 1, bias=bias, relu=False, ws=ws)
        ybig = torch.full((b, dout + 3), 7.0, device=dev, dtype=torch.bfloat16)
        y16 = ybig[:, 1:dout + 1]
        imbd.mlp_local_fwd(wd, xd, y16, 1, 1, bias=bias, relu=True, ws=ws)
        dx = torch.empty((b, din), device=dev)
        dxbig = torch.full((b, din + 1), 7.0, device=dev)
        dw = torch.empty((dout, din), device=dev)
        imbd.mlp_local_bwd(wd, dyd, xd, dw, 1, 1, dx_part=dx, mask_relu=True, ws=ws)
        imbd.mlp_local_bwd(wd, dyd, xd, dw, 1, 1, dx_part=dxbig[:, :din], mask_relu=False, ws=ws)
        torch.cuda.synchronize()
    assert nrm_err(host(y32), ref) < 1e-5
    assert nrm_err(host(y16), oracle.relu(ref)) < 2.0 ** -8 + 1e-5
    assert torch.all(ybig[:, 0] == 7.0).item() and torch.all(ybig[:, dout + 1:] == 7.0).item()
    assert nrm_err(host(dx), oracle.relu_mask(oracle.input_grad(W, DY), X)) < 1e-5
    assert nrm_err(host(dxbig[:, :din]), oracle.input_grad(W, DY)) < 1e-5
    assert torch.all(dxbig[:, din] == 7.0).item()
