"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test names what fixes the expected value: a hand-worked example, a closed form,
a library routine, central finite differences, an invariant of the mathematics, or
the partition identities of the paper's 1.5D grid (Sec. 2.3, Appendix A). Every
oracle function is covered by at least one pin that a plausible mistake (a dropped
term, a wrong sign or index, a transposed operand) would fail.
"""
import math
import os

import numpy as np
import pytest
import scipy.special

import oracle
from synthdata import make_mlp_inputs, scaled_mlp, to_bf16_bits, bf16_bits_to_f32

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_golden(name):
    vals = {}
    for line in open(os.path.join(GOLDEN, name)):
        line = line.split("#", 1)[0].strip()
        if not line:
            continue
        key, rest = line.split(None, 1)
        rows = [[float(t) for t in r.split()] for r in rest.split(";")]
        arr = np.array(rows if len(rows) > 1 else rows[0])
        vals[key] = arr[0] if arr.size == 1 else arr
    return vals


def _nrm(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


# --------------------------------------------------------------------- hand example
def test_hand_two_layer_example():
    g = _read_golden("hand_two_layer.txt")
    ws = [g["W1"], g["W2"]]
    bs = [np.zeros(2), np.zeros(2)]
    x = g["x"].reshape(1, 2)
    lab = np.array([int(g["label"])], np.int32)
    st = oracle.train_step(ws, bs, x, lab, float(g["eta"]), "f64", want_dx1=True)
    assert np.array_equal(st["acts"][1][0], g["X2"])
    assert np.array_equal(st["logits"][0], g["Z"])
    assert st["loss"] == pytest.approx(float(g["loss"]), abs=1e-15)
    assert np.array_equal(st["dY"][1][0], g["dZ"])
    assert np.array_equal(st["dW"][1], g["dW2"])
    assert np.array_equal(st["db"][1], g["db2"])
    assert np.array_equal(st["dY"][0][0], g["dY1"])
    assert np.array_equal(st["dW"][0], g["dW1"])
    assert np.array_equal(st["db"][0], g["db1"])
    assert np.array_equal(st["dx1"][0], g["dX1"])
    np.testing.assert_allclose(st["w"][0], g["W1new"], atol=1e-15)
    np.testing.assert_allclose(st["w"][1], g["W2new"], atol=1e-15)
    np.testing.assert_allclose(st["b"][0], g["b1new"], atol=1e-15)
    np.testing.assert_allclose(st["b"][1], g["b2new"], atol=1e-15)
    st2 = oracle.forward(st["w"], st["b"], x, lab, "f64")
    np.testing.assert_allclose(st2["logits"][0], g["Znew"], atol=1e-12)
    assert st2["loss"] == pytest.approx(float(g["lossnew"]), abs=1e-10)


def test_hand_example_duplicated_batch_gives_same_mean_gradient():
    """Eq. (1) averages over the batch: two copies of the sample leave the gradient as is."""
    g = _read_golden("hand_two_layer.txt")
    ws, bs = [g["W1"], g["W2"]], [np.zeros(2), np.zeros(2)]
    x = np.vstack([g["x"], g["x"]])
    st = oracle.train_step(ws, bs, x, np.array([0, 0], np.int32), 0.01)
    assert np.array_equal(st["dW"][0], g["dW1"])
    assert np.array_equal(st["dW"][1], g["dW2"])
    assert st["loss"] == pytest.approx(math.log(2), abs=1e-15)


# ------------------------------------------------------------- library-routine pins
def test_affine_fwd_matches_numpy_matmul():
    rng = np.random.default_rng(1)
    W, X, b = rng.standard_normal((37, 53)), rng.standard_normal((11, 53)), rng.standard_normal(37)
    np.testing.assert_allclose(oracle.affine_fwd(W, X, b), X @ W.T + b, rtol=1e-12, atol=1e-12)
    # a transposed operand would break a non-square case
    with pytest.raises(AssertionError):
        oracle.affine_fwd(W, rng.standard_normal((11, 37)))


def test_weight_and_input_grad_match_numpy():
    rng = np.random.default_rng(2)
    dY, X, W = rng.standard_normal((9, 21)), rng.standard_normal((9, 34)), rng.standard_normal((21, 34))
    dW, db = oracle.weight_grad(dY, X, 0.25)
    np.testing.assert_allclose(dW, 0.25 * dY.T @ X, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, 0.25 * dY.sum(0), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.input_grad(W, dY), dY @ W, rtol=1e-12, atol=1e-12)


def test_softmax_xent_matches_scipy_logsumexp():
    rng = np.random.default_rng(3)
    Z = rng.standard_normal((13, 10)) * 30.0      # large logits exercise the max shift
    lab = rng.integers(0, 10, 13).astype(np.int32)
    loss, dZ, rows = oracle.softmax_xent(Z, lab, 1.0 / 13)
    lse = scipy.special.logsumexp(Z, axis=1)
    np.testing.assert_allclose(rows, lse - Z[np.arange(13), lab], rtol=1e-12, atol=1e-12)
    assert loss == pytest.approx(np.mean(lse - Z[np.arange(13), lab]), rel=1e-13)
    P = scipy.special.softmax(Z, axis=1)
    P[np.arange(13), lab] -= 1.0
    np.testing.assert_allclose(dZ, P / 13, rtol=1e-10, atol=1e-14)


def test_round_bf16_matches_torch_cast():
    rng = np.random.default_rng(4)
    f = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * np.float32(10.0) ** rng.integers(-40, 38, 20000).astype(np.float32),
        # exact ties: bf16 value + half an ulp, both parities of the last kept bit
        (np.arange(1, 2000, dtype=np.uint32) << 16 | np.uint32(0x8000)).view(np.float32),
        np.array([1e-45, -1e-45, 1.2e-38, 3.3e38, 3.4e38, -3.4e38, 0.0, -0.0], np.float32),
    ]).astype(np.float32)
    f = f[np.isfinite(f)]
    ref = bf16_bits_to_f32(to_bf16_bits(f)).astype(np.float64)
    got = oracle.round_bf16(f.astype(np.float64))
    assert np.array_equal(got, ref)


def test_round_bf16_hand_cases():
    r = oracle.round_bf16
    u = 2.0 ** -7                        # bf16 ulp at 1
    assert r([1 + u / 2])[0] == 1.0                  # tie, 1 is even
    assert r([1 + 3 * u / 2])[0] == 1 + 2 * u        # tie, rounds up to even
    assert r([1 + u / 2 + 2 ** -30])[0] == 1 + u     # just above the tie
    assert r([-(1 + 3 * u / 2)])[0] == -(1 + 2 * u)
    big = float.fromhex("0x1.fep127")                 # largest finite bf16
    assert r([float.fromhex("0x1.ffp127")])[0] == np.inf   # overflow tie rounds to even -> inf
    assert r([big])[0] == big
    assert r([float.fromhex("0x1.fe7p127")])[0] == big
    assert r([2.0 ** -133 * 1.5])[0] == 2.0 ** -132  # subnormal tie -> even
    assert np.isnan(r([np.nan])[0])


def _nearest_f32_brute_force(x: float) -> float:
    """The binary32 value nearest to x, ties to the even significand, found by exact
    rational comparison of the neighbours of x in the binary32 grid (independent of the
    C conversion the oracle uses)."""
    from fractions import Fraction
    if x == 0.0:
        return x
    big = np.float32(np.finfo(np.float32).max)
    if abs(x) > float(big):
        lo = big
        hi_val = Fraction(2) ** 128          # where the grid would continue past the maximum
    else:
        lo = np.float32(x)                   # a grid point next to x (either side)
        if Fraction(float(lo)) > Fraction(x):
            lo = np.nextafter(lo, np.float32(-np.inf))
        hi = np.nextafter(lo, np.float32(np.inf))
        hi_val = Fraction(float(hi))
    fx, flo = Fraction(x), Fraction(float(lo))
    dlo, dhi = fx - flo, hi_val - fx
    if dlo < dhi:
        return float(lo)
    if dhi < dlo:
        return float(hi_val) if hi_val < Fraction(2) ** 128 else np.inf
    even_lo = int(np.array(lo, np.float32).view(np.uint32)) % 2 == 0
    if even_lo:
        return float(lo)
    return float(hi_val) if hi_val < Fraction(2) ** 128 else np.inf


def test_round_f32_matches_numpy_cast_and_brute_force():
    """binary32 storage rounding (masters, biases, gradients and logits of the bf16 and f32
    modes): against numpy's double -> float cast over the whole binary32 range, and on a
    subset against the exact nearest grid point."""
    rng = np.random.default_rng(14)
    x = np.concatenate([
        rng.standard_normal(20000) * 10.0 ** rng.integers(-46, 39, 20000),
        rng.standard_normal(2000) * 2.0 ** -140,                              # subnormal range
    ])
    f = rng.standard_normal(4000).astype(np.float32)
    f = f[np.isfinite(f) & (f != 0)]
    up = np.nextafter(f, np.float32(np.inf)).astype(np.float64)
    mid = (f.astype(np.float64) + up) / 2.0                                   # exact ties, both parities
    x = np.concatenate([x, mid, [0.0, -0.0, 2.0 ** -150, -(2.0 ** -150), 1.5 * 2.0 ** -149]])
    x = x[np.abs(x) < 3.0e38]
    got = oracle.round_to(x, "f32")
    assert np.array_equal(got, x.astype(np.float32).astype(np.float64))
    for v in np.concatenate([x[::97], mid[:200]]):
        assert oracle.round_to([v], "f32")[0] == _nearest_f32_brute_force(float(v)), v


def test_round_f32_hand_cases():
    r = lambda v: oracle.round_to([v], "f32")[0]
    u = 2.0 ** -23                                    # binary32 ulp at 1
    assert r(1 + u / 2) == 1.0                        # tie, 1 is even
    assert r(1 + 3 * u / 2) == 1 + 2 * u              # tie, rounds up to even
    assert r(1 + u / 2 + 2.0 ** -50) == 1 + u         # just above the tie
    assert r(-(1 + 3 * u / 2)) == -(1 + 2 * u)
    assert r(2.0 ** -150) == 0.0                      # half the smallest subnormal: tie to 0
    assert r(1.5 * 2.0 ** -149) == 2.0 ** -148        # subnormal tie, to even
    assert r(2.0 ** -150 * (1 + 2.0 ** -20)) == 2.0 ** -149
    fmax = float(np.finfo(np.float32).max)
    assert r(fmax) == fmax
    assert r(fmax + 2.0 ** 103) == np.inf             # midpoint to 2^128: tie to even -> inf
    assert r(fmax + 2.0 ** 102) == fmax
    assert np.isnan(r(np.nan)) and r(np.inf) == np.inf


# ------------------------------------------------------------------- closed forms
def test_zero_top_layer_gives_log_c_and_uniform_gradient():
    cfg = scaled_mlp((20, 16, 10), 8, "f32", x_dist="uniform01")
    d = make_mlp_inputs(cfg, seed=5)
    ws = [d["w"][0], np.zeros((10, 16))]
    st = oracle.train_step(ws, [np.zeros(16), np.zeros(10)], d["x"], d["labels"], 0.01)
    assert st["loss"] == pytest.approx(math.log(10), abs=1e-14)
    onehot = np.eye(10)[d["labels"]]
    np.testing.assert_allclose(st["dY"][1], (0.1 - onehot) / 8, atol=1e-16)
    assert np.all(st["dW"][0] == 0) and np.all(st["db"][0] == 0)
    assert math.log(1000) == pytest.approx(6.907755279, abs=1e-9)


def test_single_layer_is_multinomial_logistic_regression():
    rng = np.random.default_rng(6)
    W, X = rng.standard_normal((7, 12)) * 0.3, rng.standard_normal((16, 12))
    lab = rng.integers(0, 7, 16).astype(np.int32)
    st = oracle.train_step([W], [np.zeros(7)], X, lab, 0.05)
    P = scipy.special.softmax(X @ W.T, axis=1)
    Yh = np.eye(7)[lab]
    np.testing.assert_allclose(st["dW"][0], (P - Yh).T @ X / 16, rtol=1e-10, atol=1e-14)


# --------------------------------------------------------------- finite differences
@pytest.mark.parametrize("seed", [0, 1])
def test_gradients_match_central_finite_differences(seed):
    rng = np.random.default_rng(100 + seed)
    dims = (5, 4, 3, 3)
    ws = [rng.standard_normal((dims[i + 1], dims[i])) for i in range(3)]
    bs = [rng.standard_normal(dims[i + 1]) * 0.5 for i in range(3)]
    x = rng.standard_normal((4, 5))
    lab = rng.integers(0, 3, 4).astype(np.int32)
    st = oracle.train_step(ws, bs, x, lab, 0.0, "f64", want_dx1=True)
    # no pre-activation near the ReLU kink
    for i in range(2):
        Y = x @ ws[0].T + bs[0] if i == 0 else st["acts"][1] @ ws[1].T + bs[1]
        if np.min(np.abs(Y)) < 1e-3:
            pytest.skip("sample too close to the kink")
    h = 1e-6
    for li in range(3):
        for arr, grad in ((ws[li], st["dW"][li]), (bs[li], st["db"][li])):
            fd = np.zeros_like(arr)
            for idx in np.ndindex(arr.shape):
                old = arr[idx]
                arr[idx] = old + h
                lp = oracle.loss_only(ws, bs, x, lab)
                arr[idx] = old - h
                lm = oracle.loss_only(ws, bs, x, lab)
                arr[idx] = old
                fd[idx] = (lp - lm) / (2 * h)
            np.testing.assert_allclose(grad, fd, rtol=1e-6, atol=1e-9)
    fdx = np.zeros_like(x)
    for idx in np.ndindex(x.shape):
        old = x[idx]
        x[idx] = old + h
        lp = oracle.loss_only(ws, bs, x, lab)
        x[idx] = old - h
        lm = oracle.loss_only(ws, bs, x, lab)
        x[idx] = old
        fdx[idx] = (lp - lm) / (2 * h)
    np.testing.assert_allclose(st["dx1"], fdx, rtol=1e-6, atol=1e-9)


# ----------------------------------------------------------------------- invariants
def test_invariants_of_one_step():
    cfg = scaled_mlp((30, 24, 16, 10), 8, "f32", x_dist="uniform01")
    d = make_mlp_inputs(cfg, seed=7)
    st = oracle.train_step(d["w"], d["b"], d["x"], d["labels"], 0.01)
    # each column of the top gradient sums to zero (softmax sums to one)
    np.testing.assert_allclose(st["dY"][2].sum(axis=1), 0.0, atol=1e-16)
    assert abs(st["db"][2].sum()) < 1e-15
    # eta = 0 leaves the weights bit-identical
    st0 = oracle.train_step(d["w"], d["b"], d["x"], d["labels"], 0.0)
    for a, b in zip(st0["w"], d["w"]):
        assert np.array_equal(a, b)
    # the update is linear in the gradient
    for i in range(3):
        np.testing.assert_allclose(st["w"][i] - d["w"][i], -0.01 * st["dW"][i], atol=1e-15)
    # W = I, b = 0 reproduces the input
    X = np.random.default_rng(8).standard_normal((5, 6))
    assert np.array_equal(oracle.affine_fwd(np.eye(6), X), X)
    # ReLU mask: entries with zero activation get zero gradient
    for i in (1, 2):
        assert np.all(st["dY"][i - 1][st["acts"][i] == 0] == 0)


def test_shared_relu_decisions_replace_only_the_mask():
    """Passing the iteration's own decisions changes nothing; deciding every unit off
    zeroes every gradient below the top layer and leaves the forward pass and the top
    layer's gradient as they were."""
    cfg = scaled_mlp((20, 12, 8, 5), 6, "bf16")
    d = make_mlp_inputs(cfg, seed=12)
    x = bf16_bits_to_f32(d["x_bits"])
    own = oracle.train_step(d["w"], d["b"], x, d["labels"], 0.01, "bf16")
    same = oracle.train_step(d["w"], d["b"], x, d["labels"], 0.01, "bf16", relu_decisions=own["acts"])
    for k in ("dY", "dW", "db", "w", "b"):
        for a, b in zip(own[k], same[k]):
            assert np.array_equal(a, b), k
    off = [None] + [np.zeros_like(a) for a in own["acts"][1:]]
    z = oracle.train_step(d["w"], d["b"], x, d["labels"], 0.01, "bf16", relu_decisions=off)
    assert np.array_equal(z["logits"], own["logits"]) and z["loss"] == own["loss"]
    assert np.array_equal(z["dY"][2], own["dY"][2]) and np.array_equal(z["dW"][2], own["dW"][2])
    for i in (0, 1):
        assert not z["dY"][i].any() and not z["dW"][i].any() and not z["db"][i].any()


def test_bf16_mode_rounds_exactly_at_storage_points():
    cfg = scaled_mlp((64, 48, 32, 10), 16, "bf16")
    d = make_mlp_inputs(cfg, seed=9)
    x = bf16_bits_to_f32(d["x_bits"])
    st = oracle.train_step(d["w"], d["b"], x, d["labels"], 0.01, "bf16")
    for a in st["acts"][1:] + st["dY"] + st["w_op"] + st["w_bf16"]:
        assert np.array_equal(oracle.round_bf16(a), a)
    for a in st["w"] + st["b"] + [st["logits"]]:
        assert np.array_equal(oracle.round_to(a, "f32"), a)
    ref = oracle.train_step(d["w"], d["b"], x, d["labels"], 0.01, "f64")
    assert abs(st["loss"] - ref["loss"]) < 2e-2 * abs(ref["loss"])


# ------------------------------------------------------------ 1.5D partition identities
@pytest.mark.parametrize("P_r,P_c", [(2, 4), (4, 2), (1, 4), (4, 1), (3, 2)])
def test_grid_partials_reassemble_the_unpartitioned_layer(P_r, P_c):
    """App. A: Y blocks concatenate over r; dW partials sum over c; dX partials sum over r.
    P_r = 1 is pure batch parallelism, P_c = 1 pure model parallelism (Sec. 2.2)."""
    rng = np.random.default_rng(10)
    dout, din, B = 12, 10, 8
    W, b = rng.standard_normal((dout, din)), rng.standard_normal(dout)
    X, dY = rng.standard_normal((B, din)), rng.standard_normal((B, dout))
    mask_src = np.maximum(rng.standard_normal((B, din)), 0)
    Y, dW, db, dX = oracle.grid_layer(W, b, X, dY, P_r, P_c, 1.0 / B, mask_src)
    np.testing.assert_allclose(Y, X @ W.T + b, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dW, dY.T @ X / B, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, dY.sum(0) / B, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dX, (dY @ W) * (mask_src > 0), rtol=1e-12, atol=1e-12)


def test_grid_detects_a_missing_process():
    """A dropped rank (one partial lost) must show up in the reassembled gradient."""
    rng = np.random.default_rng(11)
    W, X, dY = rng.standard_normal((8, 6)), rng.standard_normal((8, 6)), rng.standard_normal((8, 8))
    full, _ = oracle.weight_grad(dY, X, 1 / 8)
    part = np.zeros_like(full)
    for c in range(3):                               # process column 3 of 4 never reports
        cs = oracle.block_rows(8, 4, c)
        part += oracle.local_bwd(W, dY[cs], X[cs], 1 / 8)[0]
    assert not np.allclose(part, full)
    with pytest.raises(ValueError):
        oracle.block_rows(10, 4, 0)


def test_grid_simulation_of_a_whole_network_step():
    """Run every layer of a 3-layer step through the software grid and compare with the
    unpartitioned step (the top layer's softmax on the gathered logits: softmax needs whole
    columns, so each process slices its rows of the gradient afterwards)."""
    cfg = scaled_mlp((24, 16, 16, 8), 8, "f32", x_dist="normal")
    d = make_mlp_inputs(cfg, seed=12)
    ref = oracle.train_step(d["w"], d["b"], d["x"], d["labels"], 0.01)
    P_r, P_c = 2, 4
    acts = [np.asarray(d["x"], np.float64)]
    for i in range(3):
        Y, *_ = oracle.grid_layer(d["w"][i], d["b"][i], acts[i], np.zeros((8, cfg.dims[i + 1])),
                                  P_r, P_c, 1.0 / 8, apply_relu=i < 2)
        acts.append(Y)
    loss, dZ, _ = oracle.softmax_xent(acts[3], d["labels"], 1.0 / 8)
    assert loss == pytest.approx(ref["loss"], rel=1e-12)
    dY = dZ * 8   # raw per-sample gradient; partials carry 1/B_global
    for i in range(2, -1, -1):
        mask = acts[i] if i > 0 else None
        _, dW, db, dX = oracle.grid_layer(d["w"][i], d["b"][i], acts[i], dY, P_r, P_c, 1.0 / 8, mask)
        np.testing.assert_allclose(dW, ref["dW"][i], rtol=1e-11, atol=1e-14)
        np.testing.assert_allclose(db, ref["db"][i], rtol=1e-11, atol=1e-14)
        if i > 0:
            np.testing.assert_allclose(dX / 8, ref["dY"][i - 1], rtol=1e-11, atol=1e-14)
        dY = dX


# ---------------------------------------------------------------------- conv pins
def _full_conv_numpy(x_pad, w):
    """Library cross-check: scipy correlate per (o, c) pair (textbook definition)."""
    import scipy.signal
    N, Hp, Wp, Ci = x_pad.shape
    Co = w.shape[0]
    y = np.zeros((N, Hp - 2, Wp - 2, Co))
    for n in range(N):
        for o in range(Co):
            for c in range(Ci):
                y[n, :, :, o] += scipy.signal.correlate2d(x_pad[n, :, :, c], w[o, :, :, c], mode="valid")
    return y


def test_conv_fwd_matches_scipy_correlate():
    rng = np.random.default_rng(13)
    xp, w = rng.standard_normal((2, 7, 6, 3)), rng.standard_normal((4, 3, 3, 3))
    np.testing.assert_allclose(oracle.conv3x3_fwd(xp, w), _full_conv_numpy(xp, w), rtol=1e-12, atol=1e-12)


def test_conv_1x1_and_delta_kernels():
    rng = np.random.default_rng(14)
    xp = rng.standard_normal((2, 6, 5, 4))
    w = np.zeros((3, 3, 3, 4))
    A = rng.standard_normal((3, 4))
    w[:, 1, 1, :] = A                                     # 1x1 conv = GEMM over channels
    np.testing.assert_allclose(oracle.conv3x3_fwd(xp, w), xp[:, 1:-1, 1:-1, :] @ A.T, rtol=1e-12)
    d = np.zeros((4, 3, 3, 4))
    d[:, 1, 1, :] = np.eye(4)                             # centre tap = identity copies the interior
    assert np.array_equal(oracle.conv3x3_fwd(xp, d), xp[:, 1:-1, 1:-1, :])


def test_conv_stitched_tiles_equal_full_image():
    """Domain parallelism (Sec. 2.2): a 2x2 split with exchanged halos reproduces the
    full-image conv, the summed dW and the full dX."""
    rng = np.random.default_rng(15)
    N, H, W, Ci, Co = 2, 8, 6, 3, 4
    x = rng.standard_normal((N, H, W, Ci))
    dy = rng.standard_normal((N, H, W, Co))
    w = rng.standard_normal((Co, 3, 3, Ci))
    xpf = np.pad(x, ((0, 0), (1, 1), (1, 1), (0, 0)))
    dypf = np.pad(dy, ((0, 0), (1, 1), (1, 1), (0, 0)))
    y_full = oracle.conv3x3_fwd(xpf, w)
    dx_full = oracle.conv3x3_dgrad(dypf, w)
    dw_full = oracle.conv3x3_wgrad(xpf, dypf)
    th, tw = H // 2, W // 2
    y = np.zeros_like(y_full)
    dx = np.zeros_like(dx_full)
    dw = np.zeros_like(dw_full)
    for ti in range(2):
        for tj in range(2):
            hs, ws_ = ti * th, tj * tw
            xt = xpf[:, hs:hs + th + 2, ws_:ws_ + tw + 2]
            dyt = dypf[:, hs:hs + th + 2, ws_:ws_ + tw + 2]
            y[:, hs:hs + th, ws_:ws_ + tw] = oracle.conv3x3_fwd(xt, w)
            dx[:, hs:hs + th, ws_:ws_ + tw] = oracle.conv3x3_dgrad(dyt, w)
            dw += oracle.conv3x3_wgrad(xt, dyt)
    np.testing.assert_allclose(y, y_full, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dx, dx_full, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw, dw_full, rtol=1e-12, atol=1e-12)


def test_conv_gradients_match_finite_differences():
    """L = 0.5 * sum(y * g) for a fixed g: dL/dw = wgrad(x, g) and dL/dx = dgrad(g)."""
    rng = np.random.default_rng(16)
    N, H, W, Ci, Co = 1, 4, 4, 2, 2
    x = rng.standard_normal((N, H, W, Ci))
    w = rng.standard_normal((Co, 3, 3, Ci))
    g = rng.standard_normal((N, H, W, Co))
    gp = np.pad(g, ((0, 0), (1, 1), (1, 1), (0, 0)))

    def L(x_, w_):
        return float(np.sum(oracle.conv3x3_fwd(np.pad(x_, ((0, 0), (1, 1), (1, 1), (0, 0))), w_) * g))

    h = 1e-6
    fdw = np.zeros_like(w)
    for idx in np.ndindex(w.shape):
        o = w[idx]
        w[idx] = o + h; lp = L(x, w)
        w[idx] = o - h; lm = L(x, w)
        w[idx] = o
        fdw[idx] = (lp - lm) / (2 * h)
    fdx = np.zeros_like(x)
    for idx in np.ndindex(x.shape):
        o = x[idx]
        x[idx] = o + h; lp = L(x, w)
        x[idx] = o - h; lm = L(x, w)
        x[idx] = o
        fdx[idx] = (lp - lm) / (2 * h)
    xp = np.pad(x, ((0, 0), (1, 1), (1, 1), (0, 0)))
    np.testing.assert_allclose(oracle.conv3x3_wgrad(xp, gp), fdw, rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose(oracle.conv3x3_dgrad(gp, w), fdx, rtol=1e-6, atol=1e-8)


def test_conv_sampled_entry_points_agree_with_full():
    rng = np.random.default_rng(17)
    xp, w, dyp = rng.standard_normal((2, 6, 7, 3)), rng.standard_normal((5, 3, 3, 3)), rng.standard_normal((2, 6, 7, 5))
    y, dx, dw = oracle.conv3x3_fwd(xp, w), oracle.conv3x3_dgrad(dyp, w), oracle.conv3x3_wgrad(xp, dyp)
    for full, fn, a, b in ((y, oracle.conv3x3_fwd_at, xp, w), (dx, oracle.conv3x3_dgrad_at, dyp, w),
                           (dw, oracle.conv3x3_wgrad_at, xp, dyp)):
        idx = rng.choice(full.size, 40, replace=False)
        np.testing.assert_allclose(fn(a, b, idx), full.reshape(-1)[idx], rtol=1e-12, atol=1e-12)
