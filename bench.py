"""Throughput of the data-parallel hot path on one MI355X.

A step is one full SGD iteration of the 9216-4096-4096-1000 fully connected stack at
B = 256 (AlexNet-style FC layers, bf16 operands, fp32 accumulation, fp32 master weights,
ReLU, softmax cross-entropy, update fused into the weight-gradient kernels), on one fixed
synthetic batch already resident in HBM.

Prints one JSON line: the metric (algorithmic TFLOP/s of fwd + bwd + SGD), samples/s,
fraction of the bf16 MFMA peak, a roofline entry for the dominant kernel (the layer-1
weight-gradient kernel with the fused update, timed with HIP events inside the timed
region's twin) and the CPU oracle timed on a bounded sample of the same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
(--workload conv3x3_tile measures the domain-parallel conv tile instead of the FC step;
--workload batch_sweep times the FC step at batch sizes 1..2048, --stack alexnet|vgg;
--workload alexnet_fc_local_4x16 times one process's local blocks of a 4 x 16 grid;
--workload grid_model times one process's local blocks of the FC stack for every P_r x P_c
grid of --procs and picks the grid with the cost model of paper_1712_04432_amd.gridmodel)
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "fwd+bwd+SGD TFLOP/s and samples/s per GPU; % of MFMA dense peak"
PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "dw_sgd_alexnet_l1_traffic.txt")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_1712_04432_amd", "csrc", f) for f in ("dw_sgd.hip", "cdna4.h", "common.h")]


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per launch of the dominant kernel from rocprofv3 FETCH_SIZE/WRITE_SIZE
    runs, kept only for the workload they were taken on and while the kernel source is the
    one the counters were taken on."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    kv = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_hash") != kernel_source_hash() or kv.get("workload") != workload:
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def dw_sgd_bytes(d_out: int, d_in: int, batch: int, act_bytes: int = 2) -> int:
    """Algorithmic bytes of one fused weight-gradient + update launch: the fp32 master is
    read and written, the bf16 copy written (10 B per parameter; 8 B for an fp32 network,
    whose master is its operand), X and Delta_Y read once."""
    copy = 2 if act_bytes == 2 else 0
    return d_out * d_in * (4 + 4 + copy) + batch * (d_in + d_out) * act_bytes


def cpu_model() -> str:
    """The host CPU's model name (as lscpu prints it), or "unknown"."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, sample_batch: int = 0, min_seconds: float = 10.0, single_thread_batch: int = 16,
                 relu_decisions=None):
    """The oracle, as it is, on SGD iterations of the same network over `sample_batch`
    samples (0: the whole batch; the full weights and update are processed either way),
    repeated until `min_seconds` have passed; the rate is over all iterations. Then one
    iteration on one thread over `single_thread_batch` samples (0: skip).

    Returns (record, first iteration's result): the latter is the oracle's own step from the
    seeded state over the whole batch (None when the sample is smaller), against which the
    device's first step is compared. relu_decisions (whole batch only): the device's ReLU
    derivative decisions of that step, taken by the oracle's backward pass (see
    oracle.train_step)."""
    import numpy as np

    import oracle
    from synthdata import bf16_bits_to_f32, make_mlp_inputs
    n = sample_batch or cfg.batch
    d = make_mlp_inputs(cfg, seed=0, batch=n)
    bf16 = cfg.dtype == "bf16"
    mode = "bf16" if bf16 else "f32"
    xv = (bf16_bits_to_f32(d["x_bits"]) if bf16 else d["x"]).astype(np.float64)
    iters, first = 0, None
    threads = oracle.threads()
    t0 = time.perf_counter()
    dec = relu_decisions if n == cfg.batch else None
    while True:
        r = oracle.train_step(d["w"], d["b"], xv, d["labels"], cfg.lr, mode, relu_decisions=dec)
        if iters == 0 and n == cfg.batch:
            first = {"loss": r["loss"], "w": r["w"], "b": r["b"], "acts": r["acts"]}
        del r
        iters += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    flops = iters * cfg.gemm_flops(batch=n)
    whole = "all" if n == cfg.batch else f"{n} of the"
    rec = {"value": round(flops / dt / 1e12, 9), "unit": "TFLOP/s", "cores": threads,
           "kind": "oracle", "cpu_model": cpu_model(),
           "sample": f"{iters} SGD iteration(s) of the {'-'.join(map(str, cfg.dims))} stack on {whole} "
                     f"{cfg.batch} samples (full weights and update), "
                     f"{'bf16-mirrored' if bf16 else 'fp32-mirrored'} fp64 oracle, "
                     f"{dt:.2f} s = {iters * n / dt:.3f} samples/s"}
    if single_thread_batch:
        m1 = min(single_thread_batch, cfg.batch)
        sl = slice(0, m1)
        oracle.set_threads(1)
        try:
            t1 = time.perf_counter()
            oracle.train_step(d["w"], d["b"], xv[sl], d["labels"][sl], cfg.lr, mode)
            dt1 = time.perf_counter() - t1
        finally:
            oracle.set_threads(threads)
        rec["single_thread"] = {
            "value": round(cfg.gemm_flops(batch=m1) / dt1 / 1e12, 9), "unit": "TFLOP/s", "cores": 1,
            "sample": f"1 SGD iteration on {m1} of the {cfg.batch} samples (full weights and update), "
                      f"{dt1:.2f} s = {m1 / dt1:.3f} samples/s"}
    return rec, first


def parity_vs_oracle(first_dev, w0, b0, ref):
    """Normwise errors max|g - o| / max|o| of the device's first step against the oracle's
    first iteration from the same seeded state: the hidden activations, the update W' - W
    and b' - b of every layer and the loss; and how many ReLU derivative decisions the two
    sides took differently (the oracle's backward pass takes the device's)."""
    import numpy as np
    errs = {"loss": abs(first_dev["loss"] - ref["loss"]) / abs(ref["loss"])}
    flips = {}
    for i, xd in enumerate(first_dev["acts"], start=1):
        xr = ref["acts"][i]
        errs[f"X{i + 1}"] = float(np.max(np.abs(xd - xr)) / np.max(np.abs(xr)))
        flips[f"X{i + 1}"] = int(((xd > 0) != (xr > 0)).sum())
    for i, (wn, bn) in enumerate(zip(first_dev["w"], first_dev["b"])):
        for tag, new, old, o in (("dW", wn, w0[i], ref["w"][i]), ("db", bn, b0[i], ref["b"][i])):
            g = new.astype(np.float64) - old
            r = o - old
            den = np.max(np.abs(r))
            errs[f"{tag}{i + 1}"] = float(np.max(np.abs(g - r)) / den) if den > 0 else float(np.max(np.abs(g)))
    return {"max_normwise_err": max(errs.values()), "per_tensor": {k: float(f"{v:.3e}") for k, v in errs.items()},
            "relu_decisions_differing": flips,
            "compared": "first fused step from the seeded state: hidden activations, W' - W and b' - b of every "
                        "layer, loss (ReLU derivative decisions shared)",
            "oracle_mode": "bf16-mirrored fp64"}


def conv_cpu_baseline(cfg, images: int = 8):
    """The oracle's three conv passes on `images` of the tile's images."""
    import numpy as np

    import oracle
    from synthdata import bf16_bits_to_f32, make_conv_inputs
    d = make_conv_inputs(images, cfg.tile_h, cfg.tile_w, cfg.c_in, cfg.c_out, seed=0)
    xv = bf16_bits_to_f32(d["x_bits"]).astype(np.float64)
    wv = bf16_bits_to_f32(d["w_bits"]).astype(np.float64)
    dyv = bf16_bits_to_f32(d["dy_bits"]).astype(np.float64)
    t0 = time.perf_counter()
    oracle.conv3x3_fwd(xv, wv)
    oracle.conv3x3_dgrad(dyv, wv)
    oracle.conv3x3_wgrad(xv, dyv)
    dt = time.perf_counter() - t0
    flops = 3 * 2 * images * cfg.tile_h * cfg.tile_w * cfg.c_out * 9 * cfg.c_in
    return {"value": round(flops / dt / 1e12, 9), "unit": "TFLOP/s", "cores": oracle.threads(), "kind": "oracle",
            "sample": f"forward + input gradient + weight gradient of the 3x3 tile on {images} of the "
                      f"{cfg.batch} images, fp64 oracle, {dt:.2f} s"}


def bench_conv(args):
    """Domain-parallel conv tile: forward + input gradient + weight gradient per step."""
    import numpy as np
    import torch

    import paper_1712_04432_amd as m
    from synthdata import get_config, make_conv_inputs

    m.load()
    cfg = get_config("conv3x3_tile")
    dev = torch.device("cuda:0")
    N, H, W, Ci, Co = cfg.batch, cfg.tile_h, cfg.tile_w, cfg.c_in, cfg.c_out
    log(f"bench: conv tile {N}x{H}x{W}, {Ci}->{Co}")
    d = make_conv_inputs(N, H, W, Ci, Co, seed=0)
    as_bf16 = lambda b: torch.from_numpy(b.view(np.int16)).to(dev).view(torch.bfloat16)
    x, w, dy = as_bf16(d["x_bits"]), as_bf16(d["w_bits"]), as_bf16(d["dy_bits"])
    y = torch.empty((N, H, W, Co), dtype=torch.bfloat16, device=dev)
    dx = torch.empty((N, H, W, Ci), dtype=torch.bfloat16, device=dev)
    dw = torch.empty((Co, 3, 3, Ci), device=dev)
    ws = torch.zeros(max(m.conv3x3_wgrad_workspace_bytes(N, H, W, Ci, Co), 16), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        m.conv3x3_tile_fwd(x, w, y, stream=stream)
        m.conv3x3_tile_dgrad(dy, w, dx, stream=stream)
        m.conv3x3_tile_wgrad(x, dy, dw, ws=ws, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(args.steps):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(stop) / args.steps
    per_pass = 2 * N * H * W * Co * 9 * Ci
    flops = 3 * per_pass
    tflops = flops / (ms_step * 1e-3) / 1e12
    kinfo = {}
    for name, cls in (("forward", m.IMBD_K_CONV_FWD), ("input_grad", m.IMBD_K_CONV_DGRAD),
                      ("weight_grad", m.IMBD_K_CONV_WGRAD)):
        m.timing_begin(cls, -1, args.steps)
        for _ in range(args.steps):
            step()
        n, kms = m.timing_end()
        kinfo[name] = kms / max(n, 1)
    torch.cuda.synchronize()
    dom = max(kinfo, key=kinfo.get)
    achieved = per_pass / (kinfo[dom] * 1e-3) / 1e12
    result = {
        "metric": METRIC, "value": round(tflops, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) activations and gradients, N(0, 2/(9*256)) weights)",
        "config": {"workload": f"conv3x3_tile: 3x3 stride-1 conv, {Ci}->{Co} channels, {H}x{W} tile of a "
                               f"224x224 image split 4x4, 1-pixel halo supplied, batch {N}; forward + input "
                               f"gradient + weight gradient", "global_batch": N, "parallelism": "single GPU"},
        "samples_per_s": round(N / (ms_step * 1e-3), 1),
        "pct_bf16_mfma_peak": round(100.0 * tflops / PEAK_BF16_TFLOPS, 3),
        "gflop_per_step": round(flops / 1e9, 4),
        "roofline": {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": None,
                     "kernel": f"conv tile {dom} pass", "algorithmic_flops_per_launch": per_pass,
                     "avg_launch_ms": {k: round(v, 5) for k, v in kinfo.items()}},
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = conv_cpu_baseline(cfg)
    print(json.dumps(result), flush=True)


def step_hbm_bytes(dims, batch: int) -> int:
    """Algorithmic HBM bytes of one fused SGD iteration of a bf16 FC stack: per layer the
    bf16 weights read by the forward and Delta_X products, the fp32 master read and written
    and the bf16 copy written by the fused update (10 B per weight), and the activations,
    gradients and logits read or written once per product."""
    total = 0
    L = len(dims) - 1
    for i in range(1, L + 1):
        din, dout = dims[i - 1], dims[i]
        w = din * dout
        total += 2 * w + 2 * batch * (din + dout)                       # forward
        if i >= 2:
            total += 2 * w + 2 * batch * dout + 4 * batch * din         # Delta_X (+ mask)
        total += 10 * w + 2 * batch * (din + dout)                      # Delta_W + update
    total += 8 * batch * dims[L]                                        # logits, softmax
    return total


def bench_batch_sweep(args):
    """Step time of the FC stack against the batch size (the single-GPU analogue of the
    paper's per-batch timing of the forward and backward passes): one fixed synthetic batch
    per size, the weights shared, fused SGD as in the default workload."""
    import numpy as np
    import torch

    import paper_1712_04432_amd as m
    from synthdata import get_config, make_mlp_inputs, scaled_mlp

    m.load()
    base = get_config("alexnet_fc_b256" if args.stack == "alexnet" else "vgg_fc_b512")
    dev = torch.device("cuda:0")
    batches = [int(b) for b in args.batches.split(",")]
    d = make_mlp_inputs(base, seed=0, batch=1)
    w32 = [torch.from_numpy(w).to(dev) for w in d["w"]]
    rows = []
    for B in batches:
        cfg = scaled_mlp(base.dims, B, "bf16", x_dist=base.x_dist, name=f"{base.name.split('_b')[0]}_b{B}")
        db = make_mlp_inputs(cfg, seed=1, batch=B)
        net = m.MLP(cfg.dims, B, "bf16")
        layers = []
        for w, b in zip(w32, db["b"]):
            wm = w.clone()
            wlp = torch.empty(w.shape, dtype=torch.bfloat16, device=dev)
            m.cast_f32_bf16(wm, wlp)
            layers.append({"w": wm, "w_lp": wlp, "b": torch.from_numpy(b).to(dev)})
        x = torch.from_numpy(db["x_bits"].view(np.int16)).to(dev).view(torch.bfloat16)
        lab = torch.from_numpy(db["labels"]).to(dev)
        ws = torch.zeros(m.mlp_workspace_bytes(net), dtype=torch.uint8, device=dev)
        loss = torch.zeros(1, device=dev)
        stream = torch.cuda.current_stream()
        for _ in range(args.warmup):
            m.mlp_train_step(net, layers, x, lab, ws, cfg.lr, loss, stream=stream)
        torch.cuda.synchronize()
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(stream)
        for _ in range(args.steps):
            m.mlp_train_step(net, layers, x, lab, ws, cfg.lr, loss, stream=stream)
        stop.record(stream)
        torch.cuda.synchronize()
        ms = start.elapsed_time(stop) / args.steps
        flops = cfg.gemm_flops()
        hbm = step_hbm_bytes(cfg.dims, B)
        t_hbm_ms = hbm / (PEAK_HBM_GBS * 1e9) * 1e3
        t_mfma_ms = flops / (PEAK_BF16_TFLOPS * 1e12) * 1e3
        rows.append({"batch": B, "ms_per_step": round(ms, 5), "tflops": round(flops / (ms * 1e-3) / 1e12, 3),
                     "samples_per_s": round(B / (ms * 1e-3), 1),
                     "pct_bf16_mfma_peak": round(100.0 * flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 3),
                     "roofline_ms": round(max(t_hbm_ms, t_mfma_ms), 5),
                     "roofline_bound": "hbm" if t_hbm_ms >= t_mfma_ms else "mfma",
                     "frac_of_roofline": round(max(t_hbm_ms, t_mfma_ms) / ms, 4),
                     "loss": round(loss.item(), 5)})
        log(f"bench: B={B} {ms * 1e3:.1f} us/step, {rows[-1]['tflops']} TFLOP/s")
        del layers, x, lab, ws, net
        torch.cuda.empty_cache()
    print(json.dumps({"metric": "FC step time and TFLOP/s against the batch size", "unit": "TFLOP/s",
                      "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "dtype": "bf16",
                      "data": "synthetic (seeded inputs and labels per batch size, He-initialised weights)",
                      "config": {"workload": f"batch_sweep: {'-'.join(map(str, base.dims))} FC stack, fused SGD",
                                 "parallelism": "single GPU"},
                      "sweep": rows}), flush=True)


# Collective parameters for the grid model (assumptions, not measured: one GPU here).
# xGMI inside an 8-GPU node: ~2 us per message, ring all-reduce bus bandwidth ~300 GB/s;
# between nodes: ~5 us, ~50 GB/s per GPU (8 x 400 Gb/s NICs per node); the paper's Cori
# simulation: 2 us, 6 GB/s.
NETWORKS = {"xgmi_node": (2e-6, 1 / 300e9), "multi_node": (5e-6, 1 / 50e9), "paper_cori": (2e-6, 1 / 6e9)}


def bench_grid_model(args):
    """Per-process compute of the 1.5D layout measured on the device (local forward, local
    backward with the Delta_W and Delta_X partials, SGD of the process's weight block, bf16
    blocks of the FC stack as the grid cuts them, the largest block when the cut is uneven)
    and the grid each network's collective parameters select (Sec. 2.3 cost + compute)."""
    import torch

    import paper_1712_04432_amd as m
    from paper_1712_04432_amd import gridmodel as gm
    from synthdata import get_config

    m.load()
    base = get_config("alexnet_fc_b256" if args.stack == "alexnet" else "vgg_fc_b512")
    dims, B = base.dims, args.grid_batch
    layers = [gm.FC(dims[i - 1], dims[i]) for i in range(1, len(dims))]
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    cache = {}

    def time_layer(d_out, d_in, b, first):
        key = (d_out, d_in, b, first)
        if key in cache:
            return cache[key]
        g = torch.Generator(device=dev).manual_seed(0)
        w = (torch.randn(d_out, d_in, device=dev, generator=g) * 0.01)
        wl = w.to(torch.bfloat16)
        x = torch.randn(b, d_in, device=dev, generator=g).relu().to(torch.bfloat16)
        y = torch.empty(b, d_out, dtype=torch.bfloat16, device=dev)
        dy = (torch.randn(b, d_out, device=dev, generator=g) * 0.01).to(torch.bfloat16)
        dw = torch.empty(d_out, d_in, device=dev)
        db = torch.empty(d_out, device=dev)
        bias = torch.zeros(d_out, device=dev)
        dx = None if first else torch.empty(b, d_in, device=dev)
        wsz = max(m.mlp_local_workspace_bytes(0, m.IMBD_BF16, d_out, d_in, b),
                  m.mlp_local_workspace_bytes(1, m.IMBD_BF16, d_out, d_in, b), 16)
        ws = torch.zeros(wsz, dtype=torch.uint8, device=dev)

        def run():
            m.mlp_local_fwd(wl, x, y, 1, 1, bias=bias, relu=True, ws=ws, stream=stream)
            m.mlp_local_bwd(wl, dy, x, dw, 1, 1, db_part=db, dx_part=dx, mask_relu=not first, ws=ws,
                            stream=stream)
            m.sgd_step(w, dw, 0.01, 1.0 / B, w_lp=wl, stream=stream)
        for _ in range(2):
            run()
        torch.cuda.synchronize()
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record(stream)
        for _ in range(args.steps):
            run()
        s1.record(stream)
        torch.cuda.synchronize()
        cache[key] = s0.elapsed_time(s1) / args.steps * 1e-3
        return cache[key]

    def t_comp(P_r, P_c):
        b = -(-B // P_c)
        return sum(time_layer(-(-l.d_out // P_r), l.d_in, b, i == 0) for i, l in enumerate(layers))

    procs = [int(p) for p in args.procs.split(",")]
    out = {"metric": "1.5D grid choice for the FC stack: modelled time per iteration (s)", "n_gpus": 1,
           "config": {"workload": f"grid_model: {'-'.join(map(str, dims))} FC stack, B = {B}, bf16 local blocks",
                      "networks": {k: {"alpha_s": a, "bandwidth_GBs": round(1 / b / 1e9, 1)}
                                   for k, (a, b) in NETWORKS.items()}},
           "grids": []}
    for P in procs:
        comp = {(r, P // r): t_comp(r, P // r) for r, _ in gm.grids(P)}
        entry = {"P": P, "comp_s": {f"{r}x{c}": round(v, 7) for (r, c), v in comp.items()}, "choice": {}}
        for name, (a, bt) in NETWORKS.items():
            best, rows = gm.select_grid(layers, B, P, a, bt, elem_bytes=4, t_comp=lambda r, c: comp[(r, c)],
                                        divisible=False)
            pure = [r for r in rows if r["P_r"] == 1][0]
            bestrow = [r for r in rows if (r["P_r"], r["P_c"]) == best][0]
            entry["choice"][name] = {"grid": f"{best[0]}x{best[1]}", "total_s": round(bestrow["total"], 7),
                                     "comm_s": round(bestrow["comm"], 7),
                                     "batch_grid_total_s": round(pure["total"], 7),
                                     "speedup_over_batch": round(pure["total"] / bestrow["total"], 3)}
        log(f"bench: P={P} " + " ".join(f"{k}:{v['grid']}" for k, v in entry["choice"].items()))
        out["grids"].append(entry)
    print(json.dumps(out), flush=True)


def local_block_bytes(d_out: int, d_in: int, b: int, first: bool) -> int:
    """Algorithmic bytes of one layer's local forward + backward (bf16 blocks): W_blk read by
    the forward and (past the first layer) the Delta_X product, the fp32 Delta_W partial
    written, X_blk read twice (forward, Delta_W), Y_blk (bf16) written, Delta_Y_blk read
    twice, the fp32 Delta_X partial written and its ReLU mask read."""
    w = d_out * d_in * (2 + (0 if first else 2) + 4)
    act = b * d_in * 2 * 2 + b * d_out * 2 + b * d_out * 2 * 2
    if not first:
        act += b * d_in * (4 + 2)
    return w + act


def bench_local(args, cfg):
    """One process's share of the 1.5D grid (the local-block variant): for every layer the
    local forward (bias + ReLU; the top layer's logits are gathered before softmax, so its
    block stores them plain) and the local backward (fp32 Delta_W partial, bias partial,
    masked fp32 Delta_X partial from layer 2 on), on the blocks of a P_r x P_c grid. The
    partials are left unreduced, as the collectives of Sec. 2.3 would take them."""
    import numpy as np
    import torch

    import paper_1712_04432_amd as m
    from synthdata import make_local_inputs

    m.load()
    P_r, P_c = cfg.grid
    b = cfg.batch // P_c
    dims = cfg.dims
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    L = len(dims) - 1
    jobs, flops, hbm = [], 0, 0
    for i in range(1, L + 1):
        d_out, d_in, first = -(-dims[i] // P_r), dims[i - 1], i == 1
        d = make_local_inputs(d_out, d_in, b, seed=i)
        w = torch.from_numpy(d["w_bits"].view(np.int16)).to(dev).view(torch.bfloat16)
        x = torch.from_numpy(d["x_bits"].view(np.int16)).to(dev).view(torch.bfloat16)
        dy = torch.from_numpy(d["dy_bits"].view(np.int16)).to(dev).view(torch.bfloat16)
        bias = torch.from_numpy(d["b"]).to(dev)
        y = torch.empty(b, d_out, dtype=torch.bfloat16, device=dev)
        dw = torch.empty(d_out, d_in, device=dev)
        db = torch.empty(d_out, device=dev)
        dx = None if first else torch.empty(b, d_in, device=dev)
        wsz = max(m.mlp_local_workspace_bytes(0, m.IMBD_BF16, d_out, d_in, b),
                  m.mlp_local_workspace_bytes(1, m.IMBD_BF16, d_out, d_in, b), 16)
        ws = torch.zeros(wsz, dtype=torch.uint8, device=dev)
        jobs.append((w, x, dy, bias, y, dw, db, dx, ws, first, i < L))
        flops += 2 * d_out * d_in * b * (2 if first else 3)
        hbm += local_block_bytes(d_out, d_in, b, first)

    def step(st):
        for w, x, dy, bias, y, dw, db, dx, ws, first, hidden in jobs:
            m.mlp_local_fwd(w, x, y, P_r, P_c, bias=bias, relu=hidden, ws=ws, stream=st)
            m.mlp_local_bwd(w, dy, x, dw, P_r, P_c, db_part=db, dx_part=dx, mask_relu=not first, ws=ws,
                            stream=st)
    for _ in range(args.warmup):
        step(stream)
    torch.cuda.synchronize()
    # The step is nine launches of 3-11 us from six calls, and the host's marshalling and planning
    # of those calls takes about as long as the GPU (~53 us a step): launched from Python the timed
    # steps measure the host after a long warm-up. The K timed steps are therefore captured once
    # into a HIP graph (the library launches only kernels on the stream it is given: no
    # allocation, copy, fill or synchronisation) and replayed; one untimed replay precedes the
    # timed one.
    graph, cap = torch.cuda.CUDAGraph(), torch.cuda.Stream()
    cap.wait_stream(stream)
    with torch.cuda.stream(cap):
        with torch.cuda.graph(graph, stream=cap):
            for _ in range(args.steps):
                step(cap)
    torch.cuda.synchronize()
    graph.replay()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    graph.replay()
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    tflops = flops / (ms * 1e-3) / 1e12
    t_roof = max(hbm / (PEAK_HBM_GBS * 1e9), flops / (PEAK_BF16_TFLOPS * 1e12)) * 1e3
    print(json.dumps({
        "metric": METRIC, "value": round(tflops, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded N(0,1) blocks, He-initialised weights)",
        "config": {"workload": f"{cfg.name}: one process's local blocks of the {'-'.join(map(str, dims))} FC stack "
                               f"on a {P_r}x{P_c} grid, global B = {cfg.batch} (local {b}), forward + backward "
                               f"partials, unreduced", "global_batch": cfg.batch, "local_batch": b,
                   "parallelism": f"one process of P_r x P_c = {P_r}x{P_c}"},
        "samples_per_s": round(b / (ms * 1e-3), 1),
        "pct_bf16_mfma_peak": round(100.0 * tflops / PEAK_BF16_TFLOPS, 3), "gflop_per_step": round(flops / 1e9, 4),
        "algorithmic_hbm_bytes": hbm, "roofline_ms": round(t_roof, 5), "frac_of_roofline": round(t_roof / ms, 4),
        "launch": "the timed steps replayed from one captured HIP graph",
    }), flush=True)


def bench_copy(args):
    """A plain device-to-device copy of 512 MiB: the calibration run for the HBM byte
    counters (FETCH_SIZE / WRITE_SIZE per dispatch against the known 512 MiB each way)
    and the practical copy bandwidth of the part."""
    import torch
    n = 512 << 20
    a = torch.empty(n, dtype=torch.uint8, device="cuda:0")
    b = torch.empty_like(a)
    a.fill_(1)
    for _ in range(args.warmup):
        b.copy_(a)
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        b.copy_(a)
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    print(json.dumps({"metric": "device copy bandwidth (read + write)", "value": round(2 * n / (ms * 1e-3) / 1e9, 1),
                      "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
                      "ms_per_step": round(ms, 5), "bytes_each_way": n}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    # The first warm-up step is kept for the parity check. The GPU reaches its steady clocks only
    # after some 20 ms of sustained work: with 5 warm-up steps the B = 256 step timed 0.213-0.215
    # ms, with 100 or 400 0.206 ms (the same GPU; the seeded state timed after a warm GPU gives the
    # warm figure too), so the default warm-up covers that time at every workload.
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default="alexnet_fc_b256")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-batch", type=int, default=0, help="samples in the oracle's timed step (0: the whole batch)")
    ap.add_argument("--stack", default="alexnet", choices=("alexnet", "vgg"))
    ap.add_argument("--batches", default="1,2,4,8,16,32,64,128,256,512,1024,2048")
    ap.add_argument("--procs", default="8,64,512")
    ap.add_argument("--grid-batch", type=int, default=2048)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}); the multi-GPU "
              f"1.5D grid is not part of it", file=sys.stderr)
        sys.exit(2)

    if args.workload == "conv3x3_tile":
        return bench_conv(args)
    if args.workload == "hbm_copy":
        return bench_copy(args)
    if args.workload == "batch_sweep":
        return bench_batch_sweep(args)
    if args.workload == "grid_model":
        return bench_grid_model(args)

    import numpy as np
    import torch

    import paper_1712_04432_amd as m
    from synthdata import get_config, make_mlp_inputs

    cfg = get_config(args.workload)
    if tuple(cfg.grid) != (1, 1):
        return bench_local(args, cfg)
    m.load()
    dev = torch.device("cuda:0")
    log(f"bench: workload {cfg.name} dims {cfg.dims} B={cfg.batch} dtype={cfg.dtype}")
    d = make_mlp_inputs(cfg, seed=0)
    net = m.MLP(cfg.dims, cfg.batch, cfg.dtype)
    bf16 = cfg.dtype == "bf16"
    layers = []
    for w, b in zip(d["w"], d["b"]):
        w32 = torch.from_numpy(w).to(dev)
        if bf16:
            wlp = torch.empty(w.shape, dtype=torch.bfloat16, device=dev)
            m.cast_f32_bf16(w32, wlp)
        else:
            wlp = w32  # an fp32 network computes on its masters
        layers.append({"w": w32, "w_lp": wlp, "b": torch.from_numpy(b).to(dev)})
    if bf16:
        x = torch.from_numpy(d["x_bits"].view(np.int16)).to(dev).view(torch.bfloat16)
    else:
        x = torch.from_numpy(d["x"]).to(dev)
    lab = torch.from_numpy(d["labels"]).to(dev)
    ws = torch.zeros(m.mlp_workspace_bytes(net), dtype=torch.uint8, device=dev)
    loss = torch.zeros(1, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        m.mlp_train_step(net, layers, x, lab, ws, cfg.lr, loss, stream=stream)

    # the first warm-up step starts from the seeded state: kept for the comparison with the oracle
    first_dev = None
    if args.warmup >= 1 and not args.no_cpu_baseline:
        step()
        torch.cuda.synchronize()
        first_dev = {"loss": loss.item(), "w": [l["w"].cpu().numpy() for l in layers],
                     "b": [l["b"].cpu().numpy() for l in layers],
                     "acts": [m.ws_view(net, ws, m.IMBD_WS_ACT, i).float().cpu().numpy().astype(np.float64)
                              for i in range(1, cfg.n_layers)]}
    for _ in range(max(args.warmup - 1, 0)):
        step()
    torch.cuda.synchronize()
    loss0 = loss.item()
    log(f"bench: warmup done, loss {loss0:.5f}")

    # timed region: K steps between two synchronisations
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = start.elapsed_time(stop)
    ms_step = ms_total / args.steps
    log(f"bench: {args.steps} steps in {ms_total:.3f} ms (wall {wall * 1e3:.3f} ms), loss {loss.item():.5f}")

    # the same K steps again with HIP events around the dominant kernel (layer-1 fused dW+SGD)
    m.timing_begin(m.IMBD_K_GEMM_DW, 1, args.steps)
    for _ in range(args.steps):
        step()
    n_launch, k_ms = m.timing_end()
    torch.cuda.synchronize()
    k_avg_ms = k_ms / max(n_launch, 1)
    flops = cfg.gemm_flops()
    tflops = flops / (ms_step * 1e-3) / 1e12
    dom_bytes = dw_sgd_bytes(cfg.dims[1], cfg.dims[0], cfg.batch, act_bytes=2 if bf16 else 4)
    peak = PEAK_BF16_TFLOPS if bf16 else PEAK_F32_TFLOPS
    achieved = dom_bytes / (k_avg_ms * 1e-3) / 1e9
    traffic = measured_traffic(cfg.name)
    result = {
        "metric": METRIC,
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32",
        "data": ("synthetic (seeded N(0,1) inputs clamped at 0, uniform labels, He-initialised weights)" if bf16
                 else "synthetic (seeded U(0,1) inputs, uniform labels, He-initialised weights)"),
        "config": {"workload": f"{cfg.name}: {'-'.join(map(str, cfg.dims))} FC stack, ReLU, softmax "
                               f"cross-entropy, " + ("bf16 operands / fp32 accumulation / fp32 masters"
                                                     if bf16 else "fp32") + ", fused SGD",
                   "global_batch": cfg.batch, "layers": cfg.n_layers, "parallelism": "single GPU (P_r = P_c = 1)"},
        "samples_per_s": round(cfg.batch / (ms_step * 1e-3), 1),
        ("pct_bf16_mfma_peak" if bf16 else "pct_fp32_mfma_peak"): round(100.0 * tflops / peak, 3),
        "us_per_step": round(ms_step * 1e3, 2),
        "gflop_per_step": round(flops / 1e9, 4),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4),
                     "traffic": traffic,
                     "kernel": f"layer-1 weight gradient with fused SGD ({cfg.dims[1]}x{cfg.dims[0]} update, "
                               f"K={cfg.batch})",
                     "algorithmic_bytes_per_launch": dom_bytes, "avg_launch_ms": round(k_avg_ms, 5),
                     "launches_timed": n_launch},
        "loss_first": round(loss0, 6),
    }
    if not args.no_cpu_baseline:
        log("bench: timing the CPU oracle on a bounded sample")
        dec = None if first_dev is None else [None] + first_dev["acts"]
        result["cpu_baseline"], ref = cpu_baseline(cfg, args.cpu_sample_batch, relu_decisions=dec)
        if ref is not None and first_dev is not None:
            w0 = [np.asarray(w, np.float64) for w in d["w"]]
            b0 = [np.asarray(b, np.float64) for b in d["b"]]
            result["parity"] = parity_vs_oracle(first_dev, w0, b0, ref)
            log(f"bench: first step against the oracle, max normwise error "
                f"{result['parity']['max_normwise_err']:.2e}")
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
