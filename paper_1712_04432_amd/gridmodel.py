"""Communication cost model of the paper's parallel layouts and the process-grid selector.

Host-side planning tool (no GPU code): the alpha-beta costs of Sec. 2.2 (pure model, pure
batch and pure domain parallelism, and the batch-to-model redistribution), of Sec. 2.3
(the integrated 1.5D model + batch layout on a P_r x P_c grid) and of Sec. 2.4 (model or
domain partitioning per layer on the P_r groups), and a selector that picks the grid with
the least modelled time per iteration: communication from these costs plus the compute
time of one process's local blocks, which a caller supplies (for the FC layers, timed on
the device by ``bench.py --workload grid_model``).

Conventions and readings of the paper:
* ``alpha`` is the latency of one message (s), ``beta`` the inverse bandwidth (s/byte);
  volumes are element counts times ``elem_bytes``.
* All-gather uses Bruck's algorithm and all-reduce the ring algorithm (Sec. 2.2): a
  collective over p processes costs alpha*ceil(log2 p) plus the per-process volume times
  (p-1)/p; the all-reduce is charged twice (reduce-scatter + all-gather).
* Layers are numbered 1..L; the paper's all-reduce sums written from i = 0 run over the
  same L layers (there is no layer 0 with weights).
* Collectives over a single process cost nothing (ceil(log2 1) = 0 and (p-1)/p = 0).
* d_i is the number of output activations of layer i per sample (Y_H*Y_W*Y_C for a
  convolution) and |W_i| its parameter count.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Callable, Iterable, Sequence


@dataclass(frozen=True)
class FC:
    """Fully connected layer: d_in inputs, d_out outputs per sample."""
    d_in: int
    d_out: int

    @property
    def d(self) -> int:
        return self.d_out

    @property
    def d_prev(self) -> int:
        return self.d_in

    @property
    def weights(self) -> int:
        return self.d_in * self.d_out


@dataclass(frozen=True)
class Conv:
    """Convolution with a k_h x k_w filter bank (Sec. 2.1): input X_H x X_W x X_C, output
    Y_H x Y_W x Y_C, |W| = k_h k_w X_C Y_C."""
    x_h: int
    x_w: int
    x_c: int
    y_h: int
    y_w: int
    y_c: int
    k_h: int
    k_w: int

    @property
    def d(self) -> int:
        return self.y_h * self.y_w * self.y_c

    @property
    def d_prev(self) -> int:
        return self.x_h * self.x_w * self.x_c

    @property
    def weights(self) -> int:
        return self.k_h * self.k_w * self.x_c * self.y_c


def _lat(alpha: float, p: int) -> float:
    """Latency of a collective over p processes: alpha * ceil(log2 p)."""
    return alpha * math.ceil(math.log2(p)) if p > 1 else 0.0


def _share(p: int) -> float:
    """(p - 1) / p, the fraction of the data a process receives in a collective."""
    return (p - 1) / p


# ----------------------------------------------------------------- Sec. 2.2: pure layouts
def t_model(layers: Sequence, B: int, P: int, alpha: float, beta: float, elem_bytes: int = 4) -> float:
    """Pure model parallelism (Sec. 2.2): an all-gather of every layer's output activations
    (B d_i values) after the layer, and an all-reduce of the activation gradient
    (B d_{i-1} values) for layers 2..L in the backward pass."""
    bb = beta * elem_bytes
    t = sum(_lat(alpha, P) + bb * B * _share(P) * l.d for l in layers)
    t += 2 * sum(_lat(alpha, P) + bb * B * _share(P) * l.d_prev for l in layers[1:])
    return t


def t_batch(layers: Sequence, P: int, alpha: float, beta: float, elem_bytes: int = 4) -> float:
    """Pure batch parallelism (Sec. 2.2, the batch-parallel cost equation): a ring all-reduce
    of every layer's weight gradient (|W_i| values)."""
    bb = beta * elem_bytes
    return 2 * sum(_lat(alpha, P) + bb * _share(P) * l.weights for l in layers)


def t_redistribute(layer, B: int, P: int, alpha: float, beta: float, elem_bytes: int = 4) -> float:
    """Switching one layer from the batch to the model layout (Sec. 2.2): one all-gather of
    its B d_i activations."""
    return _lat(alpha, P) + beta * elem_bytes * B * _share(P) * layer.d


def volume_ratio_batch_over_model(conv: Conv, B: int) -> float:
    """Sec. 2.2: communication volume of pure batch over pure model parallelism for one
    convolution, 2|W| / (3 B d) = 2 k_h k_w X_C / (3 B Y_H Y_W); above 1 model parallelism
    moves less data."""
    return 2.0 * conv.weights / (3.0 * B * conv.d)


def model_beats_batch_below(conv: Conv) -> int:
    """Largest batch for which pure model parallelism moves less data than pure batch
    parallelism on this convolution (the volume ratio above 1)."""
    b_star = 2.0 * conv.k_h * conv.k_w * conv.x_c / (3.0 * conv.y_h * conv.y_w)
    return math.ceil(b_star) - 1 if float(b_star).is_integer() else math.floor(b_star)


def t_domain(layers: Sequence[Conv], B: int, P: int, alpha: float, beta: float, elem_bytes: int = 4) -> float:
    """Pure domain parallelism (Sec. 2.2, the domain-parallel cost equation): per layer a
    halo exchange of the input rows in the forward pass (B X_W X_C floor(k_h/2) values) and
    of the output-gradient rows in the backward pass (B Y_W Y_C floor(k_w/2)), each one
    pairwise message, plus the ring all-reduce of the weight gradient."""
    bb = beta * elem_bytes
    t = sum(alpha + bb * B * l.x_w * l.x_c * (l.k_h // 2) for l in layers)
    t += sum(alpha + bb * B * l.y_w * l.y_c * (l.k_w // 2) for l in layers)
    t += 2 * sum(_lat(alpha, P) + bb * _share(P) * l.weights for l in layers)
    return t


# ------------------------------------------------------------ Sec. 2.3: the 1.5D layout
def t_15d_terms(layers: Sequence, B: int, P_r: int, P_c: int, alpha: float, beta: float,
                elem_bytes: int = 4) -> dict:
    """The three sums of the integrated model + batch cost (Sec. 2.3), on a P_r x P_c grid:
    all-gather of the (d_i x B/P_c) outputs over P_r, all-reduce of the activation-gradient
    partials over P_r (layers 2..L), all-reduce of the weight-gradient partials of the
    process's 1/P_r share of |W_i| over P_c."""
    bb = beta * elem_bytes
    bl = B / P_c
    gather = sum(_lat(alpha, P_r) + bb * bl * _share(P_r) * l.d for l in layers)
    dx = 2 * sum(_lat(alpha, P_r) + bb * bl * _share(P_r) * l.d_prev for l in layers[1:])
    dw = 2 * sum(_lat(alpha, P_c) + bb * _share(P_c) * l.weights / P_r for l in layers)
    return {"allgather_y": gather, "allreduce_dx": dx, "allreduce_dw": dw}


def t_15d(layers: Sequence, B: int, P_r: int, P_c: int, alpha: float, beta: float, elem_bytes: int = 4) -> float:
    return sum(t_15d_terms(layers, B, P_r, P_c, alpha, beta, elem_bytes).values())


# ---------------------------------------------- Sec. 2.4: model or domain per layer
def t_15d_domain(layers: Sequence, domain: Iterable[int], B: int, P_r: int, P_c: int, alpha: float,
                 beta: float, elem_bytes: int = 4) -> float:
    """Integrated model, batch and domain parallelism (Sec. 2.4): the layers whose indices
    (0-based) are in ``domain`` split their activations' domain over the P_r groups (halo
    exchange of the B/P_c local samples' rows, all-reduce of the whole weight gradient over
    all P processes); the others split their model over P_r as in the 1.5D layout. The
    backward halo of a domain layer carries the next layer's input rows (its own output)."""
    dom = set(domain)
    P = P_r * P_c
    bb = beta * elem_bytes
    bl = B / P_c
    lm = [l for i, l in enumerate(layers) if i not in dom]
    t = 0.0
    t += sum(_lat(alpha, P_r) + bb * bl * _share(P_r) * l.d for l in lm)
    # activation-gradient all-reduce for model layers past the first layer of the network
    t += 2 * sum(_lat(alpha, P_r) + bb * bl * _share(P_r) * l.d_prev
                 for i, l in enumerate(layers) if i not in dom and i >= 1)
    t += 2 * sum(_lat(alpha, P_c) + bb * _share(P_c) * l.weights / P_r for l in lm)
    for i in sorted(dom):
        l = layers[i]
        t += alpha + bb * bl * l.x_w * l.x_c * (l.k_h // 2)
        t += alpha + bb * bl * l.y_w * l.y_c * (l.k_w // 2)
        t += 2 * (_lat(alpha, P) + bb * _share(P) * l.weights)
    return t


# ------------------------------------------------------------------- grid selection
def grids(P: int):
    """Every P_r x P_c factorisation of P, P_r ascending."""
    return [(r, P // r) for r in range(1, P + 1) if P % r == 0]


def select_grid(layers: Sequence, B: int, P: int, alpha: float, beta: float, elem_bytes: int = 4,
                t_comp: Callable[[int, int], float] | None = None, divisible: bool = True):
    """The grid with the least modelled time per iteration, T_comm (Sec. 2.3) + T_comp.

    t_comp(P_r, P_c): compute time of one process's local blocks (None: communication only).
    divisible: only grids with P_c | B and P_r | d_i for every layer (even blocks, as the
    paper's layouts assume). Returns (best (P_r, P_c), rows), rows being one dict per grid
    with the terms, sorted by P_r."""
    rows = []
    for P_r, P_c in grids(P):
        if divisible and (B % P_c or any(l.d % P_r for l in layers)):
            continue
        terms = t_15d_terms(layers, B, P_r, P_c, alpha, beta, elem_bytes)
        comm = sum(terms.values())
        comp = t_comp(P_r, P_c) if t_comp else 0.0
        rows.append({"P_r": P_r, "P_c": P_c, **terms, "comm": comm, "comp": comp, "total": comm + comp})
    if not rows:
        raise ValueError(f"no admissible {P}-process grid for B = {B}")
    best = min(rows, key=lambda r: (r["total"], r["P_r"]))
    return (best["P_r"], best["P_c"]), rows
