"""The communication cost model and grid selector (paper_1712_04432_amd.gridmodel), pinned
against what the paper states about its own equations: the 1.5D cost reduces to the pure
batch and pure model costs at the ends of the grid range and the integrated model + batch +
domain cost to the 1.5D cost without domain layers (Sec. 2.3, Sec. 2.4); the redistribution
is a third of a model-parallel layer's traffic (Sec. 2.2); the batch/model volume ratio of
the AlexNet 3x3 convolution on 13x13x384 activations crosses 1 between B = 13 and 14 (the
paper says model parallelism wins for B <= 12; its own formula gives B < 13.6, and the
formula is what is pinned); the weight all-reduce volume falls by P_r; and the selector returns
the brute-force minimum."""
import math

import pytest

from paper_1712_04432_amd import gridmodel as gm

ALEXNET_FC = [gm.FC(9216, 4096), gm.FC(4096, 4096), gm.FC(4096, 1000)]
CONV4 = gm.Conv(13, 13, 384, 13, 13, 384, 3, 3)      # AlexNet conv4: 3x3, 384 -> 384 on 13x13
A, BETA = 2e-6, 1.0 / 6e9                             # the paper's simulation parameters


@pytest.mark.parametrize("P", [2, 8, 64, 512])
def test_15d_is_batch_parallel_on_a_1_by_P_grid(P):
    assert gm.t_15d(ALEXNET_FC, 2048, 1, P, A, BETA) == pytest.approx(gm.t_batch(ALEXNET_FC, P, A, BETA), rel=1e-12)


@pytest.mark.parametrize("P", [2, 8, 64, 512])
def test_15d_is_model_parallel_on_a_P_by_1_grid(P):
    assert gm.t_15d(ALEXNET_FC, 2048, P, 1, A, BETA) == pytest.approx(gm.t_model(ALEXNET_FC, 2048, P, A, BETA),
                                                                       rel=1e-12)


@pytest.mark.parametrize("P_r,P_c", [(1, 8), (4, 16), (16, 32), (512, 1)])
def test_integrated_cost_without_domain_layers_is_the_15d_cost(P_r, P_c):
    layers = [CONV4, CONV4] + ALEXNET_FC
    assert gm.t_15d_domain(layers, [], 2048, P_r, P_c, A, BETA) == pytest.approx(
        gm.t_15d(layers, 2048, P_r, P_c, A, BETA), rel=1e-12)


def test_domain_layers_on_one_group_row_cost_like_pure_domain():
    # P_r groups of one process each split nothing but the batch: with P_r = P the domain
    # layers' terms are the pure domain-parallel cost at B / P_c = B
    convs = [CONV4, CONV4]
    P = 16
    assert gm.t_15d_domain(convs, [0, 1], 256, P, 1, A, BETA) == pytest.approx(gm.t_domain(convs, 256, P, A, BETA),
                                                                               rel=1e-12)


def test_redistribution_is_a_third_of_a_model_parallel_layer():
    # a layer with as many inputs as outputs: the model-parallel step moves its output once
    # (all-gather) and its input gradient twice (ring all-reduce)
    sq = [gm.FC(4096, 4096), gm.FC(4096, 4096)]
    P, B = 64, 1024
    per_layer_2 = gm.t_model(sq, B, P, 0.0, BETA) - gm.t_model(sq[:1], B, P, 0.0, BETA)
    assert per_layer_2 == pytest.approx(3 * gm.t_redistribute(sq[1], B, P, 0.0, BETA), rel=1e-12)


def test_model_beats_batch_on_alexnet_conv4_up_to_b13():
    assert gm.volume_ratio_batch_over_model(CONV4, 13) > 1.0 > gm.volume_ratio_batch_over_model(CONV4, 14)
    assert gm.model_beats_batch_below(CONV4) == 13
    # the ratio is that of the two costs' bandwidth terms for one such layer
    one = [CONV4, CONV4]
    vb = gm.t_batch(one[1:], 10**9, 0.0, BETA)
    vm = gm.t_model(one, 13, 10**9, 0.0, BETA) - gm.t_model(one[:1], 13, 10**9, 0.0, BETA)
    assert vb / vm == pytest.approx(gm.volume_ratio_batch_over_model(CONV4, 13), rel=1e-6)


@pytest.mark.parametrize("P_r", [2, 4, 16])
def test_weight_allreduce_volume_falls_by_P_r(P_r):
    P_c = 32
    t_r = gm.t_15d_terms(ALEXNET_FC, 2048, P_r, P_c, 0.0, BETA)["allreduce_dw"]
    t_1 = gm.t_15d_terms(ALEXNET_FC, 2048, 1, P_c, 0.0, BETA)["allreduce_dw"]
    assert t_r == pytest.approx(t_1 / P_r, rel=1e-12)


def test_single_process_needs_no_communication():
    assert gm.t_15d(ALEXNET_FC, 256, 1, 1, A, BETA) == 0.0


def test_latency_terms_count_messages():
    # beta = 0: Bruck / ring latency alpha*ceil(log2 p) per collective, 3 + 2*2 on P_r, 2*3 on P_c
    t = gm.t_15d(ALEXNET_FC, 2048, 8, 64, A, 0.0)
    assert t == pytest.approx(A * (3 * 3 + 2 * 2 * 3 + 2 * 3 * 6), rel=1e-12)


@pytest.mark.parametrize("P", [8, 12, 64, 512])
def test_selector_returns_the_brute_force_minimum(P):
    def comp(pr, pc):                       # any positive compute model
        return 1e-3 * (1.0 + 0.1 * pr) / pc + 2e-4 * math.log2(pr + 1)
    best, rows = gm.select_grid(ALEXNET_FC, 2048, P, A, BETA, t_comp=comp, divisible=False)
    brute = min(((gm.t_15d(ALEXNET_FC, 2048, r, P // r, A, BETA) + comp(r, P // r), r)
                 for r in range(1, P + 1) if P % r == 0))
    assert best == (brute[1], P // brute[1])
    assert len(rows) == sum(1 for r in range(1, P + 1) if P % r == 0)


def test_selector_respects_even_blocks():
    best, rows = gm.select_grid(ALEXNET_FC, 96, 64, A, BETA)
    assert all(96 % r["P_c"] == 0 and all(l.d % r["P_r"] == 0 for l in ALEXNET_FC) for r in rows)
    with pytest.raises(ValueError):
        gm.select_grid([gm.FC(7, 7)], 7, 4, A, BETA)


def test_paper_trend_fc_layers_prefer_model_split_at_scale():
    # communication only, the paper's Cori parameters, B = 2048: at P = 512 a pure batch
    # grid is not the cheapest for the AlexNet FC layers (the weight all-reduce dominates)
    best, rows = gm.select_grid(ALEXNET_FC, 2048, 512, A, BETA)
    assert best[0] > 1
    pure = [r for r in rows if r["P_r"] == 1][0]
    assert min(r["comm"] for r in rows) < pure["comm"]
