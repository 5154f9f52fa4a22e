"""Pins for the oracle's optimal placement (the baseline of the paper's
placement-accuracy experiment, Sec. 6.4): the smallest mean drop over every
feasible placement of a set of models onto identical GPUs of bounded
capacity.

The enumeration is checked against closed-form counts of set partitions
and against an independent brute force over every labelled assignment
(each GPU's drops taken from the aggregation, itself pinned elsewhere);
the objective against a hand-worked dyadic example; and the optimum
against invariants (enough GPUs give 0, greedy placement is never better,
more GPUs never hurt).
"""
import itertools
import math

import numpy as np
import pytest

import oracle
from paper_2607_16784_amd import workloads as W


def tiny_problem(seed, N=7):
    rng = np.random.default_rng(seed)
    delay = rng.lognormal(0.0, 1.0, (N, N)) * (rng.random((N, N)) < 0.8)
    iso = rng.lognormal(2.0, 0.5, N)
    q = rng.integers(10, 60, N).astype(np.int32)
    return delay, iso, q


def bell(n):
    return sum(math.comb(n - 1, k) * bell(k) for k in range(n)) if n else 1


def brute_force(delay, iso, q, models, G, C, drop_mode=oracle.DROP_ISO):
    """Every labelled assignment with at most C models per GPU; drops from
    the aggregation of each GPU's members (ascending position)."""
    n = len(models)
    values = {}
    for lab in itertools.product(range(G), repeat=n):
        if max(np.bincount(lab, minlength=G)) > C:
            continue
        mu = np.zeros(n)
        for g in range(G):
            pos = [p for p in range(n) if lab[p] == g]
            if not pos:
                continue
            a = oracle.aggregate(delay, iso, q, [0, len(pos)], [models[p] for p in pos],
                                 drop_mode)
            mu[pos] = a["mu"]
        total = 0.0
        for p in range(n):
            total = total + mu[p]
        key = frozenset(frozenset(p for p in range(n) if lab[p] == g) for g in set(lab))
        values[key] = total / n
    return values


@pytest.mark.parametrize("n", range(1, 9))
def test_unrestricted_placements_are_the_set_partitions(n):
    delay, iso, q = tiny_problem(1, N=8)
    r = oracle.place_optimal(delay, iso, q, list(range(n)), n_devices=n, capacity=n)
    assert r["visited"] == bell(n)


def test_placement_counts_match_closed_forms():
    delay, iso, q = tiny_problem(2, N=8)
    # pairs only, n/2 GPUs: perfect matchings (n - 1)!!
    assert oracle.place_optimal(delay, iso, q, range(6), 3, 2)["visited"] == 15
    assert oracle.place_optimal(delay, iso, q, range(8), 4, 2)["visited"] == 105
    # two GPUs without a capacity bound: S(n,1) + S(n,2) = 2^(n-1)
    for n in (3, 5, 7):
        assert oracle.place_optimal(delay, iso, q, range(n), 2, n)["visited"] == 2 ** (n - 1)


@pytest.mark.parametrize("seed,n,G,C", [(3, 5, 3, 2), (4, 6, 3, 3), (5, 6, 4, 2), (6, 7, 3, 3),
                                        (7, 5, 5, 5), (8, 6, 2, 3)])
@pytest.mark.parametrize("drop_mode", [oracle.DROP_ISO, oracle.DROP_ADJUSTED])
def test_optimum_matches_brute_force_over_labelled_assignments(seed, n, G, C, drop_mode):
    delay, iso, q = tiny_problem(seed)
    rng = np.random.default_rng(seed)
    models = rng.integers(0, len(iso), n)          # replicas allowed
    values = brute_force(delay, iso, q, models, G, C, drop_mode)
    r = oracle.place_optimal(delay, iso, q, models, G, C, drop_mode)
    assert r["visited"] == len(values)
    ordered = sorted(values.values())
    assert r["best_mean"] == ordered[0]
    assert r["second_best"] == (ordered[1] if len(ordered) > 1 else math.inf)
    # the reported placement attains the optimum and respects the capacity
    g = r["best_gpu"]
    assert np.bincount(g).max() <= C and g.max() < G
    key = frozenset(frozenset(np.nonzero(g == b)[0].tolist()) for b in set(g.tolist()))
    assert values[key] == r["best_mean"]
    assert oracle.placement_mean_drop(delay, iso, q, models, g, G, drop_mode) == r["best_mean"]


def test_hand_worked_three_models():
    # equal isolated times (1) and kernel counts (gamma = 1); symmetric delays
    # 0.5 (models 0,1), 0.125 (0,2), 0.25 (1,2).  Two GPUs of two models:
    #   {0,1}{2}: drops 0.5, 0.5, 0     -> mean 1/3
    #   {0,2}{1}: drops 0.125, 0, 0.125 -> mean 0.25/3   (optimum)
    #   {0}{1,2}: drops 0, 0.25, 0.25   -> mean 0.5/3
    D = np.array([[0.0, 0.5, 0.125], [0.5, 0.0, 0.25], [0.125, 0.25, 0.0]])
    iso = np.ones(3)
    q = np.ones(3, np.int32)
    r = oracle.place_optimal(D, iso, q, [0, 1, 2], n_devices=2, capacity=2)
    assert r["visited"] == 3
    assert r["best_mean"] == 0.25 / 3 and r["second_best"] == 0.5 / 3
    assert list(r["best_gpu"]) == [0, 1, 0]
    # one GPU of three: drops 0.625, 0.75, 0.375 -> mean 1.75 / 3
    r = oracle.place_optimal(D, iso, q, [0, 1, 2], n_devices=1, capacity=3)
    assert r["visited"] == 1 and r["best_mean"] == 1.75 / 3
    # drop over the aggregated time: 0.625/1.625, 0.75/1.75, 0.375/1.375
    r = oracle.place_optimal(D, iso, q, [0, 1, 2], 1, 3, oracle.DROP_ADJUSTED)
    assert r["best_mean"] == pytest.approx((0.625 / 1.625 + 0.75 / 1.75 + 0.375 / 1.375) / 3,
                                           rel=1e-15)


def test_optimum_invariants():
    delay, iso, q = tiny_problem(9, N=10)
    models = np.arange(8)
    # enough GPUs: every model alone, no drop at all
    assert oracle.place_optimal(delay, iso, q, models, 8, 3)["best_mean"] == 0.0
    # no interference anywhere: 0
    z = oracle.place_optimal(np.zeros_like(delay), iso, q, models, 3, 3)
    assert z["best_mean"] == 0.0
    # more GPUs never hurt
    vals = [oracle.place_optimal(delay, iso, q, models, G, 4)["best_mean"] for G in (2, 3, 4, 5)]
    assert all(a >= b for a, b in zip(vals, vals[1:]))
    # greedy placement (no deferral) is never better than the optimum
    for G, C in ((3, 3), (4, 2), (2, 4)):
        gr = oracle.place(delay, iso, q, G, C, models, lam=np.inf)
        assert (gr["placed_device"] >= 0).all()
        gval = oracle.placement_mean_drop(delay, iso, q, models, gr["placed_device"], G)
        opt = oracle.place_optimal(delay, iso, q, models, G, C)
        assert opt["best_mean"] <= gval


def test_infeasible_and_invalid_inputs():
    delay, iso, q = tiny_problem(10)
    assert math.isnan(oracle.place_optimal(delay, iso, q, range(7), 2, 3)["best_mean"])
    assert math.isnan(oracle.place_optimal(delay, iso, q, [0, 99], 2, 2)["best_mean"])
    assert oracle.place_optimal(delay, iso, q, [], 2, 2)["best_mean"] == 0.0
