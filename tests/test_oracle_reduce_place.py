"""Pins for the oracle's reduction over the alignment set and aggregation
(Alg. 1, Sec. 3.3) and placement (Alg. 2, Sec. 3.4)."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2607_16784_amd.workloads import A100

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def test_median_conventions():
    assert oracle.median([]) == 0.0
    assert oracle.median([7.0]) == 7.0
    assert oracle.median([3.0, 1.0, 2.0]) == 2.0
    assert oracle.median([4.0, 1.0, 3.0, 2.0]) == 2.5
    assert oracle.median([1.0, 1.0, 5.0, 100.0]) == 3.0
    rng = np.random.default_rng(0)
    for n in range(1, 40):
        v = rng.lognormal(size=n)
        assert oracle.median(v) == float(np.median(v))


def test_alignment_space_size_matches_paper():
    g = _gold("alignment_scenarios.json")
    n, q = g["n_models"], g["kernels_per_model"]
    # kernels that conflict with each other whatever the pair
    lib = dict(offsets=np.arange(0, n * q + 1, q, dtype=np.int64),
               grid=np.full(n * q, 1000, np.int32), threads=np.full(n * q, 1024, np.int32),
               regs=np.full(n * q, 32, np.int32), smem=np.zeros(n * q, np.int32),
               duration=np.ones(n * q))
    assert oracle.alignment_count(A100, lib, unordered=True) == g["pairwise_alignment_scenarios"]
    assert oracle.alignment_count(A100, lib, unordered=False) == n * n * q * q


def _frac(nd):
    return float(Fraction(nd[0], nd[1]))


def test_aggregation_worked_example():
    g = _gold("worked_examples.json")["aggregation_three_models"]
    offs = np.concatenate([[0], np.cumsum([len(s) for s in g["sets"]])])
    members = np.concatenate(g["sets"])
    out = oracle.aggregate(g["delay"], g["iso_time"], g["kernel_count"], offs, members)
    want_mu = [_frac(x) for s in g["mu_num_den"] for x in s]
    assert out["mu"] == pytest.approx(want_mu, rel=1e-15, abs=0)
    assert out["mu_mean"] == pytest.approx([_frac(x) for x in g["mu_mean_num_den"]], rel=1e-15)
    assert out["status"] == 0


def test_aggregation_rejects_bad_ids():
    out = oracle.aggregate(np.zeros((2, 2)), [1.0, 1.0], [1, 1], [0, 2, 3], [0, 5, 1])
    assert np.isnan(out["mu_mean"][0]) and out["mu_mean"][1] == 0.0
    assert out["status"] & oracle.ST_BAD_MODEL_ID


def test_placement_worked_example():
    g = _gold("worked_examples.json")["placement_two_models"]
    out = oracle.place(g["delay"], g["iso_time"], g["kernel_count"], g["n_devices"],
                       g["capacity"], g["events"], g["lambda"])
    assert list(out["placed_device"]) == g["placed_device"]
    assert list(out["placed_mu_mean"]) == g["placed_mu_mean"]
    assert out["resident"].tolist() == [[0, 0], [1, 1]]


def _two_model():
    g = _gold("worked_examples.json")["placement_two_models"]
    return np.array(g["delay"]), np.array(g["iso_time"]), np.array(g["kernel_count"])


def test_zero_bound_defers_everything():
    D, T, q = _two_model()
    out = oracle.place(D, T, q, 3, 2, [0, 1, 1, 0], 0.0)
    assert list(out["placed_device"]) == [-1] * 4
    assert list(out["placed_mu_mean"]) == [0.0] * 4    # an empty GPU gives 0, not < 0


def test_full_cluster_defers_with_infinite_mean():
    D, T, q = _two_model()
    out = oracle.place(D, T, q, 1, 1, [0, 1], 0.5)
    assert list(out["placed_device"]) == [0, -1]
    assert out["placed_mu_mean"][1] == np.inf


def test_mean_equal_to_bound_is_not_eligible():
    D, T, q = _two_model()
    # {0,0} on one device has mean exactly 1/4.
    assert list(oracle.place(D, T, q, 1, 2, [0, 0], 0.25)["placed_device"]) == [0, -1]
    assert list(oracle.place(D, T, q, 1, 2, [0, 0], np.nextafter(0.25, 1))["placed_device"]) == [0, 0]


def test_departures_free_capacity():
    D, T, q = _two_model()
    # e0 -> dev0, e1 -> dev1, e2 = departure of e0, e3: dev0 empty (0) beats
    # dev1 {1,1} (1/8).  e4 departs the deferred-or-missing arrival e2? no: e2
    # is a departure -> bad event.  e5 departs e0 again -> no-op.
    ev = [0, 1, -1 - 0, 1, -1 - 2, -1 - 0]
    out = oracle.place(D, T, q, 2, 2, ev, 0.5)
    assert list(out["placed_device"]) == [0, 1, 0, 0, -1, -1]
    assert out["status"] & oracle.ST_BAD_EVENT
    assert out["resident"].tolist() == [[1, -1], [1, -1]]
    assert list(out["resident_count"]) == [1, 1]


def test_initial_residents_are_respected():
    D, T, q = _two_model()
    out = oracle.place(D, T, q, 2, 2, [1], 0.5, resident=[0, 0, 1, -1], resident_count=[2, 1])
    assert list(out["placed_device"]) == [1]
    assert out["placed_mu_mean"][0] == 0.125


def test_placement_is_argmin_over_eligible_devices():
    # Property check on random instances: every placement is the lowest-index
    # device among those with room whose mean drop is minimal, and below the
    # bound; a deferral means no device with room was below the bound.
    rng = np.random.default_rng(21)
    N, G, C = 7, 4, 3
    D = rng.uniform(0, 4, (N, N))
    T = rng.uniform(5, 20, N)
    q = rng.integers(1, 30, N).astype(np.int32)
    ev = rng.integers(0, N, 60).astype(np.int32)
    out = oracle.place(D, T, q, G, C, ev, 0.6)
    res = [[] for _ in range(G)]
    for e, m in enumerate(ev):
        means = []
        for g in range(G):
            if len(res[g]) >= C:
                means.append(np.inf)
                continue
            s = res[g] + [int(m)]
            mus = []
            for p, mp in enumerate(s):
                t = Fraction(T[mp])
                for r, mr in enumerate(s):
                    if r != p:
                        t += Fraction(max(Fraction(int(q[mp]), int(q[mr])), 1)) * Fraction(D[mp, mr])
                mus.append((t - Fraction(T[mp])) / Fraction(T[mp]))
            means.append(float(sum(mus) / len(mus)))
        best = min(means)
        got = out["placed_device"][e]
        if got >= 0:
            assert means[got] == pytest.approx(best, rel=1e-12) and best < 0.6
            assert all(means[g] > best * (1 + 1e-12) for g in range(got))
            res[got].append(int(m))
        else:
            assert not best < 0.6 * (1 - 1e-12)
