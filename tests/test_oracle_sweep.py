"""Pins for the oracle's pair sweep (Alg. 1 simulation, Sec. 3.2 timeline).

Each check compares the oracle with something it does not share code with:
an all-pairs interval intersection, a unit-time-step simulation, a worked
example derived by hand, or an algebraic identity of the method.
"""
from fractions import Fraction

import numpy as np
import pytest

import brute
import oracle
from paper_2607_16784_amd.workloads import A100, EDGE

# kernel that conflicts with any copy of itself: 32 warps x 2 blocks fill W=64
BIG = (1000, 1024, 32, 0)
# kernel too small to conflict with anything alike: 1 block of 2 warps
TINY = (1, 64, 16, 0)


def lib_from(models):
    """models: list of lists of (grid, threads, regs, smem, duration)."""
    rows = [k for m in models for k in m]
    off = np.zeros(len(models) + 1, np.int64)
    off[1:] = np.cumsum([len(m) for m in models])
    col = lambda i, dt: np.array([r[i] for r in rows], dt)  # noqa: E731
    return dict(offsets=off, grid=col(0, np.int32), threads=col(1, np.int32),
                regs=col(2, np.int32), smem=col(3, np.int32), duration=col(4, np.float64))


def random_lib(rng, n_models, qmax, integer=False, kinds=None):
    models = []
    for _ in range(n_models):
        q = int(rng.integers(1, qmax + 1))
        ks = []
        for _ in range(q):
            g = int(rng.integers(1, 600))
            t = int(rng.choice([64, 128, 256, 512, 1024]))
            r = int(rng.integers(16, 64))
            s = int(rng.integers(0, 90_000))
            d = float(rng.integers(1, 9)) if integer else float(rng.lognormal(1.0, 1.0))
            ks.append((g, t, r, s, d))
        models.append(ks)
    return lib_from(models)


def test_worked_example_two_and_four_kernels():
    # A: two kernels of 2 us; B: four kernels of 1 us; every pair conflicts and
    # all have the same active warps, so each conflict is shared 1/2 : 1/2.
    # Temporal sweep from the first kernels: four 1-us stretches, all in
    # conflict -> Delta_AB = Delta_BA = 4 * 1/2 = 2.  gamma_AB = max(2/4,1) = 1,
    # gamma_BA = max(4/2,1) = 2; mu_A = 1*2/4 = 0.5, mu_B = 2*2/4 = 1.0.
    L = lib_from([[BIG + (2.0,)] * 2, [BIG + (1.0,)] * 4])
    out = oracle.pair_matrix(A100, L)
    assert out["delay"][0, 1] == 2.0 and out["delay"][1, 0] == 2.0
    assert out["slowdown"][0, 1] == 0.5 and out["slowdown"][1, 0] == 1.0
    agg = oracle.aggregate(out["delay"], out["iso_time"], out["kernel_count"], [0, 2], [0, 1])
    assert list(agg["mu"]) == [0.5, 1.0] and agg["mu_mean"][0] == 0.75
    # Dividing by the aggregated time (the drop step of Alg. 1): T~_A = 4 + 2 = 6.
    agg1 = oracle.aggregate(out["delay"], out["iso_time"], out["kernel_count"], [0, 2], [0, 1],
                            drop_mode=oracle.DROP_ADJUSTED)
    assert agg1["mu"][0] == 2.0 / 6.0
    # Literal lockstep walk: B's first two kernels meet A's two -> 1 + ... = 1.
    lk = oracle.pair_matrix(A100, L, sweep_mode=oracle.SWEEP_LOCKSTEP)
    assert lk["delay"][1, 0] == 1.0 and lk["delay"][0, 1] == 2.0
    assert lk["slowdown"][1, 0] == 0.5


@pytest.mark.parametrize("seed", range(6))
def test_every_start_pair_matches_all_pairs_intersection(seed):
    rng = np.random.default_rng(seed)
    L = random_lib(rng, 2, 7)
    ms = [brute.Model(A100, L, m) for m in range(2)]
    for i in range(2):
        for j in range(2):
            for si in range(ms[i].q):
                for sj in range(ms[j].q):
                    want = brute.delay_all_pairs(A100, ms[i], ms[j], si, sj)
                    got = oracle.sweep_start_pair(A100, L, i, j, si, sj)
                    assert got == pytest.approx(want, rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_integer_durations_exact_against_unit_steps(seed):
    rng = np.random.default_rng(100 + seed)
    L = random_lib(rng, 3, 9, integer=True)
    ms = [brute.Model(A100, L, m) for m in range(3)]
    for i in range(3):
        for j in range(3):
            for si in range(0, ms[i].q, 2):
                for sj in range(0, ms[j].q, 3):
                    want = brute.delay_unit_steps(A100, ms[i], ms[j], si, sj)
                    exact = brute.delay_all_pairs(A100, ms[i], ms[j], si, sj, exact=True)
                    assert want == exact
                    got = oracle.sweep_start_pair(A100, L, i, j, si, sj)
                    assert got == pytest.approx(float(want), rel=1e-15, abs=0)


@pytest.mark.parametrize("seed", range(3))
def test_offsets_match_all_pairs_intersection(seed):
    rng = np.random.default_rng(200 + seed)
    L = random_lib(rng, 3, 8)
    ms = [brute.Model(EDGE, L, m) for m in range(3)]
    K = 5
    out = oracle.pair_matrix(EDGE, L, align_mode=oracle.ALIGN_OFFSETS,
                             reduce_mode=oracle.REDUCE_MAX, num_offsets=K, per_alignment=True)
    for i in range(3):
        Ti = out["iso_time"][i]
        for j in range(3):
            want = [brute.delay_all_pairs(EDGE, ms[i], ms[j], offset=Ti * r / K) for r in range(K)]
            assert out["per_alignment"][i, j] == pytest.approx(want, rel=1e-12, abs=1e-12)
            assert out["delay"][i, j] == pytest.approx(max(want), rel=1e-12, abs=1e-12)


def test_first_alignment_and_median_of_conflicting_starts():
    rng = np.random.default_rng(3)
    L = random_lib(rng, 2, 6)
    ms = [brute.Model(A100, L, m) for m in range(2)]
    first = oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_FIRST)
    starts = oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_CONFLICT_STARTS,
                                per_alignment=True)
    off = L["offsets"]
    for i in range(2):
        for j in range(2):
            assert first["delay"][i, j] == pytest.approx(
                brute.delay_all_pairs(A100, ms[i], ms[j]), rel=1e-12, abs=1e-12)
            vals = []
            for si in range(ms[i].q):
                for sj in range(ms[j].q):
                    pa = starts["per_alignment"][off[i] + si, off[j] + sj]
                    if brute.fits_together(A100, ms[i].fp[si], ms[j].fp[sj]):
                        assert np.isnan(pa)
                    else:
                        vals.append(brute.delay_all_pairs(A100, ms[i], ms[j], si, sj))
                        assert pa == pytest.approx(vals[-1], rel=1e-12, abs=1e-12)
            want = float(np.median(vals)) if vals else 0.0
            assert starts["delay"][i, j] == pytest.approx(want, rel=1e-12, abs=1e-12)


def test_lockstep_equals_temporal_for_matching_integer_durations():
    # When the walked kernels pair one-to-one with equal integer durations the
    # timeline walk and the literal lockstep walk add exactly the same terms.
    rng = np.random.default_rng(9)
    d = [float(x) for x in rng.integers(1, 20, 12)]
    ka = [(int(rng.integers(1, 900)), int(rng.choice([128, 256, 1024])), 32,
           int(rng.integers(0, 90000)), x) for x in d]
    kb = [(int(rng.integers(1, 900)), int(rng.choice([64, 512])), 40,
           int(rng.integers(0, 90000)), x) for x in d]
    L = lib_from([ka, kb])
    t = oracle.pair_matrix(A100, L)
    s = oracle.pair_matrix(A100, L, sweep_mode=oracle.SWEEP_LOCKSTEP)
    assert np.array_equal(t["delay"], s["delay"])
    assert t["delay"].max() > 0


def test_self_pair_is_half_the_self_conflicting_time():
    rng = np.random.default_rng(4)
    L = random_lib(rng, 1, 40, integer=True)
    m = brute.Model(A100, L, 0)
    out = oracle.pair_matrix(A100, L)
    want = sum(Fraction(int(m.d[k]), 2) for k in range(m.q)
               if not brute.fits_together(A100, m.fp[k], m.fp[k]))
    assert out["delay"][0, 0] == float(want)


def test_tiny_kernels_never_interfere():
    L = lib_from([[TINY + (3.0,)] * 5, [TINY + (1.5,)] * 7])
    for mode in (oracle.ALIGN_FIRST, oracle.ALIGN_CONFLICT_STARTS):
        out = oracle.pair_matrix(A100, L, align_mode=mode)
        assert np.all(out["delay"] == 0.0) and np.all(out["slowdown"] == 0.0)
    out = oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_OFFSETS, num_offsets=8,
                             reduce_mode=oracle.REDUCE_MAX)
    assert np.all(out["delay"] == 0.0)


def test_both_directions_split_the_conflicting_time():
    rng = np.random.default_rng(12)
    L = random_lib(rng, 4, 15)
    ms = [brute.Model(A100, L, m) for m in range(4)]
    out = oracle.pair_matrix(A100, L)
    for i in range(4):
        for j in range(4):
            total = brute.delay_all_pairs(A100, ms[i], ms[j], weight=False)
            assert out["delay"][i, j] + out["delay"][j, i] == pytest.approx(total, rel=1e-12)


def test_power_of_two_time_scaling_is_exact():
    rng = np.random.default_rng(13)
    L = random_lib(rng, 5, 20)
    L4 = dict(L, duration=L["duration"] * 4.0)
    for mode, red, K in ((0, 0, 1), (2, 1, 6)):
        a = oracle.pair_matrix(A100, L, align_mode=mode, reduce_mode=red, num_offsets=K)
        b = oracle.pair_matrix(A100, L4, align_mode=mode, reduce_mode=red, num_offsets=K)
        assert np.array_equal(b["delay"], 4.0 * a["delay"])
        assert np.array_equal(b["slowdown"], a["slowdown"])


def test_permuting_models_permutes_the_matrix():
    rng = np.random.default_rng(14)
    L = random_lib(rng, 6, 12)
    perm = rng.permutation(6)
    off = L["offsets"]
    idx = np.concatenate([np.arange(off[m], off[m + 1]) for m in perm])
    Lp = {k: L[k][idx] for k in ("grid", "threads", "regs", "smem", "duration")}
    Lp["offsets"] = np.concatenate([[0], np.cumsum([off[m + 1] - off[m] for m in perm])])
    a = oracle.pair_matrix(A100, L)
    b = oracle.pair_matrix(A100, Lp)
    assert np.array_equal(b["delay"], a["delay"][np.ix_(perm, perm)])
    assert np.array_equal(b["slowdown"], a["slowdown"][np.ix_(perm, perm)])


def test_entries_equal_matrix():
    rng = np.random.default_rng(15)
    L = random_lib(rng, 5, 25)
    full = oracle.pair_matrix(EDGE, L, align_mode=2, reduce_mode=1, num_offsets=7)
    pairs = np.array([(i, j) for i in range(5) for j in range(5)], np.int32)
    ent = oracle.pair_entries(EDGE, L, pairs, align_mode=2, reduce_mode=1, num_offsets=7)
    assert np.array_equal(ent["delay"], full["delay"].reshape(-1))
    assert np.array_equal(ent["slowdown"], full["slowdown"].reshape(-1))


def test_empty_model_and_bad_durations_flagged():
    L = lib_from([[BIG + (2.0,)] * 3, [], [BIG + (0.0,)] * 2])
    out = oracle.pair_matrix(A100, L)
    assert out["status"] & oracle.ST_EMPTY_MODEL
    assert out["status"] & oracle.ST_BAD_DURATION
    assert out["kernel_count"][1] == 0 and out["iso_time"][1] == 0.0
    assert np.all(out["delay"][1, :] == 0) and np.all(out["delay"][:, 1] == 0)
    assert np.all(out["slowdown"][1, :] == 0)


@pytest.mark.parametrize("align,red,K,mode", [(0, 0, 1, 0), (1, 0, 1, 0), (2, 1, 5, 0),
                                              (3, 0, 6, 0), (0, 0, 1, 2), (2, 1, 3, 2)])
def test_threaded_matrix_equals_single_thread(align, red, K, mode):
    # the all-core timing leg shares the rows out over threads; every pair is
    # still the same scalar computation, so the matrices agree bit for bit
    rng = np.random.default_rng(21)
    L = random_lib(rng, 7, 18)
    dr = None
    if align == 3:
        dr = rng.integers(0, 2**64, size=(7 * 8 // 2, K), dtype=np.uint64)
    kw = dict(align_mode=align, reduce_mode=red, num_offsets=K, sweep_mode=mode,
              per_alignment=True, start_draws=dr)
    one = oracle.pair_matrix(A100, L, **kw)
    for t in (2, 3, 7, 16):
        many = oracle.pair_matrix(A100, L, threads=t, **kw)
        for k in ("delay", "slowdown", "per_alignment", "iso_time", "kernel_count"):
            assert np.array_equal(one[k], many[k], equal_nan=k == "per_alignment"), (t, k)
        assert one["status"] == many["status"]
