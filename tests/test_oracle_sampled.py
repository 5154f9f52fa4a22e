"""Pins for the oracle's sampled start pairs (the pairwise heuristic evaluates
a sample of each model pair's start indices, Sec. 1 and Sec. 3.3 "Pairwise
interference").

A draw is a 64-bit word per sample and unordered pair; its upper half names
the start kernel of the lower-numbered model, its lower half that of the
other model, each by the multiply-shift reduction floor(w * q / 2^32).  The
tests build draws from the inverse of that reduction, w = ceil(s * 2^32 / q),
which names start kernel s (and w - 1 names s - 1), and check the oracle's
per-draw delays against the all-pairs interval intersection of tests/brute.py,
its matrices against the fully enumerated CONFLICT_STARTS set, and the
multiset and transposition rules of the alignment set.
"""
import math

import numpy as np
import pytest

import brute
import oracle
from paper_2607_16784_amd.workloads import A100, EDGE, MI355X, start_draws
from test_oracle_sweep import BIG, TINY, lib_from, random_lib

TWO32 = 1 << 32
MID = (1, 1024, 32, 0)


def word_for(s, q):
    """A 32-bit word that the multiply-shift reduction maps to s in [0, q)."""
    return -(-s * TWO32 // q)


def draw_for(a, qa, b, qb):
    """Draw naming start kernel a of the lower-numbered model (q = qa) and b
    of the higher-numbered one (q = qb)."""
    return (word_for(a, qa) << 32) | word_for(b, qb)


def pair_index(N, i, j):
    a, b = min(i, j), max(i, j)
    return a * N - a * (a - 1) // 2 + (b - a)


def q_of(L, m):
    return int(L["offsets"][m + 1] - L["offsets"][m])


def models(dev, L):
    return [brute.Model(dev, L, m) for m in range(len(L["offsets"]) - 1)]


def conflicts(dev, M, i, j, si, sj):
    return not brute.fits_together(dev, M[i].fp[si], M[j].fp[sj])


def test_inverse_words_name_their_start_kernel():
    for q in (1, 2, 3, 7, 60, 1000, 2000, 4095, 65535):
        for s in {0, 1, q // 2, q - 1} & set(range(q)):
            w = word_for(s, q)
            assert 0 <= w < TWO32
            assert (w * q) >> 32 == s
            if s > 0:
                assert ((w - 1) * q) >> 32 == s - 1


def test_each_draw_matches_the_all_pairs_intersection():
    rng = np.random.default_rng(11)
    L = random_lib(rng, 3, 9)
    N = 3
    M = models(A100, L)
    K = 12
    pairs = N * (N + 1) // 2
    draws = np.zeros((pairs, K), np.uint64)
    want = {}
    for i in range(N):
        for j in range(i, N):
            for r in range(K):
                a = int(rng.integers(0, q_of(L, i)))
                b = int(rng.integers(0, q_of(L, j)))
                draws[pair_index(N, i, j), r] = draw_for(a, q_of(L, i), b, q_of(L, j))
                want[(i, j, r)] = (a, b)
                if i != j:
                    want[(j, i, r)] = (b, a)
    out = oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_SAMPLED_STARTS, num_offsets=K,
                             start_draws=draws, per_alignment=True)
    pa = out["per_alignment"]
    for (i, j, r), (si, sj) in want.items():
        got = pa[i, j, r]
        if not conflicts(A100, M, i, j, si, sj):
            assert np.isnan(got), (i, j, r)
            continue
        ref = brute.delay_all_pairs(A100, M[i], M[j], si, sj)
        assert got == pytest.approx(ref, rel=1e-12, abs=0.0), (i, j, r)
    # the delay is the median of the members, an empty set gives 0
    for i in range(N):
        for j in range(N):
            v = pa[i, j][~np.isnan(pa[i, j])]
            assert out["delay"][i, j] == (np.median(v) if v.size else 0.0)


def test_enumerating_draws_reproduce_conflict_starts():
    # every model has q kernels, so K = q^2 draws can name every start pair of
    # every unordered pair exactly once; C_ij is then the CONFLICT_STARTS set
    rng = np.random.default_rng(5)
    q = 6
    mods = []
    for _ in range(3):
        mods.append([(int(rng.integers(1, 600)), int(rng.choice([128, 256, 512, 1024])),
                      int(rng.integers(16, 64)), int(rng.integers(0, 90_000)),
                      float(rng.lognormal(1.0, 1.0))) for _ in range(q)])
    L = lib_from(mods)
    N = 3
    K = q * q
    one = np.array([draw_for(a, q, b, q) for a in range(q) for b in range(q)], np.uint64)
    draws = np.tile(one, (N * (N + 1) // 2, 1))
    for red in (oracle.REDUCE_MEDIAN, oracle.REDUCE_MAX):
        s = oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_SAMPLED_STARTS, num_offsets=K,
                               reduce_mode=red, start_draws=draws)
        c = oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_CONFLICT_STARTS,
                               reduce_mode=red)
        assert np.array_equal(s["delay"], c["delay"])
        assert np.array_equal(s["slowdown"], c["slowdown"])
        assert np.count_nonzero(c["delay"]) > 0


def test_zero_draws_align_the_first_kernels():
    # draw 0 names (0, 0) for every pair: the FIRST alignment when the two
    # first kernels interfere, an empty set (delay 0) when they do not
    L = lib_from([[BIG + (2.0,), BIG + (3.0,)], [BIG + (1.0,)] * 4, [TINY + (5.0,)] * 3])
    N, K = 3, 4
    draws = np.zeros((N * (N + 1) // 2, K), np.uint64)
    s = oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_SAMPLED_STARTS, num_offsets=K,
                           start_draws=draws)
    f = oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_FIRST)
    M = models(A100, L)
    for i in range(N):
        for j in range(N):
            if conflicts(A100, M, i, j, 0, 0):
                assert s["delay"][i, j] == f["delay"][i, j]
            else:
                assert s["delay"][i, j] == 0.0
    # worked by hand: window min(5, 4) = 4 us, all of it in conflict at 1/2
    assert s["delay"][0, 1] == 2.0 and s["delay"][1, 0] == 2.0
    assert s["delay"][2, 2] == 0.0


def test_repeated_draws_count_as_a_multiset():
    # model 0: kernels of 1, 2, 4 us; model 1: one long kernel.  All conflict
    # with ratio 1/2, so the start pair (s, 0) gives half of model 0's time
    # from s on, capped by model 1's 10 us: (7/2, 3, 2) for s = 0, 1, 2.
    L = lib_from([[BIG + (1.0,), BIG + (2.0,), BIG + (4.0,)], [BIG + (10.0,)]])
    N = 2
    rows = np.zeros((3, 3), np.uint64)
    rows[pair_index(N, 0, 1)] = [draw_for(2, 3, 0, 1), draw_for(2, 3, 0, 1), draw_for(0, 3, 0, 1)]
    out = oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_SAMPLED_STARTS, num_offsets=3,
                             start_draws=rows, per_alignment=True)
    assert list(out["per_alignment"][0, 1]) == [2.0, 2.0, 3.5]
    assert out["delay"][0, 1] == 2.0          # a set {2, 3.5} would give 2.75
    # model 1's share of the same stretches, start pairs transposed
    assert list(out["per_alignment"][1, 0]) == [2.0, 2.0, 3.5]
    mx = oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_SAMPLED_STARTS, num_offsets=3,
                            reduce_mode=oracle.REDUCE_MAX, start_draws=rows)
    assert mx["delay"][0, 1] == 3.5


def test_draws_outside_the_interference_set_are_dropped():
    # MID (one block of 32 warps) fits beside another MID but not beside BIG
    # (64 warps): draws that start model 0 on its MID kernel are not in C_ij
    L = lib_from([[BIG + (2.0,), MID + (2.0,), BIG + (2.0,)], [MID + (8.0,)]])
    N = 2
    rows = np.zeros((3, 2), np.uint64)
    rows[pair_index(N, 0, 1)] = [draw_for(1, 3, 0, 1), draw_for(1, 3, 0, 1)]
    out = oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_SAMPLED_STARTS, num_offsets=2,
                             start_draws=rows, per_alignment=True)
    assert np.isnan(out["per_alignment"][0, 1]).all()
    assert np.isnan(out["per_alignment"][1, 0]).all()
    assert out["delay"][0, 1] == 0.0 and out["delay"][1, 0] == 0.0
    rows[pair_index(N, 0, 1)] = [draw_for(1, 3, 0, 1), draw_for(2, 3, 0, 1)]
    out = oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_SAMPLED_STARTS, num_offsets=2,
                             start_draws=rows, per_alignment=True)
    assert np.isnan(out["per_alignment"][0, 1, 0])
    assert out["delay"][0, 1] == 1.0 and out["delay"][1, 0] == 1.0


@pytest.mark.parametrize("dev", [A100, EDGE, MI355X])
def test_both_directions_split_the_conflicting_time(dev):
    # C_ji is C_ij transposed and the window is symmetric, so the two
    # directions of one draw share every conflicting stretch in full
    rng = np.random.default_rng(23)
    L = random_lib(rng, 4, 10)
    N, K = 4, 9
    draws = start_draws(N, K, seed=3)
    out = oracle.pair_matrix(dev, L, align_mode=oracle.ALIGN_SAMPLED_STARTS, num_offsets=K,
                             start_draws=draws, per_alignment=True)
    pa = out["per_alignment"]
    M = models(dev, L)
    members = 0
    for i in range(N):
        for j in range(i + 1, N):
            for r in range(K):
                x = int(draws[pair_index(N, i, j), r])
                si = ((x >> 32) * q_of(L, i)) >> 32
                sj = ((x & (TWO32 - 1)) * q_of(L, j)) >> 32
                assert np.isnan(pa[i, j, r]) == np.isnan(pa[j, i, r])
                if np.isnan(pa[i, j, r]):
                    continue
                members += 1
                total = brute.delay_all_pairs(dev, M[i], M[j], si, sj, weight=False)
                assert pa[i, j, r] + pa[j, i, r] == pytest.approx(total, rel=1e-12)
    assert members > 0


def test_empty_model_has_no_sampled_start_pairs():
    L = lib_from([[BIG + (2.0,)] * 3, [], [BIG + (1.0,)]])
    N, K = 3, 5
    draws = start_draws(N, K, seed=9)
    out = oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_SAMPLED_STARTS, num_offsets=K,
                             start_draws=draws, per_alignment=True)
    assert np.isnan(out["per_alignment"][1]).all() and np.isnan(out["per_alignment"][:, 1]).all()
    assert (out["delay"][1] == 0).all() and (out["delay"][:, 1] == 0).all()
    assert out["delay"][0, 2] > 0


def test_missing_or_short_draws_are_rejected():
    L = lib_from([[BIG + (2.0,)], [BIG + (1.0,)]])
    with pytest.raises(ValueError):
        oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_SAMPLED_STARTS, num_offsets=2)
    with pytest.raises(ValueError):
        oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_SAMPLED_STARTS, num_offsets=2,
                           start_draws=np.zeros(5, np.uint64))


def test_draws_are_seeded_and_uniform_over_start_kernels():
    a = start_draws(5, 7, seed=1)
    assert a.shape == (15, 7) and a.dtype == np.uint64
    assert np.array_equal(a, start_draws(5, 7, seed=1))
    big = start_draws(40, 64, seed=2).reshape(-1)
    q = 2000
    s = ((big >> np.uint64(32)) * np.uint64(q)) >> np.uint64(32)
    hist = np.bincount(s.astype(np.int64), minlength=q)
    expect = big.size / q
    # chi-square with q - 1 degrees of freedom, far from its 1e-6 tail
    chi2 = float(((hist - expect) ** 2 / expect).sum())
    assert chi2 < (q - 1) + 6 * math.sqrt(2 * (q - 1))
