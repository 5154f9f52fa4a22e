"""Pins for the oracle's occupancy (Sec. 3.1, Eq. 1) and Eq. (2) predicate."""
from fractions import Fraction

import numpy as np
import pytest

import brute
import oracle
from paper_2607_16784_amd.workloads import A100, EDGE, MI355X

LIM_W, LIM_R, LIM_M, LIM_B = 1, 2, 4, 8

# (threads, regs, smem) -> (b, limiter, a, o); values worked out by hand from
# Eq. (1): W = 2048/32 = 64 warps, 32 block slots, 65536 registers and
# 167936 bytes of shared memory per SM for the A100-class descriptor.
A100_CASES = [
    ((256, 32, 0), (8, LIM_W | LIM_R, 64, 1.0)),       # 64/8 = 8, 65536/8192 = 8
    ((1024, 64, 0), (1, LIM_R, 32, 0.5)),               # 65536/65536 = 1 < 64/32 = 2
    ((128, 16, 49152), (3, LIM_M, 12, 0.1875)),         # 167936/49152 = 3.4
    ((64, 16, 0), (32, LIM_W | LIM_B, 64, 1.0)),        # 64/2 = 32 = slot limit
    ((1024, 65, 0), (0, LIM_R, 0, 0.0)),                # 66560 registers > 65536
]
# Edge descriptor: W = 1536/32 = 48, 16 slots.
EDGE_CASES = [
    ((1024, 32, 0), (1, LIM_W, 32, 32 / 48)),           # 48/32 = 1 < 65536/32768 = 2
    ((64, 16, 0), (16, LIM_B, 32, 32 / 48)),            # 48/2 = 24 > 16 slots
]

# MI355X (gfx950): wavefronts of 64, W = 2048/64 = 32 per CU, 32 workgroup
# slots, 131072 VGPR lanes and 163840 bytes of LDS per CU.
MI355X_CASES = [
    ((256, 128, 0), (4, LIM_R, 16, 0.5)),               # 32/4 = 8 > 131072/32768 = 4
    ((64, 32, 0), (32, LIM_W | LIM_B, 32, 1.0)),        # 32/1 = 32 = slots < 131072/2048
    ((1024, 128, 0), (1, LIM_R, 16, 0.5)),              # 131072/131072 = 1 < 32/16 = 2
    ((256, 64, 65536), (2, LIM_M, 8, 0.25)),            # 163840/65536 = 2.5
    ((100, 16, 0), (16, LIM_W, 32, 1.0)),               # W_b = ceil(100/64) = 2: 32/2 = 16
    ((512, 256, 0), (1, LIM_R, 8, 0.25)),               # 131072/131072 = 1 < 32/8 = 4
    ((1024, 129, 0), (0, LIM_R, 0, 0.0)),               # 132096 VGPR lanes > 131072
]


def _occ(dev, cases, grid=10_000):
    g = np.full(len(cases), grid, np.int32)
    t = np.array([c[0][0] for c in cases], np.int32)
    r = np.array([c[0][1] for c in cases], np.int32)
    s = np.array([c[0][2] for c in cases], np.int32)
    return oracle.occupancy(dev, g, t, r, s)


@pytest.mark.parametrize("dev,cases", [(A100, A100_CASES), (EDGE, EDGE_CASES),
                                      (MI355X, MI355X_CASES)])
def test_closed_form_cases(dev, cases):
    out = _occ(dev, cases)
    for idx, (_, (b, lim, a, o)) in enumerate(cases):
        assert out["blocks_per_sm"][idx] == b
        assert out["limiter"][idx] == lim
        assert out["active_warps"][idx] == a
        assert out["occupancy"][idx] == o
    infeasible = any(c[1][0] == 0 for c in cases)
    assert bool(out["status"] & oracle.ST_INFEASIBLE_KERNEL) == infeasible


def test_resident_blocks_follow_grid():
    # 200 blocks over 108 SMs put at most 2 on one SM.
    t = np.array([256, 1024, 64], np.int32)
    r = np.array([32, 64, 16], np.int32)
    out = oracle.occupancy(A100, np.full(3, 200, np.int32), t, r, np.zeros(3, np.int32))
    assert list(out["resident_blocks"]) == [2, 1, 2]
    out = oracle.occupancy(A100, np.full(3, 1, np.int32), t, r, np.zeros(3, np.int32))
    assert list(out["resident_blocks"]) == [1, 1, 1]
    # 300 workgroups over 256 CUs put at most 2 on one CU; 256 put 1
    out = oracle.occupancy(MI355X, np.array([300, 300, 256], np.int32),
                           np.array([256, 1024, 64], np.int32), np.array([128, 128, 32], np.int32),
                           np.zeros(3, np.int32))
    assert list(out["resident_blocks"]) == [2, 1, 1]


def test_invalid_configuration_flagged():
    out = oracle.occupancy(A100, np.array([0, 5], np.int32), np.array([128, 0], np.int32),
                           np.array([32, 32], np.int32), np.array([0, 0], np.int32))
    assert list(out["blocks_per_sm"]) == [0, 0]
    assert out["status"] & oracle.ST_INVALID_CONFIG
    assert out["status"] & oracle.ST_INFEASIBLE_KERNEL


@pytest.mark.parametrize("dev", [A100, EDGE, MI355X])
def test_blocks_match_counting_and_invariants(dev):
    rng = np.random.default_rng(11)
    n = 3000
    g = rng.integers(1, 5000, n).astype(np.int32)
    t = rng.choice([32, 64, 96, 128, 256, 512, 1024], n).astype(np.int32)
    r = rng.integers(0, 256, n).astype(np.int32)
    s = rng.integers(0, 120_000, n).astype(np.int32)
    out = oracle.occupancy(dev, g, t, r, s)
    W = dev["max_threads_per_sm"] // dev["warp_size"]
    for u in range(n):
        b = brute.blocks_by_counting(dev, int(t[u]), int(r[u]), int(s[u]))
        assert out["blocks_per_sm"][u] == b
        wb = -(-int(t[u]) // dev["warp_size"])
        assert out["active_warps"][u] == wb * b <= W
        # Eq. (1), exact: the fp64 value is the correctly rounded a / W.
        assert out["occupancy"][u] == float(Fraction(wb * b, W))
        beta = out["resident_blocks"][u]
        assert 0 <= beta <= b <= dev["max_blocks_per_sm"]
        if b > 0:
            assert beta >= 1
            f, _ = brute.footprint(dev, int(g[u]), int(t[u]), int(r[u]), int(s[u]))
            assert brute.fits_together(dev, f, (0, 0, 0, 0))


def test_conflict_predicate_by_fit():
    rng = np.random.default_rng(5)
    n = 400
    g = rng.integers(1, 400, n).astype(np.int32)
    t = rng.choice([64, 128, 256, 512, 1024], n).astype(np.int32)
    r = rng.integers(16, 64, n).astype(np.int32)
    s = rng.integers(0, 60_000, n).astype(np.int32)
    fps = [brute.footprint(A100, int(g[u]), int(t[u]), int(r[u]), int(s[u]))[0] for u in range(n)]
    seen = set()
    for _ in range(3000):
        u, v = (int(x) for x in rng.integers(0, n, 2))
        want = not brute.fits_together(A100, fps[u], fps[v])
        seen.add(want)
        assert oracle.conflict(A100, g, t, r, s, u, v) == want
        assert oracle.conflict(A100, g, t, r, s, v, u) == want
    assert seen == {True, False}


def test_conflict_boundaries_are_strict():
    # Two kernels of 32 warps each fill W = 64 exactly: no conflict; one more
    # warp on either side is a conflict (Eq. 2 uses '>').
    g = np.array([108, 108, 108], np.int32)          # one block per SM
    t = np.array([1024, 1024, 1056], np.int32)       # 32, 32, 33 warps
    r = np.array([16, 16, 16], np.int32)
    s = np.zeros(3, np.int32)
    assert not oracle.conflict(A100, g, t, r, s, 0, 1)
    assert oracle.conflict(A100, g, t, r, s, 0, 2)
    # Shared memory: 83968 + 83968 = 167936 fits, +1 byte does not.
    g2 = np.array([108, 108, 108], np.int32)
    t2 = np.array([64, 64, 64], np.int32)
    r2 = np.array([16, 16, 16], np.int32)
    s2 = np.array([83968, 83968, 83969], np.int32)
    assert not oracle.conflict(A100, g2, t2, r2, s2, 0, 1)
    assert oracle.conflict(A100, g2, t2, r2, s2, 0, 2)
