"""Pins for the oracle's adjusted-occupancy simulation (Sec. 3.2, Eqs. 3-4).

The oracle is compared with things it shares no code with: the two-phase
formulas of Eqs. (3)-(4) evaluated by hand for two single kernels, block counts
found by adding one block at a time, an exact-arithmetic event simulation
written independently (tests/brute.py), and identities of the method.
"""
from fractions import Fraction

import numpy as np
import pytest

import brute
import oracle
from paper_2607_16784_amd.workloads import A100, EDGE, MI355X

ADJ = oracle.SWEEP_ADJUSTED

# A100-class kernels (W = 64 warps, 64 Ki registers, 164 KiB, 32 slots):
# FULL: 4 blocks of 16 warps on the busiest SM (grid 432 = 4 x 108 SMs) fill
#       all 64 warps; next to a copy of itself each keeps 32 warps = 2 blocks.
FULL = (432, 512, 16, 0)
# HALF: 2 blocks of 16 warps (32 warps).  Beside FULL: FULL may hold only 32
#       warps, so HALF keeps both its blocks, FULL keeps 2 of 4.
HALF = (216, 512, 16, 0)
# HOG: one block with 100000 B of shared memory (more than half of 164 KiB);
#      two of them cannot share an SM in space.
HOG = (108, 256, 16, 100_000)
# TINY: one 2-warp block; never interferes with the kernels above.
TINY = (1, 64, 16, 0)


def lib_from(models):
    rows = [k for m in models for k in m]
    off = np.zeros(len(models) + 1, np.int64)
    off[1:] = np.cumsum([len(m) for m in models])
    col = lambda i, dt: np.array([r[i] for r in rows], dt)  # noqa: E731
    return dict(offsets=off, grid=col(0, np.int32), threads=col(1, np.int32),
                regs=col(2, np.int32), smem=col(3, np.int32), duration=col(4, np.float64))


def eq3_pair(d_k, slow_k, d_l, slow_l):
    """Eqs. (3)-(4) for two single kernels that start together: delays of both.

    d~e = d * o/o~; Delta = min over the two; the kernel that ends first takes
    d~e, the other Delta + (d~e - Delta) * o~/o (the remainder at full speed).
    """
    de_k, de_l = Fraction(d_k) * slow_k, Fraction(d_l) * slow_l
    D = min(de_k, de_l)
    tk = de_k if de_k <= D else D + (de_k - D) / slow_k
    tl = de_l if de_l <= D else D + (de_l - D) / slow_l
    return tk - d_k, tl - d_l


@pytest.mark.parametrize("k,l,slow_k,slow_l", [
    (FULL, FULL, Fraction(2), Fraction(2)),   # 2 of 4 blocks each
    (FULL, HALF, Fraction(2), Fraction(1)),   # FULL squeezed, HALF unaffected
    (HALF, FULL, Fraction(1), Fraction(2)),
    (HOG, HOG, Fraction(2), Fraction(2)),     # cannot co-reside: alternate
])
@pytest.mark.parametrize("d_k,d_l", [(4.0, 6.0), (6.0, 4.0), (5.0, 5.0), (1.0, 16.0)])
def test_single_kernels_follow_eq3(k, l, slow_k, slow_l, d_k, d_l):
    L = lib_from([[k + (d_k,)], [l + (d_l,)]])
    out = oracle.pair_matrix(A100, L, sweep_mode=ADJ)
    want_k, want_l = eq3_pair(d_k, slow_k, d_l, slow_l)
    assert out["delay"][0, 1] == float(want_k)
    assert out["delay"][1, 0] == float(want_l)


def test_worked_example_sequence_against_one_long_kernel():
    # A = two FULL kernels of 2; B = one FULL kernel of 8; every pair runs at
    # half speed.  A's first kernel ends at 4 (delay 2) with B 2 units in;
    # A's second ends at 8 (delay 2 more) with B 4 units in; A is done, so
    # B finishes alone: Delta_A = 4, Delta_B = 4 (T~_B = 12).
    L = lib_from([[FULL + (2.0,)] * 2, [FULL + (8.0,)]])
    out = oracle.pair_matrix(A100, L, sweep_mode=ADJ)
    assert out["delay"][0, 1] == 4.0 and out["delay"][1, 0] == 4.0
    # slowdown uses the same gamma as Alg. 1: gamma_AB = max(2/1, 1) = 2
    assert out["slowdown"][0, 1] == 2.0 * 4.0 / 4.0
    assert out["slowdown"][1, 0] == 4.0 / 8.0


def test_adjusted_blocks_hand_cases():
    L = lib_from([[FULL + (1.0,)], [HALF + (1.0,)], [HOG + (1.0,)], [TINY + (1.0,)]])
    g, t, r, s = L["grid"], L["threads"], L["regs"], L["smem"]
    assert oracle.adjusted_blocks(A100, g, t, r, s, 0, 0) == 2
    assert oracle.adjusted_blocks(A100, g, t, r, s, 0, 1) == 2
    assert oracle.adjusted_blocks(A100, g, t, r, s, 1, 0) == 2
    assert oracle.adjusted_blocks(A100, g, t, r, s, 2, 2) == 0   # 100000 B > 83968 B left
    assert oracle.adjusted_blocks(A100, g, t, r, s, 0, 3) == 3   # TINY holds 2 warps: 62 / 16
    assert oracle.adjusted_blocks(A100, g, t, r, s, 3, 0) == 1   # TINY keeps its one block


def random_kernels(rng, n, dev):
    ks = []
    while len(ks) < n:
        t = int(rng.choice([64, 128, 256, 512, 1024]))
        r = int(rng.integers(16, 129))
        if r * t > dev["regs_per_sm"]:
            continue
        g = int(rng.integers(1, 8 * dev["num_sm"]))
        s = int(rng.choice([0, int(rng.integers(0, dev["smem_per_sm"] // 2 + 20_000))]))
        ks.append((g, t, r, s))
    return ks


@pytest.mark.parametrize("dev", [A100, EDGE, MI355X], ids=["a100", "edge", "mi355x"])
def test_adjusted_blocks_match_counting(dev):
    rng = np.random.default_rng(7)
    ks = random_kernels(rng, 60, dev)
    L = lib_from([[k + (1.0,)] for k in ks])
    g, t, r, s = L["grid"], L["threads"], L["regs"], L["smem"]
    sk = [brute.SimKernel(dev, *k, 1.0) for k in ks]
    for u in range(len(ks)):
        for v in range(len(ks)):
            if sk[u].beta == 0 or sk[v].beta == 0:
                continue
            want = brute.blocks_beside(dev, sk[u], sk[v])
            assert oracle.adjusted_blocks(dev, g, t, r, s, u, v) == want, (ks[u], ks[v])


def random_lib(rng, n_models, qmax, dev, dyadic=False):
    models = []
    for _ in range(n_models):
        q = int(rng.integers(1, qmax + 1))
        ks = random_kernels(rng, q, dev)
        if dyadic:
            ds = [float(rng.integers(1, 17)) / 4 for _ in range(q)]
        else:
            ds = [float(rng.lognormal(1.0, 1.0)) for _ in range(q)]
        models.append([k + (d,) for k, d in zip(ks, ds)])
    return lib_from(models)


def close(got, want, rel=1e-12):
    want = float(want)
    return abs(got - want) <= rel * max(abs(want), 1e-300) or got == want


@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("dev", [A100, EDGE, MI355X], ids=["a100", "edge", "mi355x"])
def test_first_and_starts_match_exact_simulation(seed, dev):
    rng = np.random.default_rng(100 + seed)
    L = random_lib(rng, 3, 8, dev)
    ms = [brute.sim_model(dev, L, m) for m in range(3)]
    out = oracle.pair_matrix(dev, L, sweep_mode=ADJ)
    for i in range(3):
        for j in range(3):
            want, _ = brute.adjusted_delays(dev, ms[i], ms[j])
            assert close(out["delay"][i, j], want), (i, j)
            for si in range(len(ms[i])):
                for sj in range(len(ms[j])):
                    got = oracle.sweep_start_pair(dev, L, i, j, si, sj, sweep_mode=ADJ)
                    want, _ = brute.adjusted_delays(dev, ms[i], ms[j], si, sj)
                    assert close(got, want), (i, j, si, sj)


@pytest.mark.parametrize("seed", range(4))
def test_offsets_match_exact_simulation(seed):
    rng = np.random.default_rng(200 + seed)
    L = random_lib(rng, 2, 8, EDGE)
    ms = [brute.sim_model(EDGE, L, m) for m in range(2)]
    K = 6
    out = oracle.pair_matrix(EDGE, L, align_mode=oracle.ALIGN_OFFSETS, reduce_mode=oracle.REDUCE_MAX,
                             num_offsets=K, sweep_mode=ADJ, per_alignment=True)
    for i in range(2):
        Ti = float(np.sum(L["duration"][L["offsets"][i]:L["offsets"][i + 1]]))
        for j in range(2):
            for r in range(K):
                tau = Ti * r / K
                want, _ = brute.adjusted_delays(EDGE, ms[i], ms[j], offset=tau)
                assert close(out["per_alignment"][i, j, r], want, 1e-11), (i, j, r)
            assert out["delay"][i, j] == max(out["per_alignment"][i, j].max(), 0.0)


def test_dyadic_traces_are_exact():
    # quarter-integer durations and speeds 1/2 or 1 keep every event time
    # dyadic, so the fp64 simulation must equal the exact one bit for bit
    rng = np.random.default_rng(11)
    models = []
    for _ in range(3):
        q = int(rng.integers(1, 9))
        models.append([(FULL if rng.random() < 0.5 else HALF) + (float(rng.integers(1, 17)) / 4,)
                       for _ in range(q)])
    L = lib_from(models)
    ms = [brute.sim_model(A100, L, m) for m in range(3)]
    out = oracle.pair_matrix(A100, L, sweep_mode=ADJ)
    for i in range(3):
        for j in range(3):
            want, _ = brute.adjusted_delays(A100, ms[i], ms[j])
            assert out["delay"][i, j] == float(want)


def test_no_interference_no_delay():
    rng = np.random.default_rng(3)
    L = lib_from([[TINY + (float(rng.lognormal()),) for _ in range(int(rng.integers(1, 20)))]
                  for _ in range(4)])
    for mode, K in ((oracle.ALIGN_FIRST, 1), (oracle.ALIGN_OFFSETS, 5)):
        out = oracle.pair_matrix(A100, L, align_mode=mode, num_offsets=K, sweep_mode=ADJ)
        assert np.all(out["delay"] == 0.0)


def test_power_of_two_scaling_is_exact():
    rng = np.random.default_rng(5)
    L = random_lib(rng, 3, 10, A100)
    a = oracle.pair_matrix(A100, L, sweep_mode=ADJ)
    L2 = dict(L, duration=L["duration"] * 8.0)
    b = oracle.pair_matrix(A100, L2, sweep_mode=ADJ)
    assert np.array_equal(b["delay"], 8.0 * a["delay"])
    assert np.array_equal(b["slowdown"], a["slowdown"])


def test_delay_bounds():
    # each kernel runs at no less than 1/beta of its isolated speed (or 1/2
    # when sharing in time), so Delta_i <= sum_k d_k (max(beta_k, 2) - 1)
    rng = np.random.default_rng(9)
    L = random_lib(rng, 4, 12, A100)
    occ = oracle.occupancy(A100, L["grid"], L["threads"], L["regs"], L["smem"])
    out = oracle.pair_matrix(A100, L, sweep_mode=ADJ)
    for i in range(4):
        a, b = L["offsets"][i], L["offsets"][i + 1]
        beta = occ["resident_blocks"][a:b]
        bound = float(np.sum(L["duration"][a:b] * (np.maximum(beta, 2) - 1)))
        assert np.all(out["delay"][i] >= 0.0)
        assert np.all(out["delay"][i] <= bound * (1 + 1e-12))


def test_first_alignment_is_symmetric_in_roles():
    # swapping which model is called i leaves the simulation unchanged, so
    # Delta_ij from the (i, j) run equals B's delay of the (j, i) run
    rng = np.random.default_rng(13)
    L = random_lib(rng, 3, 10, A100)
    ms = [brute.sim_model(A100, L, m) for m in range(3)]
    out = oracle.pair_matrix(A100, L, sweep_mode=ADJ)
    for i in range(3):
        for j in range(3):
            _, dj = brute.adjusted_delays(A100, ms[j], ms[i])
            assert close(out["delay"][i, j], dj)


# ---------------------------------------------------------------------------
# Scheduling policies of Sec. 3.2 beside equal partitioning: priority-based
# (in Delta_ij the partner j's kernels keep all their blocks) and
# first-come-first-served (the kernel already running keeps all its blocks;
# kernels that start together share equally).
# ---------------------------------------------------------------------------
PRIO, FCFS = oracle.POLICY_PRIORITY, oracle.POLICY_FCFS


def test_blocks_beside_a_whole_partner_hand_cases():
    L = lib_from([[FULL + (1.0,)], [HALF + (1.0,)], [HOG + (1.0,)], [TINY + (1.0,)]])
    g, t, r, s = L["grid"], L["threads"], L["regs"], L["smem"]
    ab = lambda u, v: oracle.adjusted_blocks(A100, g, t, r, s, u, v, PRIO)  # noqa: E731
    assert ab(0, 0) == 0   # FULL holds all 64 warps: nothing fits beside it
    assert ab(0, 1) == 2   # HALF holds 32 warps: 32 / 16 = 2 of FULL's 4 blocks
    assert ab(1, 0) == 0
    assert ab(2, 2) == 0   # 100000 B held, 67936 B left < 100000 B
    assert ab(0, 3) == 3   # TINY holds 2 warps: 62 / 16 = 3
    assert ab(3, 0) == 0   # not even TINY's 2-warp block fits beside FULL
    assert ab(3, 1) == 1


@pytest.mark.parametrize("dev", [A100, EDGE, MI355X], ids=["a100", "edge", "mi355x"])
def test_blocks_beside_a_whole_partner_match_counting(dev):
    rng = np.random.default_rng(17)
    ks = random_kernels(rng, 60, dev)
    L = lib_from([[k + (1.0,)] for k in ks])
    g, t, r, s = L["grid"], L["threads"], L["regs"], L["smem"]
    sk = [brute.SimKernel(dev, *k, 1.0) for k in ks]
    for u in range(len(ks)):
        for v in range(len(ks)):
            if sk[u].beta == 0 or sk[v].beta == 0:
                continue
            want = brute.blocks_beside_whole(dev, sk[u], sk[v])
            for pol in (PRIO, FCFS):
                assert oracle.adjusted_blocks(dev, g, t, r, s, u, v, pol) == want


def priority_single(d_k, slow_k, d_l):
    """Victim k beside partner l that keeps all its blocks (Eqs. 3-4 with l at
    its isolated speed): the run ends when the first of the two completes;
    slow_k = None: k makes no progress until then."""
    d_k, d_l = Fraction(d_k), Fraction(d_l)
    if slow_k is None:
        return d_l
    de_k = d_k * slow_k
    if de_k <= d_l:
        return de_k - d_k
    return d_l - d_l / slow_k


@pytest.mark.parametrize("k,l,slow_k", [
    (FULL, HALF, Fraction(2)),   # 2 of FULL's 4 blocks fit beside HALF's 32 warps
    (HALF, FULL, None),          # nothing fits beside FULL: HALF waits
    (HOG, HOG, None),
    (FULL, TINY, Fraction(4, 3)),
])
@pytest.mark.parametrize("d_k,d_l", [(4.0, 2.0), (2.0, 6.0), (5.0, 5.0), (1.0, 16.0)])
def test_priority_single_kernels_by_hand(k, l, slow_k, d_k, d_l):
    L = lib_from([[k + (d_k,)], [l + (d_l,)]])
    out = oracle.pair_matrix(A100, L, sweep_mode=ADJ, policy=PRIO)
    # exact except for the rounding of beta / b~ = 4/3 (one quotient)
    assert close(out["delay"][0, 1], priority_single(d_k, slow_k, d_l), 1e-15)


def test_policies_worked_sequence_against_one_long_kernel():
    # A = two FULL kernels of 2, B = one FULL kernel of 8 (nothing fits
    # beside a whole FULL kernel; equal shares give each 2 of 4 blocks).
    L = lib_from([[FULL + (2.0,)] * 2, [FULL + (8.0,)]])
    eq = oracle.pair_matrix(A100, L, sweep_mode=ADJ)
    assert eq["delay"][0, 1] == 4.0 and eq["delay"][1, 0] == 4.0
    # FCFS: both start at 0 and share equally until A's first kernel ends at
    # 4 (A +2, B 2 units in); B's kernel is now the older one and keeps the
    # SM, A's second kernel waits until B ends at 4 + 6 = 10: A +6.
    fc = oracle.pair_matrix(A100, L, sweep_mode=ADJ, policy=FCFS)
    assert fc["delay"][0, 1] == 8.0 and fc["delay"][1, 0] == 2.0
    # priority to the partner: A waits all of B's 8; B waits until both of
    # A's kernels are done at 4
    pr = oracle.pair_matrix(A100, L, sweep_mode=ADJ, policy=PRIO)
    assert pr["delay"][0, 1] == 8.0 and pr["delay"][1, 0] == 4.0


def test_fcfs_offsets_the_running_kernel_keeps_its_blocks():
    # i = one FULL kernel of 4; j = one HALF kernel of 2 joining at tau = 1
    # (OFFSETS with K = 4: tau_1 = T_i / 4 = 1).  i's kernel was running
    # first and keeps its 64 warps; HALF fits nothing and waits until i
    # ends at 4, where the run ends: Delta^1_ij = 0, Delta^1_ji (the offset
    # is T_j r / K for the pair (j, i)) is checked against the exact run.
    L = lib_from([[FULL + (4.0,)], [HALF + (2.0,)]])
    out = oracle.pair_matrix(A100, L, align_mode=oracle.ALIGN_OFFSETS,
                             reduce_mode=oracle.REDUCE_MAX, num_offsets=4, sweep_mode=ADJ,
                             policy=FCFS, per_alignment=True)
    assert out["per_alignment"][0, 1, 1] == 0.0
    # at tau = 0 both start together: equal shares (FULL 2 of 4 blocks,
    # HALF keeps both): FULL at half speed until HALF ends at 2, run ends
    assert out["per_alignment"][0, 1, 0] == 1.0
    ms = [brute.sim_model(A100, L, m) for m in range(2)]
    for r in range(4):
        want, _ = brute.adjusted_delays(A100, ms[1], ms[0], offset=Fraction(2 * r, 4),
                                        policy="fcfs")
        assert out["per_alignment"][1, 0, r] == float(want)


@pytest.mark.parametrize("seed", range(4))
def test_fcfs_equals_equal_partitioning_when_kernels_start_together(seed):
    # a model beside a copy of itself from the first kernels: every stretch
    # ends with both kernels completing, so every start is simultaneous
    rng = np.random.default_rng(300 + seed)
    L = random_lib(rng, 3, 10, A100)
    eq = oracle.pair_matrix(A100, L, sweep_mode=ADJ)
    fc = oracle.pair_matrix(A100, L, sweep_mode=ADJ, policy=FCFS)
    assert np.array_equal(np.diag(eq["delay"]), np.diag(fc["delay"]))


@pytest.mark.parametrize("policy,name", [(PRIO, "priority"), (FCFS, "fcfs")])
@pytest.mark.parametrize("dev", [A100, EDGE, MI355X], ids=["a100", "edge", "mi355x"])
def test_policies_match_exact_simulation(policy, name, dev):
    rng = np.random.default_rng(400 + policy)
    L = random_lib(rng, 3, 8, dev)
    ms = [brute.sim_model(dev, L, m) for m in range(3)]
    out = oracle.pair_matrix(dev, L, sweep_mode=ADJ, policy=policy)
    for i in range(3):
        for j in range(3):
            want, _ = brute.adjusted_delays(dev, ms[i], ms[j], policy=name)
            assert close(out["delay"][i, j], want), (i, j)
            for si in range(len(ms[i])):
                for sj in range(len(ms[j])):
                    got = oracle.sweep_start_pair(dev, L, i, j, si, sj, sweep_mode=ADJ,
                                                  policy=policy)
                    want, _ = brute.adjusted_delays(dev, ms[i], ms[j], si, sj, policy=name)
                    assert close(got, want), (i, j, si, sj)


@pytest.mark.parametrize("policy,name", [(PRIO, "priority"), (FCFS, "fcfs")])
def test_policies_offsets_match_exact_simulation(policy, name):
    rng = np.random.default_rng(500 + policy)
    L = random_lib(rng, 2, 8, EDGE)
    ms = [brute.sim_model(EDGE, L, m) for m in range(2)]
    K = 6
    out = oracle.pair_matrix(EDGE, L, align_mode=oracle.ALIGN_OFFSETS,
                             reduce_mode=oracle.REDUCE_MAX, num_offsets=K, sweep_mode=ADJ,
                             policy=policy, per_alignment=True)
    for i in range(2):
        Ti = float(np.sum(L["duration"][L["offsets"][i]:L["offsets"][i + 1]]))
        for j in range(2):
            for r in range(K):
                want, _ = brute.adjusted_delays(EDGE, ms[i], ms[j], offset=Ti * r / K,
                                                policy=name)
                assert close(out["per_alignment"][i, j, r], want, 1e-11), (i, j, r)


@pytest.mark.parametrize("policy,name", [(PRIO, "priority"), (FCFS, "fcfs")])
def test_policies_dyadic_traces_are_exact(policy, name):
    rng = np.random.default_rng(600 + policy)
    models = []
    for _ in range(3):
        q = int(rng.integers(1, 9))
        models.append([(FULL, HALF, TINY)[int(rng.integers(0, 3))] +
                       (float(rng.integers(1, 17)) / 4,) for _ in range(q)])
    L = lib_from(models)
    ms = [brute.sim_model(A100, L, m) for m in range(3)]
    out = oracle.pair_matrix(A100, L, sweep_mode=ADJ, policy=policy)
    for i in range(3):
        for j in range(3):
            want, _ = brute.adjusted_delays(A100, ms[i], ms[j], policy=name)
            assert out["delay"][i, j] == float(want), (i, j)


@pytest.mark.parametrize("policy", [PRIO, FCFS])
def test_policies_invariants(policy):
    rng = np.random.default_rng(7)
    L = lib_from([[TINY + (float(rng.lognormal()),) for _ in range(int(rng.integers(1, 20)))]
                  for _ in range(3)])
    out = oracle.pair_matrix(A100, L, sweep_mode=ADJ, policy=policy)
    assert np.all(out["delay"] == 0.0)          # no interference, no delay
    L = random_lib(rng, 3, 10, A100)
    a = oracle.pair_matrix(A100, L, sweep_mode=ADJ, policy=policy)
    b = oracle.pair_matrix(A100, dict(L, duration=L["duration"] * 4.0), sweep_mode=ADJ,
                           policy=policy)
    assert np.array_equal(b["delay"], 4.0 * a["delay"])
    assert np.all(a["delay"] >= 0.0)


def test_policy_needs_the_adjusted_simulation():
    L = lib_from([[FULL + (1.0,)], [HALF + (1.0,)]])
    with pytest.raises(ValueError):
        oracle.pair_matrix(A100, L, policy=PRIO)          # temporal sweep
    with pytest.raises(ValueError):
        oracle.pair_matrix(A100, L, sweep_mode=ADJ, policy=3)
