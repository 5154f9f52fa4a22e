"""The exact integer division of the adjusted-occupancy simulation's block
counts (Sec. 3.2): floor(n / x) for n < 2^23 as (n * mag) >> shift with
mag = floor(2^k / x) + 1, k = 23 + ceil(log2 x).  The constants are
computed the way the library computes them (the double quotient 2^k / x,
truncated), then every product is checked against exact integer floor
division: each divisor up to 4096 at the numerators around each of its
multiples and at the top of the range, every numerator below 2^16 for
divisors up to 64, powers of two and their neighbours up to 2^24, and
seeded large divisors."""
import numpy as np
import pytest

N_BITS = 23


def constants(x):
    x = np.asarray(x, dtype=np.uint64)
    l = np.zeros_like(x)
    big = x > 1
    l[big] = np.ceil(np.log2(x[big].astype(np.float64))).astype(np.uint64)
    # ceil(log2 x) exactly, without rounding surprises near powers of two
    l = np.where((np.uint64(1) << l) < x, l + np.uint64(1), l)
    l = np.where(big & ((np.uint64(1) << (l - np.uint64(1))) >= x), l - np.uint64(1), l)
    k = np.uint64(N_BITS) + l
    q = (np.ldexp(1.0, k.astype(np.int64)) / x.astype(np.float64))
    mag = q.astype(np.uint64) + np.uint64(1)
    return mag, k


def check(x, n):
    x = np.asarray(x, np.uint64)
    n = np.asarray(n, np.uint64)
    mag, k = constants(x)
    assert np.all(mag < (np.uint64(1) << np.uint64(32)))
    got = (n * mag) >> k
    assert np.array_equal(got, n // x), (x[got != n // x][:5], n[got != n // x][:5])


def test_every_divisor_up_to_4096_at_its_multiples():
    # the product's excess grows with n, so the multiples at the top of the
    # range are the tightest: the first and last 64 multiples of every
    # divisor and 256 seeded ones, each with its neighbours
    top = (1 << N_BITS) - 1
    rng = np.random.default_rng(3)
    xs, ns = [], []
    for x in range(1, 4097):
        last = top // x
        m = np.concatenate([np.arange(0, min(64, last + 1)), np.arange(max(0, last - 63), last + 2),
                            rng.integers(0, last + 1, 256)]).astype(np.uint64) * np.uint64(x)
        n = np.concatenate([m, m - np.uint64(1), m + np.uint64(1), [top, top - 1]])
        n = n[n <= top]   # m - 1 wraps for m = 0
        xs.append(np.full(n.shape, x, np.uint64))
        ns.append(n)
    check(np.concatenate(xs), np.concatenate(ns))


@pytest.mark.parametrize("x", range(1, 65))
def test_every_numerator_below_2_16_for_small_divisors(x):
    n = np.arange(1 << 16, dtype=np.uint64)
    check(np.full(n.shape, x), n)


def test_powers_of_two_and_neighbours():
    top = (1 << N_BITS) - 1
    xs = sorted({v for e in range(25) for v in ((1 << e) - 1, 1 << e, (1 << e) + 1)
                 if 1 <= v < (1 << 24)})
    rng = np.random.default_rng(5)
    for x in xs:
        n = np.concatenate([rng.integers(0, top + 1, 20000, dtype=np.uint64),
                            np.arange(0, top + 1, x, dtype=np.uint64)[:100000]])
        n = np.concatenate([n, n + np.uint64(x - 1), [top]])
        n = n[n <= top]
        check(np.full(n.shape, x), n)


def test_seeded_large_divisors():
    rng = np.random.default_rng(11)
    top = (1 << N_BITS) - 1
    x = rng.integers(4097, 1 << 24, 200000, dtype=np.uint64)
    q = rng.integers(0, 2048, x.shape[0], dtype=np.uint64)
    n = np.minimum(q * x + rng.integers(0, 3, x.shape[0], dtype=np.uint64) - np.uint64(1), top)
    n = np.where(q * x == 0, np.uint64(0), n)
    check(x, n)
    check(x, rng.integers(0, top + 1, x.shape[0], dtype=np.uint64))
