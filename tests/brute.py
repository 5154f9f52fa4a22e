"""Independent pure-Python formulations used to pin the oracle on tiny inputs.

None of these follows the oracle's code path:
  * resident blocks per SM are found by counting blocks up until one more
    would not fit, instead of the minimum of integer quotients;
  * interference is "the two footprints do not fit on one SM together";
  * the delay of an alignment sums the clipped intersection of EVERY pair of
    kernel intervals (O(q_i q_j)), instead of a two-pointer walk;
  * for integer durations, a unit-time-step simulation gives the same delay;
  * the Sec. 3.2 adjusted-occupancy simulation counts blocks one at a time
    and runs an absolute clock over work done, in exact arithmetic.
All arithmetic here is exact (fractions) where that matters.
"""
from __future__ import annotations

from fractions import Fraction


def blocks_by_counting(dev, threads, regs, smem):
    """Largest n such that n blocks fit one SM (0 when none fits)."""
    W = dev["max_threads_per_sm"] // dev["warp_size"]
    wb = -(-threads // dev["warp_size"])
    n = 0
    while True:
        m = n + 1
        fits = (m * wb <= W and m * regs * threads <= dev["regs_per_sm"]
                and m * smem <= dev["smem_per_sm"] and m <= dev["max_blocks_per_sm"])
        if not fits:
            return n
        n = m


def footprint(dev, grid, threads, regs, smem):
    """(warps, registers, shared bytes, blocks) used on the busiest SM, and a."""
    b = blocks_by_counting(dev, threads, regs, smem)
    wb = -(-threads // dev["warp_size"])
    beta = min(b, -(-grid // dev["num_sm"]))
    return (beta * wb, beta * regs * threads, beta * smem, beta), wb * b


def fits_together(dev, f1, f2):
    W = dev["max_threads_per_sm"] // dev["warp_size"]
    cap = (W, dev["regs_per_sm"], dev["smem_per_sm"], dev["max_blocks_per_sm"])
    return all(x + y <= c for x, y, c in zip(f1, f2, cap))


class Model:
    def __init__(self, dev, lib, m):
        a, b = int(lib["offsets"][m]), int(lib["offsets"][m + 1])
        self.q = b - a
        self.d = [float(x) for x in lib["duration"][a:b]]
        self.fp = []
        self.a = []
        for u in range(a, b):
            f, act = footprint(dev, int(lib["grid"][u]), int(lib["threads"][u]),
                               int(lib["regs"][u]), int(lib["smem"][u]))
            self.fp.append(f)
            self.a.append(act)


def _timeline(d, start, shift=0.0):
    t = [shift]
    for x in d[start:]:
        t.append(t[-1] + x)
    return t


def delay_all_pairs(dev, mi, mj, s_i=0, s_j=0, offset=None, exact=False, weight=True):
    """Delay of model i over one alignment by summing every interval pair.

    With offset=None the alignment is the start pair (s_i, s_j); otherwise
    model j starts `offset` after model i (both from their first kernel).
    weight=False returns the total conflicting overlap time instead.
    """
    num = Fraction if exact else float
    if offset is None:
        x = _timeline([num(v) for v in mi.d], s_i, num(0))
        y = _timeline([num(v) for v in mj.d], s_j, num(0))
        ki, lj, w0 = s_i, s_j, num(0)
    else:
        x = _timeline([num(v) for v in mi.d], 0, num(0))
        y = _timeline([num(v) for v in mj.d], 0, num(offset))
        ki, lj, w0 = 0, 0, num(offset)
    w1 = min(x[-1], y[-1])
    total = num(0)
    for k in range(len(x) - 1):
        for l in range(len(y) - 1):
            lo = max(x[k], y[l], w0)
            hi = min(x[k + 1], y[l + 1], w1)
            if hi > lo and not fits_together(dev, mi.fp[ki + k], mj.fp[lj + l]):
                ak, al = mi.a[ki + k], mj.a[lj + l]
                share = (Fraction(ak, ak + al) if exact else ak / (ak + al)) if weight else 1
                total += (hi - lo) * share
    return total


def delay_unit_steps(dev, mi, mj, s_i=0, s_j=0):
    """Same delay for integer durations by stepping time one unit at a time."""
    x = _timeline([int(v) for v in mi.d], s_i)
    y = _timeline([int(v) for v in mj.d], s_j)
    w1 = min(x[-1], y[-1])
    total = Fraction(0)
    k = l = 0
    for t in range(int(w1)):
        while x[k + 1] <= t:
            k += 1
        while y[l + 1] <= t:
            l += 1
        if not fits_together(dev, mi.fp[s_i + k], mj.fp[s_j + l]):
            ak, al = mi.a[s_i + k], mj.a[s_j + l]
            total += Fraction(ak, ak + al)
    return total


# ---------------------------------------------------------------------------
# Sec. 3.2 adjusted-occupancy simulation, written independently of the oracle:
# blocks are counted one at a time, time is an absolute clock, progress is
# tracked as work done (not work left), and all arithmetic is exact.
# ---------------------------------------------------------------------------

def capacities(dev):
    W = dev["max_threads_per_sm"] // dev["warp_size"]
    return (W, dev["regs_per_sm"], dev["smem_per_sm"], dev["max_blocks_per_sm"])


class SimKernel:
    def __init__(self, dev, grid, threads, regs, smem, d):
        self.fp, _ = footprint(dev, grid, threads, regs, smem)
        self.beta = self.fp[3]
        wb = -(-threads // dev["warp_size"])
        self.per_block = (wb, regs * threads, smem, 1)
        self.d = Fraction(d)


def sim_model(dev, lib, m):
    a, b = int(lib["offsets"][m]), int(lib["offsets"][m + 1])
    return [SimKernel(dev, int(lib["grid"][u]), int(lib["threads"][u]), int(lib["regs"][u]),
                      int(lib["smem"][u]), float(lib["duration"][u])) for u in range(a, b)]


def blocks_beside(dev, k, l):
    """Blocks of k that fit once l holds at most half of every resource."""
    cap = capacities(dev)
    held = [min(l.fp[r], cap[r] // 2) for r in range(4)]
    n = 0
    while n < k.beta:
        need = [(n + 1) * k.per_block[r] for r in range(4)]
        if any(held[r] + need[r] > cap[r] for r in range(4)):
            break
        n += 1
    return n


def blocks_beside_whole(dev, k, l):
    """Blocks of k that fit while l keeps every block it has on the SM."""
    cap = capacities(dev)
    n = 0
    while n < k.beta:
        need = [(n + 1) * k.per_block[r] for r in range(4)]
        if any(l.fp[r] + need[r] > cap[r] for r in range(4)):
            break
        n += 1
    return n


def speeds(dev, k, l, first=None):
    """Fraction of isolated speed of k and l while they run together.
    first = None: equal partitioning; "k" or "l": that kernel keeps all its
    blocks and the other gets what is left (speed 0 when nothing fits)."""
    if fits_together(dev, k.fp, l.fp):
        return Fraction(1), Fraction(1)
    if first == "k":
        return Fraction(1), Fraction(blocks_beside_whole(dev, l, k), l.beta)
    if first == "l":
        return Fraction(blocks_beside_whole(dev, k, l), k.beta), Fraction(1)
    bk, bl = blocks_beside(dev, k, l), blocks_beside(dev, l, k)
    if bk == 0 or bl == 0:               # no space sharing: alternate in time
        return Fraction(1, 2), Fraction(1, 2)
    return Fraction(bk, k.beta), Fraction(bl, l.beta)


def adjusted_delays(dev, A, B, start_a=0, start_b=0, offset=0, policy="equal"):
    """Exact delays of A and B when B joins `offset` after A (from kernels
    start_a, start_b), until either runs out of kernels.  policy: "equal",
    "priority" (B's kernels keep all their blocks) or "fcfs" (the kernel
    that was running first keeps all its blocks; equal when they started
    at the same time)."""
    now = Fraction(0)
    ka, kb = start_a, start_b
    done_a = done_b = Fraction(0)       # work completed on the current kernels
    # A alone until the offset
    offset = Fraction(offset)
    while ka < len(A) and now + (A[ka].d - done_a) <= offset:
        now += A[ka].d - done_a
        ka, done_a = ka + 1, Fraction(0)
    if ka < len(A):
        done_a += offset - now
    now = offset
    started_a = started_b = now          # start times of the running kernels
    if ka < len(A) and done_a > 0:
        started_a = now - done_a
    delay_a = delay_b = Fraction(0)
    while ka < len(A) and kb < len(B):
        if policy == "priority":
            first = "l"
        elif policy == "fcfs" and started_a != started_b:
            first = "k" if started_a < started_b else "l"
        else:
            first = None
        sa, sb = speeds(dev, A[ka], B[kb], first)
        # absolute completion times; a kernel at speed 0 does not complete
        ends = []
        if sa > 0:
            ends.append(now + (A[ka].d - done_a) / sa)
        if sb > 0:
            ends.append(now + (B[kb].d - done_b) / sb)
        nxt = min(ends)
        span = nxt - now
        delay_a += span - span * sa
        delay_b += span - span * sb
        done_a += span * sa
        done_b += span * sb
        now = nxt
        if done_a == A[ka].d:
            ka, done_a, started_a = ka + 1, Fraction(0), now
        if done_b == B[kb].d:
            kb, done_b, started_b = kb + 1, Fraction(0), now
    return delay_a, delay_b
