"""Limits of the HIP path against the oracle.

Covered here:
- pairs that fill the staging buffer exactly (q_i + q_j = RM_MAX_PAIR_KERNELS);
- an understated size hint on those pairs;
- the widest footprint packing, where a_k + a_l reaches 254;
- offset sets whose size is not a multiple of the workgroup's waves, with
  median and per-alignment output;
- a library wide enough that every persistent workgroup of the pair sweeps
  walks several rows."""
import numpy as np
import pytest

import oracle
from gpu_common import assert_rel, gpu_pair
from paper_2607_16784_amd import api
from paper_2607_16784_amd import workloads as W

pytestmark = pytest.mark.gpu

MAX_PAIR = 4096     # RM_MAX_PAIR_KERNELS


def sized_library(counts, seed, kernels="uniform", dev=W.A100):
    """Models with the given kernel counts (same draws as make_library)."""
    parts = [W.make_library(1, int(q), kernels, dev, seed=seed + m) for m, q in enumerate(counts)]
    offs = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    cat = {k: np.concatenate([p[k] for p in parts]) for k in
           ("grid", "threads", "regs", "smem", "duration")}
    cat["offsets"] = offs
    return cat


def test_pairs_at_the_staging_capacity():
    half = MAX_PAIR // 2
    L = sized_library([half, half, half - 1, 1], seed=900)
    for mode, K, red in ((0, 1, 0), (2, 3, 1)):
        ref = oracle.pair_matrix(W.A100, L, align_mode=mode, reduce_mode=red, num_offsets=K)
        for hint in (0, half):          # both size the buffer for q_i + q_j <= 4096
            got = gpu_pair(W.A100, L, align_mode=mode, reduce_mode=red, num_offsets=K,
                           max_kernels_per_model=hint)
            assert got["status"] == ref["status"]
            assert_rel(got["delay"], ref["delay"], what=f"delay mode {mode} hint {hint}")
            assert_rel(got["slowdown"], ref["slowdown"], what=f"slowdown mode {mode}")
        # one kernel short of the buffer: the full pairs are swept from
        # memory, with the same values and no status bit
        got = gpu_pair(W.A100, L, align_mode=mode, reduce_mode=red, num_offsets=K,
                       max_kernels_per_model=half - 1)
        q = np.diff(L["offsets"])
        too_long = q[:, None] + q[None, :] > 2 * (half - 1)
        assert too_long.any()
        assert got["status"] == ref["status"]
        assert_rel(got["delay"], ref["delay"], what=f"delay mode {mode}, pairs from memory")
        assert_rel(got["slowdown"], ref["slowdown"], what=f"slowdown mode {mode}, from memory")


def test_widest_footprint_packing():
    # W = 127 warps per SM (the packing limit) and 32-thread blocks: up to 127
    # blocks of one warp each, so a_k + a_l runs up to 254
    dev = dict(num_sm=4, max_threads_per_sm=127 * 32, max_blocks_per_sm=127,
               regs_per_sm=65536, smem_per_sm=160 * 1024, warp_size=32)
    rng = np.random.default_rng(31)
    n = 5 * 80
    L = {"offsets": np.arange(0, n + 1, 80, dtype=np.int64),
         "grid": rng.integers(1, 2000, n).astype(np.int32),
         "threads": rng.choice(np.array([32, 64, 96], np.int32), n),
         "regs": rng.integers(0, 16, n).astype(np.int32),
         "smem": np.where(rng.random(n) < 0.5, 0, rng.integers(0, 4096, n)).astype(np.int32),
         "duration": rng.lognormal(np.log(10.0), 1.0, n)}
    occ = oracle.occupancy(dev, L["grid"], L["threads"], L["regs"], L["smem"])
    assert occ["active_warps"].max() == 127
    for mode, K in ((0, 1), (2, 4)):
        ref = oracle.pair_matrix(dev, L, align_mode=mode, num_offsets=K)
        got = gpu_pair(dev, L, align_mode=mode, num_offsets=K)
        assert_rel(got["delay"], ref["delay"], what=f"delay mode {mode}")
        assert_rel(got["slowdown"], ref["slowdown"], what=f"slowdown mode {mode}")


@pytest.mark.parametrize("K,red", [(1, 0), (7, 0), (7, 1), (66, 0)])
def test_offsets_counts_and_per_alignment(K, red):
    rng = np.random.default_rng(40 + K)
    counts = rng.integers(0, 90, 9)
    counts[3] = 0                          # an empty model among them
    L = sized_library(counts, seed=70 + K, kernels="cnn")
    ref = oracle.pair_matrix(W.A100, L, align_mode=2, reduce_mode=red, num_offsets=K,
                             per_alignment=True)
    got = gpu_pair(W.A100, L, align_mode=2, reduce_mode=red, num_offsets=K, per_alignment=True)
    N = len(counts)
    assert_rel(got["per_alignment"].reshape(N, N, K), ref["per_alignment"], what="per offset")
    assert_rel(got["delay"], ref["delay"], what="delay")
    assert_rel(got["slowdown"], ref["slowdown"], what="slowdown")


def test_wide_library_many_rows_per_workgroup():
    L = W.make_library(300, (1, 60), "decode", W.A100, seed=301)
    ref = oracle.pair_matrix(W.A100, L)
    got = gpu_pair(W.A100, L, max_kernels_per_model=60)
    assert_rel(got["delay"], ref["delay"], what="FIRST delay")
    ref = oracle.pair_matrix(W.A100, L, align_mode=2, reduce_mode=1, num_offsets=2)
    got = gpu_pair(W.A100, L, align_mode=2, reduce_mode=1, num_offsets=2,
                   max_kernels_per_model=60)
    assert_rel(got["delay"], ref["delay"], what="OFFSETS delay")
