"""HIP path (through the C ABI) against the CPU oracle on the same seeded
inputs: occupancy bit-exact, delays/slowdowns within 1e-6 relative with
exact zeros, iso times bit-exact (same sequential sums)."""
import sys

import numpy as np
import pytest
import torch

import oracle
from gpu_common import assert_rel, edge_row_pairs, gpu_pair, to_np
from paper_2607_16784_amd import api
from paper_2607_16784_amd import workloads as W

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("cid", ["single_pair", "cnn_64", "placement_128", "decode_256", "edge_128"])
def test_occupancy_bit_exact(cid):
    cfg = W.CONFIGS[cid]
    L = W.config_library(cid)
    say("occupancy config", cid, L["grid"].shape)
    dev = cfg["device"]
    ref = oracle.occupancy(dev, L["grid"], L["threads"], L["regs"], L["smem"])
    T = api.library_to_device(L)
    st = api.new_status()
    out = api.rm_occupancy(dev, T["grid"], T["threads"], T["regs"], T["smem"], status=st)
    torch.cuda.synchronize()
    for k in ("blocks_per_sm", "resident_blocks", "active_warps", "limiter"):
        assert np.array_equal(to_np(out[k]), ref[k]), k
    assert np.array_equal(to_np(out["occupancy"]), ref["occupancy"])
    assert int(st.item()) == ref["status"]


def test_occupancy_edge_configurations():
    rng = np.random.default_rng(3)
    n = 5000
    g = rng.integers(-2, 5000, n).astype(np.int32)
    t = rng.choice([0, 1, 31, 32, 64, 100, 1024, 1056, 2048, 4096], n).astype(np.int32)
    r = rng.integers(-1, 300, n).astype(np.int32)
    s = rng.integers(-1, 200_000, n).astype(np.int32)
    for dev in (W.A100, W.EDGE):
        ref = oracle.occupancy(dev, g, t, r, s)
        st = api.new_status()
        tt = [torch.as_tensor(x).cuda() for x in (g, t, r, s)]
        out = api.rm_occupancy(dev, *tt, status=st)
        torch.cuda.synchronize()
        for k in ("blocks_per_sm", "resident_blocks", "active_warps", "limiter"):
            assert np.array_equal(to_np(out[k]), ref[k]), k
        assert np.array_equal(to_np(out["occupancy"]), ref["occupancy"])
        assert int(st.item()) == ref["status"]


@pytest.mark.parametrize("cid", ["single_pair", "cnn_64", "placement_128"])
def test_first_alignment_full_matrix(cid):
    cfg = W.CONFIGS[cid]
    L = W.config_library(cid)
    say("FIRST full matrix config", cid)
    ref = oracle.pair_matrix(cfg["device"], L, align_mode=oracle.ALIGN_FIRST)
    got = gpu_pair(cfg["device"], L, align_mode=api.ALIGN_FIRST, per_alignment=True)
    assert np.array_equal(got["kernel_count"], ref["kernel_count"])
    assert np.array_equal(got["iso_time"], ref["iso_time"])
    e1 = assert_rel(got["delay"], ref["delay"], what="delay")
    e2 = assert_rel(got["slowdown"], ref["slowdown"], what="slowdown")
    assert_rel(got["per_alignment"], ref["delay"], what="per_alignment")
    assert got["status"] == ref["status"]
    say(f"  max rel err delay {e1:.2e} slowdown {e2:.2e}")
    assert_self_pairs_consistent(got)


def assert_self_pairs_consistent(got):
    """A self pair's two directions are one value, written by two waves: its
    slowdown (gamma = 1) is its delay over its isolated time, bit for bit."""
    d = np.diag(got["delay"])
    assert np.array_equal(np.diag(got["slowdown"]), d / got["iso_time"])
    if "per_alignment" in got:
        assert np.array_equal(np.diag(got["per_alignment"].reshape(got["delay"].shape)), d)


def test_first_alignment_hint_sizes_staging():
    cfg = W.CONFIGS["cnn_64"]
    L = W.config_library("cnn_64")
    q = np.diff(L["offsets"])
    ref = oracle.pair_matrix(cfg["device"], L)
    got = gpu_pair(cfg["device"], L, max_kernels_per_model=int(q.max()))
    assert_rel(got["delay"], ref["delay"], what="delay with exact hint")
    # an understated bound: the pairs it cannot stage are swept from memory,
    # with the same values and no status bit
    small = int(np.sort(q)[len(q) // 2])
    got = gpu_pair(cfg["device"], L, max_kernels_per_model=small)
    too_long = (q[:, None] + q[None, :]) > 2 * small
    assert too_long.any()
    assert got["status"] == ref["status"]
    assert_rel(got["delay"], ref["delay"], what="delay, understated bound")
    assert_rel(got["slowdown"], ref["slowdown"], what="slowdown, understated bound")


def test_conflict_starts_single_pair():
    cfg = W.CONFIGS["single_pair"]
    L = W.config_library("single_pair")
    say("CONFLICT_STARTS config 0")
    ref = oracle.pair_matrix(cfg["device"], L, align_mode=oracle.ALIGN_CONFLICT_STARTS,
                             per_alignment=True)
    got = gpu_pair(cfg["device"], L, align_mode=api.ALIGN_CONFLICT_STARTS, per_alignment=True)
    nk = L["grid"].shape[0]
    assert_rel(got["per_alignment"].reshape(nk, nk), ref["per_alignment"], what="per alignment")
    assert_rel(got["delay"], ref["delay"], what="median delay")
    assert_rel(got["slowdown"], ref["slowdown"], what="slowdown")
    for red in ("max",):
        r2 = oracle.pair_matrix(cfg["device"], L, align_mode=1, reduce_mode=oracle.REDUCE_MAX)
        g2 = gpu_pair(cfg["device"], L, align_mode=api.ALIGN_CONFLICT_STARTS, reduce_mode=red)
        assert_rel(g2["delay"], r2["delay"], what="max delay")


@pytest.mark.parametrize("red", ["max", "median"])
def test_offsets_small_library_full(red):
    L = W.make_library(9, (1, 120), "uniform", W.EDGE, seed=41)
    K = 13
    ref = oracle.pair_matrix(W.EDGE, L, align_mode=oracle.ALIGN_OFFSETS,
                             reduce_mode=oracle.REDUCE_MAX if red == "max" else oracle.REDUCE_MEDIAN,
                             num_offsets=K, per_alignment=True)
    got = gpu_pair(W.EDGE, L, align_mode=api.ALIGN_OFFSETS, reduce_mode=red, num_offsets=K,
                   per_alignment=True)
    assert_rel(got["per_alignment"], ref["per_alignment"], what="per offset")
    assert_rel(got["delay"], ref["delay"], what="delay")
    assert_rel(got["slowdown"], ref["slowdown"], what="slowdown")


def test_offsets_edge_config_full():
    cfg = W.CONFIGS["edge_128"]
    L = W.config_library("edge_128")
    K = cfg["num_offsets"]
    N = cfg["n_models"]
    say("OFFSETS config 4 full GPU matrix against the full oracle matrix")
    got = gpu_pair(cfg["device"], L, align_mode=api.ALIGN_OFFSETS, reduce_mode="max",
                   num_offsets=K, max_kernels_per_model=1000, per_alignment=True)
    ref = oracle.pair_matrix(cfg["device"], L, align_mode=oracle.ALIGN_OFFSETS,
                             reduce_mode=oracle.REDUCE_MAX, num_offsets=K, per_alignment=True)
    pa = got["per_alignment"].reshape(N, N, K)
    assert_rel(pa, ref["per_alignment"].reshape(N, N, K), what="per offset")
    assert_rel(got["delay"], ref["delay"], what="worst-case delay")
    assert_rel(got["slowdown"], ref["slowdown"], what="slowdown")
    # worst case = max over the offsets at every pair
    assert np.array_equal(got["delay"], pa.max(axis=2))
    assert np.all(np.isfinite(got["delay"]))


def test_headline_config_rows_and_draws():
    cfg = W.CONFIGS["decode_256"]
    L = W.config_library("decode_256")
    say("FIRST config 3 (256 x 2000) full GPU matrix, oracle on edge rows and draws")
    got = gpu_pair(cfg["device"], L, max_kernels_per_model=2000)
    pairs = edge_row_pairs(cfg["n_models"], 600, seed=3)
    ref = oracle.pair_entries(cfg["device"], L, pairs)
    assert_rel(got["delay"][pairs[:, 0], pairs[:, 1]], ref["delay"], what="delay")
    assert_rel(got["slowdown"][pairs[:, 0], pairs[:, 1]], ref["slowdown"], what="slowdown")
    assert_self_pairs_consistent(got)
    # isolated times: bit-exact with the in-order sum of the durations
    off = L["offsets"]
    for m in range(cfg["n_models"]):
        t = 0.0
        for d in L["duration"][off[m]:off[m + 1]].tolist():
            t += d
        assert got["iso_time"][m] == t
    assert got["status"] == 0 and np.all(got["kernel_count"] == 2000)
