"""SAMPLED_STARTS through the C ABI against the CPU oracle on the same seeded
draws: per-draw delays (NaN pattern exact, values within 1e-6 relative),
median and maximum over C_ij, slowdowns, for the temporal sweep and the
Sec. 3.2 adjusted-occupancy simulation (bit-exact), on full matrices, at
the 256 x 2000 size on sampled pairs, and at the edges (K at the wave and
workgroup boundaries, empty, one-kernel and 2000-kernel models -- a
4000-kernel pair nearly fills the staging buffer --, a pair too long for
it)."""
import sys

import numpy as np
import pytest
import torch

import oracle
from gpu_common import assert_rel, edge_row_pairs, gpu_pair
from paper_2607_16784_amd import api
from paper_2607_16784_amd import workloads as W

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_both(dev, L, K, seed, reduce_mode=0, sweep_mode=0, draws=None, **kw):
    N = len(L["offsets"]) - 1
    if draws is None:
        draws = W.start_draws(N, K, seed)
    ref = oracle.pair_matrix(dev, L, align_mode=oracle.ALIGN_SAMPLED_STARTS, num_offsets=K,
                             reduce_mode=reduce_mode, sweep_mode=sweep_mode, start_draws=draws,
                             per_alignment=True)
    got = gpu_pair(dev, L, align_mode=api.ALIGN_SAMPLED_STARTS, num_offsets=K,
                   reduce_mode=reduce_mode, sweep_mode=sweep_mode,
                   start_draws=torch.as_tensor(draws.reshape(-1)).cuda(), per_alignment=True,
                   **kw)
    return ref, got


def check(ref, got, exact=False, what=""):
    N = ref["delay"].shape[0]
    pa_g = got["per_alignment"].reshape(ref["per_alignment"].shape)
    if exact:
        assert np.array_equal(pa_g, ref["per_alignment"], equal_nan=True), what
        assert np.array_equal(got["delay"], ref["delay"]), what
        assert np.array_equal(got["slowdown"], ref["slowdown"]), what
        return 0.0
    assert_rel(pa_g, ref["per_alignment"], what=f"{what} per_alignment")
    e = assert_rel(got["delay"], ref["delay"], what=f"{what} delay")
    assert_rel(got["slowdown"], ref["slowdown"], what=f"{what} slowdown")
    assert got["delay"].shape == (N, N)
    return e


@pytest.mark.parametrize("cid,K", [("single_pair", 64), ("cnn_64", 16), ("placement_128", 8)])
@pytest.mark.parametrize("red", [0, 1])
def test_sampled_full_matrix(cid, K, red):
    cfg = W.CONFIGS[cid]
    L = W.config_library(cid)
    say("SAMPLED_STARTS full matrix config", cid, "K", K, "reduce", red)
    ref, got = run_both(cfg["device"], L, K, seed=100 + cfg["seed"], reduce_mode=red)
    e = check(ref, got, what=f"config {cid}")
    assert np.array_equal(got["iso_time"], ref["iso_time"])
    assert got["status"] == ref["status"]
    members = np.count_nonzero(~np.isnan(ref["per_alignment"]))
    say(f"  max rel err {e:.2e}, {members} members of {ref['per_alignment'].size} draws")
    assert members > 0


@pytest.mark.parametrize("K", [1, 2, 63, 64, 65, 100, 1024])
def test_sampled_draw_counts(K):
    # K <= 64: rank selection in one wave; K > 64: sort by the workgroup
    L = W.make_library(6, (20, 120), "uniform", W.A100, seed=31)
    say("SAMPLED_STARTS K", K)
    for red in (0, 1):
        ref, got = run_both(W.A100, L, K, seed=K, reduce_mode=red)
        check(ref, got, what=f"K={K} reduce={red}")


def test_sampled_hint_sizes_staging():
    L = W.config_library("cnn_64")
    q = np.diff(L["offsets"])
    say("SAMPLED_STARTS with max_kernels_per_model")
    ref, got = run_both(W.A100, L, 8, seed=4, max_kernels_per_model=int(q.max()))
    check(ref, got, what="hint")


def test_sampled_matches_enumerated_conflict_starts():
    # q^2 draws naming every start pair: the GPU's sampled matrix equals the
    # oracle's CONFLICT_STARTS matrix
    q, N = 7, 4
    L = W.make_library(N, q, "uniform", W.A100, seed=8)
    word = [-(-s * (1 << 32) // q) for s in range(q)]
    one = np.array([(word[a] << 32) | word[b] for a in range(q) for b in range(q)], np.uint64)
    draws = np.tile(one, (N * (N + 1) // 2, 1))
    say("SAMPLED_STARTS enumerating every start pair")
    for red in (0, 1):
        _, got = run_both(W.A100, L, q * q, seed=0, reduce_mode=red, draws=draws)
        c = oracle.pair_matrix(W.A100, L, align_mode=oracle.ALIGN_CONFLICT_STARTS,
                               reduce_mode=red)
        assert_rel(got["delay"], c["delay"], what=f"vs CONFLICT_STARTS reduce={red}")


def test_sampled_headline_size_sampled_pairs():
    cfg = W.CONFIGS["decode_256"]
    L = W.config_library("decode_256")
    N, K = cfg["n_models"], 64
    draws = W.start_draws(N, K, seed=303)
    say("SAMPLED_STARTS 256 x 2000, K = 64, sampled pairs")
    got = gpu_pair(cfg["device"], L, align_mode=api.ALIGN_SAMPLED_STARTS, num_offsets=K,
                   max_kernels_per_model=2000, per_alignment=True,
                   start_draws=torch.as_tensor(draws.reshape(-1)).cuda())
    pairs = edge_row_pairs(N, 512, seed=9)
    ref = oracle.pair_entries(cfg["device"], L, pairs, align_mode=oracle.ALIGN_SAMPLED_STARTS,
                              num_offsets=K, start_draws=draws, per_alignment=True)
    pa = got["per_alignment"].reshape(N, N, K)
    assert_rel(got["delay"][pairs[:, 0], pairs[:, 1]], ref["delay"], what="delay")
    assert_rel(got["slowdown"][pairs[:, 0], pairs[:, 1]], ref["slowdown"], what="slowdown")
    assert_rel(pa[pairs[:, 0], pairs[:, 1]], ref["per_alignment"], what="per_alignment")
    # properties at every pair: C_ji is C_ij transposed (same NaN pattern),
    # delays are finite and non-negative, an empty set gives 0
    assert np.array_equal(np.isnan(pa), np.isnan(pa.transpose(1, 0, 2)))
    assert np.all(got["delay"] >= 0) and np.all(np.isfinite(got["delay"]))
    empty = np.isnan(pa).all(axis=2)
    assert np.all(got["delay"][empty] == 0)
    assert got["status"] == 0


def test_sampled_ragged_and_degenerate_models():
    rng = np.random.default_rng(12)
    parts = [W.make_library(1, q, "uniform", W.A100, seed=int(rng.integers(1 << 30)))
             for q in (0, 1, 2, 2000, 57, 1)]
    L = {k: np.concatenate([p[k] for p in parts]) for k in ("grid", "threads", "regs", "smem",
                                                          "duration")}
    L["offsets"] = np.concatenate([[0], np.cumsum([len(p["grid"]) for p in parts])]).astype(
        np.int64)
    say("SAMPLED_STARTS ragged library with empty, one-kernel and 2000-kernel models")
    for red in (0, 1):
        ref, got = run_both(W.A100, L, 40, seed=77, reduce_mode=red)
        check(ref, got, what=f"ragged reduce={red}")
        assert got["status"] == ref["status"]


def test_sampled_pair_too_long_is_swept_from_memory():
    # a hint of 100 kernels sizes the buffer for q_i + q_j <= 200; pairs with
    # the 300-kernel model do not fit and are swept from memory
    parts = [W.make_library(1, q, "uniform", W.A100, seed=s) for q, s in ((50, 1), (300, 2),
                                                                        (80, 3))]
    L = {k: np.concatenate([p[k] for p in parts]) for k in ("grid", "threads", "regs", "smem",
                                                          "duration")}
    L["offsets"] = np.array([0, 50, 350, 430], np.int64)
    say("SAMPLED_STARTS pair too long for the staging buffer")
    for red in (0, 1):
        ref, got = run_both(W.A100, L, 16, seed=5, max_kernels_per_model=100, reduce_mode=red)
        assert got["status"] == ref["status"]
        check(ref, got, what=f"pairs from memory, reduce={red}")


@pytest.mark.parametrize("cid,K", [("single_pair", 64), ("cnn_64", 8), ("edge_128", 4)])
def test_sampled_adjusted_simulation_bit_exact(cid, K):
    cfg = W.CONFIGS[cid]
    L = W.config_library(cid)
    if cid == "edge_128":   # edge descriptor, first 24 models
        n = 24
        L = {k: (v[:L["offsets"][n]] if k != "offsets" else v[:n + 1]) for k, v in L.items()}
    say("SAMPLED_STARTS adjusted simulation config", cid, "K", K)
    for red in (0, 1):
        ref, got = run_both(cfg["device"], L, K, seed=200 + cfg["seed"], reduce_mode=red,
                            sweep_mode=api.SWEEP_ADJUSTED)
        check(ref, got, exact=True, what=f"adjusted config {cid} reduce={red}")


def test_sampled_argument_errors():
    L = api.library_to_device(W.make_library(3, 10, "uniform", W.A100, seed=1))
    args = (W.A100, L["offsets"], L["grid"], L["threads"], L["regs"], L["smem"], L["duration"])
    with pytest.raises(ValueError):
        api.rm_pair_slowdown_matrix(*args, align_mode=api.ALIGN_SAMPLED_STARTS, num_offsets=4)
    short = torch.zeros(5, dtype=torch.uint64, device="cuda")
    with pytest.raises(ValueError):
        api.rm_pair_slowdown_matrix(*args, align_mode=api.ALIGN_SAMPLED_STARTS, num_offsets=4,
                                    start_draws=short)
    many = torch.zeros(6 * 2000, dtype=torch.uint64, device="cuda")
    with pytest.raises((ValueError, RuntimeError)):
        api.rm_pair_slowdown_matrix(*args, align_mode=api.ALIGN_SAMPLED_STARTS,
                                    num_offsets=2000, start_draws=many)
