"""The predictor targeting MI355X itself: the gfx950 descriptor against the
device's reported limits, and the whole path -- occupancy, pair matrix
(temporal sweep, adjusted simulation, sampled start pairs), placement -- on
gfx950-shaped kernel launches against that descriptor, through the C ABI,
compared with the CPU oracle (occupancy, iso times and the adjusted
simulation bit-exact, temporal delays within 1e-6 relative)."""
import sys

import numpy as np
import pytest
import torch

import oracle
from gpu_common import assert_rel, gpu_pair, to_np
from paper_2607_16784_amd import api
from paper_2607_16784_amd import workloads as W

pytestmark = pytest.mark.gpu
CFG = W.CONFIGS["gfx950"]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def subset(L, n):
    return {k: (v[:L["offsets"][n]] if k != "offsets" else v[:n + 1]) for k, v in L.items()}


@pytest.fixture(scope="module")
def lib():
    return W.config_library("gfx950")


def test_descriptor_matches_the_device():
    # compute units, threads per CU and wavefront size as the runtime reports
    # them (registers and workgroups per CU differ between runtime versions)
    p = torch.cuda.get_device_properties(0)
    if not p.gcnArchName.startswith("gfx950"):
        pytest.skip(f"device is {p.gcnArchName}, not gfx950")
    assert p.multi_processor_count == W.MI355X["num_sm"]
    assert p.max_threads_per_multi_processor == W.MI355X["max_threads_per_sm"]
    assert p.warp_size == W.MI355X["warp_size"]


def test_occupancy_bit_exact(lib):
    say("gfx950 occupancy", lib["grid"].shape)
    ref = oracle.occupancy(W.MI355X, lib["grid"], lib["threads"], lib["regs"], lib["smem"])
    T = api.library_to_device(lib)
    st = api.new_status()
    out = api.rm_occupancy(W.MI355X, T["grid"], T["threads"], T["regs"], T["smem"], status=st)
    torch.cuda.synchronize()
    for k in ("blocks_per_sm", "resident_blocks", "active_warps", "limiter"):
        assert np.array_equal(to_np(out[k]), ref[k]), k
    assert np.array_equal(to_np(out["occupancy"]), ref["occupancy"])
    assert int(st.item()) == ref["status"]


def test_first_full_matrix(lib):
    say("gfx950 FIRST full matrix, 128 models")
    ref = oracle.pair_matrix(W.MI355X, lib)
    got = gpu_pair(W.MI355X, lib, per_alignment=True)
    assert np.array_equal(got["iso_time"], ref["iso_time"])
    assert_rel(got["delay"], ref["delay"], what="delay")
    assert_rel(got["slowdown"], ref["slowdown"], what="slowdown")
    assert np.count_nonzero(ref["delay"]) > 0
    assert got["status"] == ref["status"]


def test_adjusted_simulation_bit_exact(lib):
    L = subset(lib, 48)
    say("gfx950 adjusted simulation, 48 models")
    ref = oracle.pair_matrix(W.MI355X, L, sweep_mode=oracle.SWEEP_ADJUSTED)
    got = gpu_pair(W.MI355X, L, sweep_mode=api.SWEEP_ADJUSTED)
    assert np.array_equal(got["delay"], ref["delay"])
    assert np.array_equal(got["slowdown"], ref["slowdown"])


def test_sampled_start_pairs(lib):
    L = subset(lib, 32)
    K = 16
    draws = W.start_draws(32, K, seed=950)
    say("gfx950 sampled start pairs, 32 models, K = 16")
    ref = oracle.pair_matrix(W.MI355X, L, align_mode=oracle.ALIGN_SAMPLED_STARTS, num_offsets=K,
                             start_draws=draws, per_alignment=True)
    got = gpu_pair(W.MI355X, L, align_mode=api.ALIGN_SAMPLED_STARTS, num_offsets=K,
                   start_draws=torch.as_tensor(draws.reshape(-1)).cuda(), per_alignment=True)
    assert_rel(got["per_alignment"].reshape(ref["per_alignment"].shape), ref["per_alignment"],
               what="per_alignment")
    assert_rel(got["delay"], ref["delay"], what="delay")


def test_placement_from_the_same_delays(lib):
    say("gfx950 placement, 1000 arrivals onto 16 x 4")
    ref = oracle.pair_matrix(W.MI355X, lib)
    ev = W.arrival_stream(1000, 128, seed=1950, departures=True)
    want = oracle.place(ref["delay"], ref["iso_time"], ref["kernel_count"], 16, 4, ev, 0.5)
    D = torch.as_tensor(ref["delay"].reshape(-1)).cuda()
    got = api.rm_place(D, torch.as_tensor(ref["iso_time"]).cuda(),
                       torch.as_tensor(ref["kernel_count"]).cuda(), 16, 4,
                       torch.as_tensor(ev).cuda(), 0.5)
    torch.cuda.synchronize()
    assert np.array_equal(to_np(got["placed_device"])[:len(ev)], want["placed_device"])
    assert np.array_equal(to_np(got["placed_mu_mean"])[:len(ev)], want["placed_mu_mean"],
                          equal_nan=True)
    assert (want["placed_device"] >= 0).sum() > 64
