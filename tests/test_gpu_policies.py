"""The adjusted-occupancy simulation under the priority-based and
first-come-first-served scheduling policies (Sec. 3.2) on the GPU against
the CPU oracle, through the C ABI: bit-exact, as for equal partitioning
(every quotient is correctly rounded and the events run in the oracle's
order)."""
import sys

import numpy as np
import pytest
import torch

import oracle
from gpu_common import edge_row_pairs, gpu_pair
from paper_2607_16784_amd import api
from paper_2607_16784_amd import workloads as W
from test_gpu_adjusted import same

pytestmark = pytest.mark.gpu
ADJ = api.SWEEP_ADJUSTED
POLICIES = [(api.POLICY_PRIORITY, oracle.POLICY_PRIORITY, "priority"),
            (api.POLICY_FCFS, oracle.POLICY_FCFS, "fcfs")]
IDS = [p[2] for p in POLICIES]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("gp,op,name", POLICIES, ids=IDS)
@pytest.mark.parametrize("cid", ["single_pair", "cnn_64", "placement_128"])
def test_first_full_matrix(gp, op, name, cid):
    cfg = W.CONFIGS[cid]
    L = W.config_library(cid)
    say(f"ADJUSTED FIRST {name} full matrix, config {cid}")
    ref = oracle.pair_matrix(cfg["device"], L, sweep_mode=oracle.SWEEP_ADJUSTED, policy=op)
    got = gpu_pair(cfg["device"], L, sweep_mode=ADJ, policy=gp, per_alignment=True)
    same(got["delay"], ref["delay"], f"{name} delay")
    same(got["slowdown"], ref["slowdown"], f"{name} slowdown")
    same(got["per_alignment"], ref["delay"], f"{name} per_alignment")
    assert got["status"] == ref["status"]
    assert np.count_nonzero(ref["delay"]) > 0


@pytest.mark.parametrize("gp,op,name", POLICIES, ids=IDS)
def test_first_headline_size(gp, op, name):
    # the 256 x 2000 library: the full GPU matrix (under PRIORITY each pair
    # is run twice) against the oracle on every pair of rows 0, 1, N-2 and
    # N-1 and seeded draws
    cfg = W.CONFIGS["decode_256"]
    L = W.config_library("decode_256")
    say(f"ADJUSTED FIRST {name} 256 x 2000 full GPU matrix, oracle on edge rows and draws")
    got = gpu_pair(cfg["device"], L, sweep_mode=ADJ, policy=gp)
    pairs = edge_row_pairs(cfg["n_models"], 300, seed=77)
    ref = oracle.pair_entries(cfg["device"], L, pairs, sweep_mode=oracle.SWEEP_ADJUSTED,
                              policy=op)
    same(got["delay"][pairs[:, 0], pairs[:, 1]], ref["delay"], f"{name} delay")
    same(got["slowdown"][pairs[:, 0], pairs[:, 1]], ref["slowdown"], f"{name} slowdown")
    assert got["status"] == 0
    assert np.all(np.isfinite(got["delay"])) and np.all(got["delay"] >= 0.0)


@pytest.mark.parametrize("gp,op,name", POLICIES, ids=IDS)
@pytest.mark.parametrize("red,K", [("max", 13), ("median", 64)])
def test_offsets_full(gp, op, name, red, K):
    L = W.make_library(9, (1, 120), "uniform", W.EDGE, seed=41)
    say(f"ADJUSTED OFFSETS({K}) {name} {red}")
    ref = oracle.pair_matrix(W.EDGE, L, align_mode=oracle.ALIGN_OFFSETS,
                             reduce_mode=oracle.REDUCE_MAX if red == "max" else oracle.REDUCE_MEDIAN,
                             num_offsets=K, sweep_mode=oracle.SWEEP_ADJUSTED, policy=op,
                             per_alignment=True)
    got = gpu_pair(W.EDGE, L, align_mode=api.ALIGN_OFFSETS, reduce_mode=red, num_offsets=K,
                   sweep_mode=ADJ, policy=gp, per_alignment=True)
    same(got["per_alignment"], ref["per_alignment"], f"{name} per offset")
    same(got["delay"], ref["delay"], f"{name} delay")
    same(got["slowdown"], ref["slowdown"], f"{name} slowdown")


@pytest.mark.parametrize("gp,op,name", POLICIES, ids=IDS)
def test_offsets_edge_config_rows(gp, op, name):
    cfg = W.CONFIGS["edge_128"]
    L = W.config_library("edge_128")
    K = cfg["num_offsets"]
    N = cfg["n_models"]
    say(f"ADJUSTED OFFSETS edge config {name}, oracle on 64 pairs")
    got = gpu_pair(cfg["device"], L, align_mode=api.ALIGN_OFFSETS, reduce_mode="max",
                   num_offsets=K, sweep_mode=ADJ, policy=gp, per_alignment=True)
    pairs = W.sample_pairs(N, 60, seed=44)
    ref = oracle.pair_entries(cfg["device"], L, pairs, align_mode=oracle.ALIGN_OFFSETS,
                              reduce_mode=oracle.REDUCE_MAX, num_offsets=K,
                              sweep_mode=oracle.SWEEP_ADJUSTED, policy=op, per_alignment=True)
    pa = got["per_alignment"].reshape(N, N, K)
    same(pa[pairs[:, 0], pairs[:, 1]], ref["per_alignment"], f"{name} per offset")
    same(got["delay"][pairs[:, 0], pairs[:, 1]], ref["delay"], f"{name} delay")


@pytest.mark.parametrize("gp,op,name", POLICIES, ids=IDS)
@pytest.mark.parametrize("red", [0, 1])
def test_conflict_starts_single_pair(gp, op, name, red):
    cfg = W.CONFIGS["single_pair"]
    L = W.config_library("single_pair")
    ref = oracle.pair_matrix(cfg["device"], L, align_mode=oracle.ALIGN_CONFLICT_STARTS,
                             reduce_mode=red, sweep_mode=oracle.SWEEP_ADJUSTED, policy=op,
                             per_alignment=True)
    got = gpu_pair(cfg["device"], L, align_mode=api.ALIGN_CONFLICT_STARTS, reduce_mode=red,
                   sweep_mode=ADJ, policy=gp, per_alignment=True)
    same(got["per_alignment"], ref["per_alignment"], f"{name} per start pair")
    same(got["delay"], ref["delay"], f"{name} delay")


@pytest.mark.parametrize("gp,op,name", POLICIES, ids=IDS)
@pytest.mark.parametrize("K", [16, 100])
def test_sampled_starts(gp, op, name, K):
    cfg = W.CONFIGS["cnn_64"]
    L = W.config_library("cnn_64")
    N = cfg["n_models"]
    draws = W.start_draws(N, K, seed=1234 + K)
    say(f"ADJUSTED SAMPLED_STARTS({K}) {name}")
    ref = oracle.pair_matrix(cfg["device"], L, align_mode=oracle.ALIGN_SAMPLED_STARTS,
                             num_offsets=K, sweep_mode=oracle.SWEEP_ADJUSTED, policy=op,
                             start_draws=draws, per_alignment=True)
    got = gpu_pair(cfg["device"], L, align_mode=api.ALIGN_SAMPLED_STARTS, num_offsets=K,
                   sweep_mode=ADJ, policy=gp, per_alignment=True,
                   start_draws=torch.as_tensor(draws.reshape(-1)).cuda())
    same(got["per_alignment"], ref["per_alignment"], f"{name} per draw")
    same(got["delay"], ref["delay"], f"{name} delay")


def test_worked_sequence_against_one_long_kernel():
    # A = two kernels of 2 that each fill the SM's warps, B = one such kernel
    # of 8 (the oracle pins: equal 4 / 4, FCFS 8 / 2, priority 8 / 4)
    full = (432, 512, 16, 0)
    rows = [full + (2.0,), full + (2.0,), full + (8.0,)]
    L = dict(offsets=np.array([0, 2, 3], np.int64),
             grid=np.array([r[0] for r in rows], np.int32),
             threads=np.array([r[1] for r in rows], np.int32),
             regs=np.array([r[2] for r in rows], np.int32),
             smem=np.array([r[3] for r in rows], np.int32),
             duration=np.array([r[4] for r in rows], np.float64))
    for gp, want in ((api.POLICY_EQUAL, (4.0, 4.0)), (api.POLICY_FCFS, (8.0, 2.0)),
                     (api.POLICY_PRIORITY, (8.0, 4.0))):
        got = gpu_pair(W.A100, L, sweep_mode=ADJ, policy=gp)
        assert (got["delay"][0, 1], got["delay"][1, 0]) == want, gp


@pytest.mark.parametrize("gp,op,name", POLICIES, ids=IDS)
def test_ragged_and_bad_durations(gp, op, name):
    L = W.make_library(5, 30, "uniform", W.A100, seed=8)
    L["duration"][3] = np.nan
    L["duration"][40] = np.inf
    L["duration"][65] = 0.0
    L["duration"][100] = -2.0
    ref = oracle.pair_matrix(W.A100, L, sweep_mode=oracle.SWEEP_ADJUSTED, policy=op)
    got = gpu_pair(W.A100, L, sweep_mode=ADJ, policy=gp)
    same(got["delay"], ref["delay"], f"{name} delay, bad durations")
    assert got["status"] & api.ST_BAD_DURATION
    R = W.make_library(6, (0, 40), "decode", W.A100, seed=9)
    ref = oracle.pair_matrix(W.A100, R, sweep_mode=oracle.SWEEP_ADJUSTED, policy=op)
    got = gpu_pair(W.A100, R, sweep_mode=ADJ, policy=gp)
    same(got["delay"], ref["delay"], f"{name} delay, ragged")


def test_policy_needs_the_adjusted_simulation():
    L = W.make_library(3, 20, "uniform", W.A100, seed=1)
    # the options are rejected (workspace size 0, RM_EINVAL from the call)
    for kw in (dict(policy=api.POLICY_PRIORITY), dict(sweep_mode=ADJ, policy=7)):
        o = api.pair_opts(**kw)
        assert api.rm_pair_workspace_bytes(3, 60, o) == 0
        with pytest.raises(ValueError, match="invalid sizes or options"):
            gpu_pair(W.A100, L, **kw)
