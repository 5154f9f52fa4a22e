"""Pairs longer than the LDS staging buffer (q_i + q_j > 4096 kernels) are
swept from the record table in memory: the same values as the oracle, for
every alignment set the temporal sweep supports, and no status bit.  The
library mixes 3000- and 3500-kernel models (pairs of 6000 to 7000 kernels)
with short models (pairs that are staged), so each kernel takes both paths
in one launch."""
import sys

import numpy as np
import pytest
import torch

import oracle
from gpu_common import assert_rel, gpu_pair
from paper_2607_16784_amd import api
from paper_2607_16784_amd import workloads as W
from test_gpu_parity_limits import sized_library

pytestmark = pytest.mark.gpu

COUNTS = [3000, 120, 3500, 1, 3000, 400]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def lib():
    return sized_library(COUNTS, seed=4400, kernels="decode")


def long_pairs():
    q = np.array(COUNTS)
    return q[:, None] + q[None, :] > 4096


def test_first_long_pairs(lib):
    say("FIRST with 3000/3500-kernel models")
    ref = oracle.pair_matrix(W.A100, lib, per_alignment=True)
    for hint in (0, 3500, 200):
        got = gpu_pair(W.A100, lib, max_kernels_per_model=hint, per_alignment=True)
        assert got["status"] == ref["status"] == 0
        assert long_pairs().any()
        assert_rel(got["delay"], ref["delay"], what=f"delay hint {hint}")
        assert_rel(got["slowdown"], ref["slowdown"], what=f"slowdown hint {hint}")
        assert_rel(got["per_alignment"], ref["delay"], what=f"per_alignment hint {hint}")
        assert np.all(got["delay"][long_pairs()] > 0)


@pytest.mark.parametrize("red,K", [(1, 8), (0, 9)])
def test_offsets_long_pairs(lib, red, K):
    say(f"OFFSETS({K}) reduce={red} with 3000/3500-kernel models")
    ref = oracle.pair_matrix(W.A100, lib, align_mode=oracle.ALIGN_OFFSETS, reduce_mode=red,
                             num_offsets=K, per_alignment=True)
    got = gpu_pair(W.A100, lib, align_mode=api.ALIGN_OFFSETS, reduce_mode=red, num_offsets=K,
                   per_alignment=True)
    N = len(COUNTS)
    assert got["status"] == ref["status"] == 0
    assert_rel(got["per_alignment"].reshape(N, N, K), ref["per_alignment"], what="per offset")
    assert_rel(got["delay"], ref["delay"], what="delay")
    assert_rel(got["slowdown"], ref["slowdown"], what="slowdown")


@pytest.mark.parametrize("red,K", [(0, 16), (1, 100)])
def test_sampled_starts_long_pairs(lib, red, K):
    N = len(COUNTS)
    draws = W.start_draws(N, K, seed=4500 + K)
    say(f"SAMPLED_STARTS({K}) reduce={red} with 3000/3500-kernel models")
    ref = oracle.pair_matrix(W.A100, lib, align_mode=oracle.ALIGN_SAMPLED_STARTS,
                             reduce_mode=red, num_offsets=K, start_draws=draws,
                             per_alignment=True)
    got = gpu_pair(W.A100, lib, align_mode=api.ALIGN_SAMPLED_STARTS, reduce_mode=red,
                   num_offsets=K, per_alignment=True,
                   start_draws=torch.as_tensor(draws.reshape(-1)).cuda())
    assert got["status"] == ref["status"] == 0
    assert_rel(got["per_alignment"].reshape(N, N, K), ref["per_alignment"], what="per draw")
    assert_rel(got["delay"], ref["delay"], what="delay")
    assert_rel(got["slowdown"], ref["slowdown"], what="slowdown")
