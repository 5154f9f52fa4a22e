"""Edge cases of the HIP path against the oracle: empty and one-kernel
models, ties from equal integer durations, kernels that never or always
interfere, infeasible kernels, non-default streams, argument errors."""
import numpy as np
import pytest
import torch

import oracle
from gpu_common import assert_rel, gpu_pair
from paper_2607_16784_amd import api
from paper_2607_16784_amd import workloads as W
from test_oracle_sweep import BIG, TINY, lib_from, random_lib

pytestmark = pytest.mark.gpu


def both(lib, dev=W.A100, **kw):
    mode = kw.get("align_mode", 0)
    red = kw.get("reduce_mode", "median")
    ref = oracle.pair_matrix(dev, lib, align_mode=mode, reduce_mode=1 if red == "max" else 0,
                             num_offsets=kw.get("num_offsets", 1))
    got = gpu_pair(dev, lib, **kw)
    return ref, got


@pytest.mark.parametrize("mode,K", [(0, 1), (1, 1), (2, 5)])
def test_empty_and_single_kernel_models(mode, K):
    L = lib_from([[BIG + (2.0,)] * 3, [], [BIG + (1.5,)], [TINY + (4.0,)], [BIG + (0.5,)] * 2])
    ref, got = both(L, align_mode=mode, num_offsets=K)
    assert np.array_equal(got["kernel_count"], ref["kernel_count"])
    assert np.array_equal(got["iso_time"], ref["iso_time"])
    assert_rel(got["delay"], ref["delay"], what="delay")
    assert_rel(got["slowdown"], ref["slowdown"], what="slowdown")
    assert got["status"] == ref["status"] and got["status"] & api.ST_EMPTY_MODEL


@pytest.mark.parametrize("seed", range(3))
def test_integer_durations_with_ties(seed):
    rng = np.random.default_rng(500 + seed)
    L = random_lib(rng, 12, 60, integer=True)
    for mode, K in ((0, 1), (2, 7)):
        ref, got = both(L, align_mode=mode, num_offsets=K, reduce_mode="max")
        assert_rel(got["delay"], ref["delay"], what=f"delay mode {mode}")
    ref, got = both(L, align_mode=1)
    assert_rel(got["delay"], ref["delay"], what="starts delay")


def test_never_and_always_interfering():
    L = lib_from([[TINY + (3.0,)] * 40, [TINY + (1.25,)] * 70])
    ref, got = both(L)
    assert np.all(got["delay"] == 0) and np.all(ref["delay"] == 0)
    L = lib_from([[BIG + (3.0,)] * 40, [BIG + (1.25,)] * 70])
    ref, got = both(L)
    assert_rel(got["delay"], ref["delay"], what="all conflict")
    assert got["delay"][0, 1] + got["delay"][1, 0] == pytest.approx(min(120.0, 87.5))


def test_infeasible_kernels_do_not_interfere():
    rng = np.random.default_rng(7)
    L = random_lib(rng, 6, 40)
    L["regs"][::5] = 255
    L["threads"][::5] = 1024       # 255 * 1024 registers: no block fits
    ref, got = both(L)
    assert ref["status"] & oracle.ST_INFEASIBLE_KERNEL
    assert got["status"] == ref["status"]
    assert_rel(got["delay"], ref["delay"], what="delay")


def test_ragged_library_many_tiles():
    L = W.make_library(40, (1, 1500), "cnn", W.A100, seed=77)
    ref, got = both(L, max_kernels_per_model=1500)
    assert_rel(got["delay"], ref["delay"], what="delay")
    assert_rel(got["slowdown"], ref["slowdown"], what="slowdown")


def test_runs_on_a_side_stream():
    L = W.config_library("cnn_64")
    ref = oracle.pair_matrix(W.A100, L)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        got = gpu_pair(W.A100, L)
    assert_rel(got["delay"], ref["delay"], what="delay on side stream")


def test_argument_errors_raise():
    L = api.library_to_device(W.config_library("single_pair"))
    with pytest.raises(RuntimeError):
        api.rm_pair_slowdown_matrix(dict(W.A100, warp_size=0), L["offsets"], L["grid"],
                                    L["threads"], L["regs"], L["smem"], L["duration"])
    with pytest.raises(ValueError):
        api.rm_pair_slowdown_matrix(W.A100, L["offsets"], L["grid"].cpu(), L["threads"],
                                    L["regs"], L["smem"], L["duration"])
    with pytest.raises(ValueError):
        api.rm_pair_slowdown_matrix(W.A100, L["offsets"], L["grid"], L["threads"], L["regs"],
                                    L["smem"], L["duration"], align_mode=2, num_offsets=0)
