"""Row-tile staging of the FIRST pair sweep against the oracle.

The sweep takes up to four row models and one column model per item and
loads the next item's column into registers while the current one is
swept.  Covered here: model counts that leave the last row tile short,
rows longer than the staging cap (swept from memory while the other rows of
the tile stay staged), pairs of one row that fit beside pairs of another
that do not, and many tile boundaries per workgroup.  Columns too long for
the registers (copied straight into LDS after the item) are covered by the
long-trace tests (a 3500-kernel hint stages one row and 3500-kernel
columns)."""
import numpy as np
import pytest

import oracle
from gpu_common import assert_rel, gpu_pair
from paper_2607_16784_amd import api
from paper_2607_16784_amd import workloads as W
from test_gpu_parity_limits import sized_library

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seed", range(3))
def test_unequal_rows_and_columns(seed):
    rng = np.random.default_rng(1000 + seed)
    n = 61                      # 31 row tiles, 961 items: several per workgroup
    counts = rng.integers(1, 300, size=n)
    counts[rng.choice(n, 4, replace=False)] = rng.integers(700, 800, size=4)
    L = sized_library(counts, seed=2000 + 100 * seed)
    ref = oracle.pair_matrix(W.A100, L)
    # cap 2 * 200: the long models fit no pair and are never staged, about
    # half of the other pairs do not fit either, and two consecutive columns
    # beside two rows often exceed the 2 * 400 slots
    hint = 200
    got = gpu_pair(W.A100, L, max_kernels_per_model=hint)
    too_long = counts[:, None] + counts[None, :] > 2 * hint
    assert too_long.any() and (~too_long).any()
    # the pairs the buffer cannot hold are swept from memory: same values,
    # no status bit
    assert got["status"] == ref["status"]
    assert_rel(got["delay"], ref["delay"], what="delay, some pairs from memory")
    assert_rel(got["slowdown"], ref["slowdown"], what="slowdown, some pairs from memory")
    # with the true bound every pair fits
    got = gpu_pair(W.A100, L, max_kernels_per_model=int(counts.max()), per_alignment=True)
    assert got["status"] == ref["status"]
    assert_rel(got["delay"], ref["delay"], what="delay")
    assert_rel(got["slowdown"], ref["slowdown"], what="slowdown")
    assert_rel(got["per_alignment"], ref["delay"], what="per_alignment")


def test_many_short_models():
    # 700 models: 350 row tiles and 122,850 items, about 480 per workgroup,
    # crossing many tile boundaries (each restages the rows)
    L = W.make_library(700, (1, 24), "decode", W.A100, seed=4242)
    ref = oracle.pair_matrix(W.A100, L)
    got = gpu_pair(W.A100, L, max_kernels_per_model=24)
    assert got["status"] == ref["status"]
    assert_rel(got["delay"], ref["delay"], what="delay")
    assert_rel(got["slowdown"], ref["slowdown"], what="slowdown")


@pytest.mark.parametrize("mode,K,red", [("first", 1, "median"), ("offsets", 4, "max"),
                                        ("sampled_starts", 8, "median")])
def test_null_optional_outputs(mode, K, red):
    # slowdown, per-alignment output and status may be NULL: the delays are
    # unchanged and nothing else is written
    import torch
    L = W.make_library(9, (5, 120), "cnn", W.A100, seed=515)
    D = api.library_to_device(L)
    N = 9
    draws = None
    if mode == "sampled_starts":
        draws = torch.as_tensor(W.start_draws(N, K, seed=3).reshape(-1)).cuda()
    args = (W.A100, D["offsets"], D["grid"], D["threads"], D["regs"], D["smem"], D["duration"])
    kw = dict(align_mode=mode, reduce_mode=red, num_offsets=K, start_draws=draws)
    full = api.rm_pair_slowdown_matrix(*args, per_alignment=True, status=api.new_status(), **kw)
    out = {"delay": torch.empty(N * N, dtype=torch.float64, device="cuda"),
           "iso_time": torch.empty(N, dtype=torch.float64, device="cuda"),
           "kernel_count": torch.empty(N, dtype=torch.int32, device="cuda")}
    bare = api.rm_pair_slowdown_matrix(*args, out=out, status=None, **kw)
    torch.cuda.synchronize()
    assert torch.equal(bare["delay"], full["delay"])
    assert torch.equal(bare["iso_time"], full["iso_time"])


def test_split_window_kept_and_abandoned():
    """The merge-path split of a lane first tries a window around its split
    against the previous column of its group.  Equal 1500-kernel models whose
    durations alternate between two scales make consecutive columns of a group
    cross the row at very different places, so the window's checks fail and
    the full search runs; columns of one scale keep it.  Both against the
    oracle."""
    base = W.make_library(12, (1500, 1500), "decode", W.A100, seed=5150)
    L = {k: v.copy() for k, v in base.items()}
    off = L["offsets"]
    scale = np.ones(L["duration"].size)
    for m in range(12):
        if (m // 2) % 2 == 1:    # columns of one group alternate: j and j + 2
            scale[off[m]:off[m + 1]] = 3.0
    L["duration"] = L["duration"] * scale
    ref = oracle.pair_matrix(W.A100, L)
    for lib, what in ((L, "alternating scales"), (base, "one scale")):
        r = ref if lib is L else oracle.pair_matrix(W.A100, lib)
        got = gpu_pair(W.A100, lib, max_kernels_per_model=1500)
        assert got["status"] == r["status"]
        assert_rel(got["delay"], r["delay"], what=f"delay, {what}")
        assert_rel(got["slowdown"], r["slowdown"], what=f"slowdown, {what}")
