"""The allocation-free entry point rm_pair_slowdown_matrix_static (static
device scratch) against rm_pair_slowdown_matrix (caller workspace): the same
kernels, so the outputs must agree bit for bit.  Two calls in a row, the
second on a smaller input, for each alignment set and both sweep modes."""
import sys

import numpy as np
import pytest
import torch

from paper_2607_16784_amd import api
from paper_2607_16784_amd import workloads as W

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run(fn, dev, lib, **kw):
    L = api.library_to_device(lib)
    st = api.new_status()
    out = fn(dev, L["offsets"], L["grid"], L["threads"], L["regs"], L["smem"], L["duration"],
             status=st, **kw)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items() if k != "workspace"}
    res["status"] = int(st.item())
    return res


def same(a, b, what):
    for k in ("delay", "slowdown", "iso_time", "kernel_count", "per_alignment", "status"):
        if k in a or k in b:
            assert np.array_equal(a[k], b[k], equal_nan=k in ("delay", "slowdown",
                                                               "per_alignment")), f"{what}: {k}"


CASES = [
    ("first", dict(), ("decode_256", 2000), (24, (1, 400), "cnn")),
    ("offsets", dict(align_mode="offsets", reduce_mode="max", num_offsets=64),
     ("edge_128", 1000), (9, (1, 120), "uniform")),
    ("adjusted", dict(sweep_mode="adjusted"), ("cnn_64", 500), (7, (5, 90), "decode")),
]


@pytest.mark.parametrize("name,kw,big,small", CASES, ids=[c[0] for c in CASES])
def test_static_scratch_matches_workspace_entry(name, kw, big, small):
    cid, qmax = big
    cfg = W.CONFIGS[cid]
    lib_big = W.config_library(cid)
    lib_small = W.make_library(small[0], small[1], small[2], cfg["device"], seed=77)
    for lib, hint, what in ((lib_big, qmax, "large"), (lib_small, small[1][1], "smaller")):
        say(f"static scratch {name}: {what} input, {lib['offsets'].size - 1} models")
        a = run(api.rm_pair_slowdown_matrix_static, cfg["device"], lib,
                max_kernels_per_model=hint, per_alignment=True, **kw)
        b = run(api.rm_pair_slowdown_matrix, cfg["device"], lib,
                max_kernels_per_model=hint, per_alignment=True, **kw)
        same(a, b, f"{name} {what}")


def test_static_scratch_sampled_then_smaller():
    cfg = W.CONFIGS["cnn_64"]
    for N, seed in ((64, 1), (10, 2)):
        lib = W.config_library("cnn_64") if N == 64 else W.make_library(N, (3, 60), "cnn",
                                                                         cfg["device"], seed)
        draws = torch.as_tensor(W.start_draws(N, 32, seed=seed).reshape(-1)).cuda()
        say(f"static scratch sampled starts: {N} models")
        kw = dict(align_mode="sampled_starts", num_offsets=32, start_draws=draws,
                  per_alignment=True, max_kernels_per_model=500)
        a = run(api.rm_pair_slowdown_matrix_static, cfg["device"], lib, **kw)
        b = run(api.rm_pair_slowdown_matrix, cfg["device"], lib, **kw)
        same(a, b, f"sampled {N}")


def test_static_scratch_rejects_inputs_beyond_its_size():
    # CONFLICT_STARTS over 3000 kernels needs 8 * 3000^2 bytes > 64 MiB: the
    # call returns RM_ETOOLARGE on the host and enqueues nothing
    lib = W.make_library(2, 1500, "uniform", W.A100, seed=5)
    o = api.pair_opts(align_mode="conflict_starts")
    assert api.rm_pair_workspace_bytes(2, 3000, o) > api.RM_STATIC_SCRATCH_BYTES
    with pytest.raises(RuntimeError, match="code 5"):
        run(api.rm_pair_slowdown_matrix_static, W.A100, lib, align_mode="conflict_starts")
