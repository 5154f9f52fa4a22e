"""The seeded input generator: shapes, ranges and determinism of the five
workloads (it holds no arithmetic of the method)."""
import numpy as np
import pytest

from paper_2607_16784_amd import workloads as W


@pytest.mark.parametrize("cid", ["single_pair", "cnn_64", "placement_128", "edge_128"])
def test_library_shapes_and_ranges(cid):
    cfg = W.CONFIGS[cid]
    L = W.config_library(cid)
    off = L["offsets"]
    assert off.dtype == np.int64 and off.shape == (cfg["n_models"] + 1,) and off[0] == 0
    q = np.diff(off)
    if np.isscalar(cfg["q"]):
        assert np.all(q == cfg["q"])
    else:
        assert q.min() >= cfg["q"][0] and q.max() <= cfg["q"][1]
    n = int(off[-1])
    for k, dt in (("grid", np.int32), ("threads", np.int32), ("regs", np.int32),
                  ("smem", np.int32), ("duration", np.float64)):
        assert L[k].dtype == dt and L[k].shape == (n,)
    spec = W.KERNELS[cfg["kernels"]]
    assert set(np.unique(L["threads"])) <= set(spec["threads"].tolist())
    assert L["regs"].min() >= spec["regs"][0] and L["regs"].max() <= spec["regs"][1]
    assert L["smem"].min() >= 0 and L["smem"].max() <= 48 * 1024
    assert np.all(L["duration"] > 0)
    dev = cfg["device"]
    assert np.all(L["regs"].astype(np.int64) * L["threads"] <= dev["regs_per_sm"])


def test_headline_library_is_decode_like():
    L = W.config_library("decode_256")
    assert L["offsets"][-1] == 256 * 2000
    assert L["grid"].min() >= 1 and L["grid"].max() <= 256
    assert set(np.unique(L["threads"]).tolist()) == {128, 256}
    med = np.median(L["duration"])
    assert 6.5 < med < 9.5          # lognormal median e^mu = 8 us


def test_cnn_grid_mix():
    L = W.config_library("cnn_64")
    frac = np.mean(L["grid"] >= 256)
    assert 0.65 < frac < 0.75


def test_determinism():
    a, b = W.config_library("cnn_64"), W.config_library("cnn_64")
    for k in a:
        assert np.array_equal(a[k], b[k])
    assert np.array_equal(W.config_events("placement_128"), W.config_events("placement_128"))


def test_arrival_stream_with_departures():
    ev = W.arrival_stream(300, 50, seed=5, departures=True)
    arrivals = ev[ev >= 0]
    assert arrivals.shape[0] == 300 and arrivals.max() < 50
    seen = set()
    for e, v in enumerate(ev):
        if v < 0:
            idx = -1 - int(v)
            assert idx < e and ev[idx] >= 0 and idx not in seen
            seen.add(idx)
