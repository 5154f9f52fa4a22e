"""Helpers shared by the GPU parity tests (HIP path vs CPU oracle)."""
import numpy as np
import torch

from paper_2607_16784_amd import api

REL = 1e-6      # slowdown / delay tolerance (fp64 accumulate, different sum order)


def to_np(t):
    return t.detach().cpu().numpy()


def assert_rel(gpu, ref, rel=REL, what=""):
    """Element-wise |g - o| <= rel * |o|, identical NaN pattern, exact zeros."""
    g = np.asarray(gpu, dtype=np.float64).reshape(-1)
    o = np.asarray(ref, dtype=np.float64).reshape(-1)
    assert g.shape == o.shape, what
    assert np.array_equal(np.isnan(g), np.isnan(o)), f"{what}: NaN pattern differs"
    zero = o == 0
    assert np.all(g[zero] == 0), f"{what}: oracle zero not exact on GPU"
    m = ~np.isnan(o) & ~zero
    err = np.abs(g[m] - o[m]) / np.abs(o[m])
    worst = float(err.max(initial=0.0))
    assert worst <= rel, f"{what}: max rel err {worst:.3e} > {rel}"
    return worst


def gpu_pair(dev, lib_np, **kw):
    L = api.library_to_device(lib_np)
    st = api.new_status()
    out = api.rm_pair_slowdown_matrix(dev, L["offsets"], L["grid"], L["threads"], L["regs"],
                                      L["smem"], L["duration"], status=st, **kw)
    torch.cuda.synchronize()
    N = L["offsets"].numel() - 1
    res = {k: to_np(v) for k, v in out.items() if k != "workspace"}
    res["delay"] = res["delay"].reshape(N, N)
    res["slowdown"] = res["slowdown"].reshape(N, N)
    res["status"] = int(st.item())
    return res


def edge_row_pairs(n_models, n_samples, seed):
    """Ordered pairs (i, j) for checks at full size: every pair with i or j in
    {0, 1, N-2, N-1} (the first and last row tiles of a row-tiled sweep and
    their mirrors) plus seeded draws, duplicates removed, sorted."""
    rows = sorted({0, 1, n_models - 2, n_models - 1} & set(range(n_models)))
    ext = {(r, c) for r in rows for c in range(n_models)}
    ext |= {(c, r) for r in rows for c in range(n_models)}
    rng = np.random.Generator(np.random.PCG64(seed))
    draws = rng.integers(0, n_models, size=(n_samples, 2))
    ext |= {(int(a), int(b)) for a, b in draws}
    return np.array(sorted(ext), np.int32)
