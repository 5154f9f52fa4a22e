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
