"""Seeded synthetic kernel-trace libraries and arrival streams.

This module only draws inputs; it holds none of the predictor's arithmetic and
is the one piece of code shared by the HIP path and the CPU oracle's tests.

A *library* is a dict of numpy arrays describing the kernels of N models laid
out back to back (structure of arrays):

  offsets   int64[N+1]  kernels of model m are offsets[m] .. offsets[m+1]-1
  grid      int32[K]    thread blocks in the launch grid
  threads   int32[K]    threads per block
  regs      int32[K]    registers per thread
  smem      int32[K]    shared memory per block, bytes
  duration  float64[K]  isolated kernel duration, microseconds

The paper's own traces (TorchVision models profiled on A100 and Jetson AGX
Xavier) and its Twitter arrival trace are not available; these seeded draws
stand in for them with the shapes listed in CONFIGS.  The only constraint
applied is launchability: a block never asks for more registers than one SM
holds (registers/thread x threads/block <= registers per SM); offending
(threads, registers) draws are redrawn.
"""
from __future__ import annotations

import numpy as np

# Device descriptors: an A100-class GPU (108 SMs, 2048 threads, 32 blocks,
# 64 Ki registers, 164 KiB shared memory per SM) and a Jetson-Xavier-class
# edge GPU (16 SMs, 1536 threads, 16 blocks, 64 Ki registers, 100 KiB).
A100 = dict(num_sm=108, max_threads_per_sm=2048, max_blocks_per_sm=32,
            regs_per_sm=65536, smem_per_sm=164 * 1024, warp_size=32)
EDGE = dict(num_sm=16, max_threads_per_sm=1536, max_blocks_per_sm=16,
            regs_per_sm=65536, smem_per_sm=100 * 1024, warp_size=32)
# MI355X (gfx950): 256 compute units, each holding 2048 threads (32
# wavefronts of 64), 32 workgroups, 131072 32-bit VGPR lanes (4 SIMDs x 512
# VGPRs x 64 lanes) and 160 KiB of LDS -- the limits the ROCm 7.2 runtime
# reports for the device.  (The ROCm 7.0 runtime that ships with PyTorch
# reports 65536 registers and 2 workgroups per CU for gfx950, which is why
# the descriptor is a constant here and not a run-time query.)
MI355X = dict(num_sm=256, max_threads_per_sm=2048, max_blocks_per_sm=32,
              regs_per_sm=131072, smem_per_sm=160 * 1024, warp_size=64)

THREAD_CHOICES = np.array([64, 128, 256, 512, 1024], np.int32)

# Per-kernel distributions.
KERNELS = {
    # uniform launch shapes, durations lognormal around 40 us
    "uniform": dict(grid=("uniform", 1, 4096), threads=THREAD_CHOICES,
                    regs=(16, 255), smem=(0, 48 * 1024), mu_us=40.0, sigma=1.0),
    # CNN-like: 70% of kernels launch >= 256 blocks, durations around 60 us
    "cnn": dict(grid=("cnn", 0.7), threads=THREAD_CHOICES,
                regs=(16, 255), smem=(0, 48 * 1024), mu_us=60.0, sigma=1.0),
    # decode-like: many small kernels, durations around 8 us
    "decode": dict(grid=("uniform", 1, 256), threads=np.array([128, 256], np.int32),
                   regs=(32, 128), smem=(0, 48 * 1024), mu_us=8.0, sigma=0.8),
    # gfx950-shaped launches: workgroups of 64..1024 lanes, VGPRs per lane up
    # to the 512 of the unified register file, LDS up to 64 KiB per
    # workgroup, grids up to 8192 workgroups, durations around 20 us
    "gfx950": dict(grid=("uniform", 1, 8192), threads=THREAD_CHOICES,
                   regs=(16, 512), smem=(0, 64 * 1024), mu_us=20.0, sigma=1.0),
}

# The five workloads.  'q' is either a fixed kernel count or an inclusive
# uniform range.  Alignment/reduction names follow the C interface.
CONFIGS = {
    "single_pair": dict(name="single-pair-2x60", n_models=2, q=60, kernels="uniform",
                        device=A100, seed=0, align="conflict_starts", reduce="median"),
    "cnn_64": dict(name="pair-matrix-64x150-500-cnn", n_models=64, q=(150, 500),
                   kernels="cnn", device=A100, seed=1, align="first", reduce="median"),
    "placement_128": dict(name="placement-128x200-800-1000arrivals", n_models=128,
                          q=(200, 800), kernels="uniform", device=A100, seed=2,
                          align="first", reduce="median", arrivals=1000, devices=16,
                          capacity=4, lam=0.5),
    "decode_256": dict(name="pair-matrix-256x2000-decode", n_models=256, q=2000,
                       kernels="decode", device=A100, seed=3, align="first",
                       reduce="median"),
    "edge_128": dict(name="phase-sweep-edge-128x1000-64offsets", n_models=128, q=1000,
                     kernels="uniform", device=EDGE, seed=4, align="offsets", reduce="max",
                     num_offsets=64),
    # the predictor targeting MI355X itself: gfx950-shaped kernel launches
    # against the gfx950 descriptor
    "gfx950": dict(name="pair-matrix-128x200-800-gfx950", n_models=128, q=(200, 800),
                   kernels="gfx950", device=MI355X, seed=5, align="first", reduce="median"),
}


def _draw_grid(rng, spec, n):
    if spec[0] == "uniform":
        return rng.integers(spec[1], spec[2] + 1, size=n)
    big = rng.random(n) < spec[1]
    g_big = rng.integers(256, 4096 + 1, size=n)
    g_small = rng.integers(1, 255 + 1, size=n)
    return np.where(big, g_big, g_small)


def _draw_model(rng, q, spec, device):
    grid = _draw_grid(rng, spec["grid"], q)
    threads = rng.choice(spec["threads"], size=q)
    regs = rng.integers(spec["regs"][0], spec["regs"][1] + 1, size=q)
    smem = rng.integers(spec["smem"][0], spec["smem"][1] + 1, size=q)
    dur = rng.lognormal(mean=np.log(spec["mu_us"]), sigma=spec["sigma"], size=q)
    # launchability: redraw (threads, regs) where one block exceeds the
    # register file of an SM
    while True:
        bad = np.nonzero(regs.astype(np.int64) * threads > device["regs_per_sm"])[0]
        if bad.size == 0:
            break
        threads[bad] = rng.choice(spec["threads"], size=bad.size)
        regs[bad] = rng.integers(spec["regs"][0], spec["regs"][1] + 1, size=bad.size)
    return grid, threads, regs, smem, dur


def make_library(n_models, q, kernels="uniform", device=A100, seed=0):
    """Draw a library of n_models traces; q is an int or an inclusive range."""
    rng = np.random.Generator(np.random.PCG64(seed))
    spec = KERNELS[kernels]
    parts = []
    counts = []
    for _ in range(n_models):
        qm = int(q) if np.isscalar(q) else int(rng.integers(q[0], q[1] + 1))
        counts.append(qm)
        parts.append(_draw_model(rng, qm, spec, device))
    offsets = np.zeros(n_models + 1, np.int64)
    offsets[1:] = np.cumsum(counts)

    def cat(i, dt):
        if not parts:
            return np.zeros(0, dt)
        return np.ascontiguousarray(np.concatenate([p[i] for p in parts]).astype(dt))

    return dict(offsets=offsets, grid=cat(0, np.int32), threads=cat(1, np.int32),
                regs=cat(2, np.int32), smem=cat(3, np.int32), duration=cat(4, np.float64))


def arrival_stream(n_arrivals, n_models, seed, departures=False, dwell=(16, 64)):
    """Arrival events (model ids, uniform) and optional departures.

    Without departures the stream is n_arrivals model ids.  With departures
    every arrival a (at time a) also leaves at time a + U{dwell} + 0.5; events
    are ordered by time and a departure is encoded as -1 - (event index of its
    arrival).  Departures later than the last arrival are dropped.  The
    departure of an arrival that was deferred is a no-op for the placer.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    models = rng.integers(0, n_models, size=n_arrivals).astype(np.int32)
    if not departures:
        return models
    stay = rng.integers(dwell[0], dwell[1] + 1, size=n_arrivals)
    timeline = [(float(a), 0, a) for a in range(n_arrivals)]
    timeline += [(a + float(stay[a]) + 0.5, 1, a) for a in range(n_arrivals)
                 if a + stay[a] + 0.5 < n_arrivals - 1]
    timeline.sort()
    index_of_arrival = {}
    events = []
    for _, kind, a in timeline:
        if kind == 0:
            index_of_arrival[a] = len(events)
            events.append(int(models[a]))
        else:
            events.append(-1 - index_of_arrival[a])
    return np.array(events, np.int32)


def config_library(cfg_id):
    cfg = CONFIGS[cfg_id]
    return make_library(cfg["n_models"], cfg["q"], cfg["kernels"], cfg["device"], cfg["seed"])


def config_events(cfg_id, departures=False, n_models=None):
    cfg = CONFIGS["placement_128" if cfg_id is None else cfg_id]
    n = cfg["n_models"] if n_models is None else n_models
    return arrival_stream(cfg.get("arrivals", 1000), n, seed=1000 + cfg["seed"],
                          departures=departures)


def start_draws(n_models, n_samples, seed):
    """Uniform 64-bit words for sampled start pairs: n_samples per unordered
    pair {a <= b} of n_models, pairs in row-major order (the layout both the
    C interface and the oracle read); shape (N(N+1)/2, n_samples)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    n_pairs = n_models * (n_models + 1) // 2
    return rng.integers(0, np.iinfo(np.uint64).max, size=(n_pairs, n_samples),
                        dtype=np.uint64, endpoint=True)


def sample_pairs(n_models, n_samples, seed):
    """Ordered pairs (i, j) for spot checks: the diagonal corners plus draws."""
    rng = np.random.Generator(np.random.PCG64(seed))
    fixed = [(0, 0), (0, n_models - 1), (n_models - 1, 0), (n_models - 1, n_models - 1)]
    draws = rng.integers(0, n_models, size=(n_samples, 2))
    pairs = np.array(fixed + [tuple(x) for x in draws], np.int32)
    return pairs
