"""Host-side counts the bench reports next to its timings."""
import sys
import os

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


def lib_of(durations):
    offs = np.concatenate([[0], np.cumsum([len(d) for d in durations])]).astype(np.int64)
    return {"offsets": offs, "duration": np.concatenate([np.asarray(d, np.float64)
                                                         for d in durations])}


def test_window_segments_worked_example():
    # A = two kernels of 2, B = four kernels of 1: the A-B window [0, 4) has
    # boundaries {1, 2, 3, 4} (the shared 2 and 4 count once) -> 4 segments
    # per direction; A-A has 2, B-B has 4.
    lib = lib_of([[2.0, 2.0], [1.0, 1.0, 1.0, 1.0]])
    assert bench.window_segments(lib) == 2 + 4 + 2 * 4


def test_window_segments_stop_at_the_first_model_to_finish():
    # A ends at 3; B's boundaries after 3 lie outside the window
    lib = lib_of([[1.5, 1.5], [1.0, 1.0, 1.0, 1.0, 1.0]])
    # A-A: {1.5, 3}; B-B: {1..5}; A-B window (0, 3]: {1, 1.5, 2, 3} -> 4
    assert bench.window_segments(lib) == 2 + 5 + 2 * 4


def test_algorithmic_bytes_headline():
    q = np.full(256, 2000)
    assert bench.algorithmic_bytes(q) == 16.0 * 2 * 256 * 512000 + 8.0 * 256 * 256


def test_unordered_segments_count_each_pair_once():
    # same library as the worked example: A-A 2, B-B 4, A-B 4 (both
    # directions share the segments)
    lib = lib_of([[2.0, 2.0], [1.0, 1.0, 1.0, 1.0]])
    assert bench.unordered_segments(lib) == 2 + 4 + 4
    lib = lib_of([[1.5, 1.5], [1.0, 1.0, 1.0, 1.0, 1.0], [0.5, 2.5]])
    # ordered count = 2 x unordered - diagonal
    diag = 2 + 5 + 2
    assert bench.window_segments(lib) == 2 * bench.unordered_segments(lib) - diag


def test_roofline_constants():
    # VALU issue: 256 CUs x 4 SIMDs x 16 lanes per clock at 2.4 GHz, half the
    # published fp64 vector peak in flops (an FMA counts two)
    assert abs(bench.VALU_PEAK_TOPS - 78.6 / 2) < 0.05
    assert abs(bench.LDS_PEAK_GBS - 78643.2) < 1e-6
