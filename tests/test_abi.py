"""The C-ABI library loads and exports every entry point include/roomie.h
declares (no compute calls: this runs without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "roomie.h")
LIB = os.path.join(ROOT, "paper_2607_16784_amd", "librm.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(rm_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2607_16784_amd import build
        build.build()
    return ctypes.CDLL(LIB)


def test_header_declares_the_four_calls_and_helpers():
    names = declared_functions()
    for want in ("rm_occupancy", "rm_pair_slowdown_matrix", "rm_aggregate_greedy", "rm_place",
                 "rm_pair_workspace_bytes", "rm_status_string"):
        assert want in names


def test_library_exports_every_declared_symbol(lib):
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_host_only_entry_points(lib):
    lib.rm_status_string.restype = ctypes.c_char_p
    assert lib.rm_status_string(0) == b"ok"
    assert b"invalid" in lib.rm_status_string(1)
    assert lib.rm_status_string(99) == b"unknown status code"

    class Opts(ctypes.Structure):   # rm_pair_opts, field for field
        _fields_ = [("align_mode", ctypes.c_int32), ("reduce_mode", ctypes.c_int32),
                    ("num_offsets", ctypes.c_int32), ("max_kernels_per_model", ctypes.c_int32),
                    ("b", ctypes.c_void_p), ("e", ctypes.c_void_p), ("sweep", ctypes.c_int32),
                    ("draws", ctypes.c_void_p), ("policy", ctypes.c_int32)]

    f = lib.rm_pair_workspace_bytes
    f.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.POINTER(Opts)]
    f.restype = ctypes.c_size_t
    first = Opts(0, 0, 1, 0, None, None)
    up = lambda v: (v + 255) // 256 * 256  # noqa: E731
    assert f(256, 512000, ctypes.byref(first)) == up(512000 * 16) + up(256 * 8) + up(256 * 16)
    starts = Opts(1, 0, 1, 0, None, None)
    assert f(2, 120, ctypes.byref(starts)) >= 120 * 16 + 2 * 24 + 120 * 120 * 8
    assert f(0, 10, ctypes.byref(first)) == 0                    # no models
    assert f(2, 10, ctypes.byref(Opts(7, 0, 1, 0, None, None))) == 0   # bad mode
    assert f(2, 10, ctypes.byref(Opts(2, 1, 0, 0, None, None))) == 0   # K = 0
    assert f(2, 10, ctypes.byref(Opts(0, 0, 1, 0, None, None, 3))) == 0   # bad sweep mode
    # a scheduling policy needs the adjusted-occupancy simulation
    assert f(2, 10, ctypes.byref(Opts(0, 0, 1, 0, None, None, 0, None, 1))) == 0
    assert f(2, 10, ctypes.byref(Opts(0, 0, 1, 0, None, None, 2, None, 3))) == 0
    assert f(2, 10, ctypes.byref(Opts(0, 0, 1, 0, None, None, 2, None, 2))) > 0
    # the adjusted-occupancy simulation adds 32 B per kernel, and for OFFSETS
    # 8 B per ordered pair and offset
    adj = Opts(0, 0, 1, 0, None, None, 2)
    assert f(256, 512000, ctypes.byref(adj)) == f(256, 512000, ctypes.byref(first)) + up(512000 * 32)
    adj_off = Opts(2, 1, 64, 0, None, None, 2)
    base_off = Opts(2, 1, 64, 0, None, None, 0)
    assert (f(128, 128000, ctypes.byref(adj_off)) ==
            f(128, 128000, ctypes.byref(base_off)) + up(128000 * 32) + up(128 * 128 * 64 * 8))


def test_argument_checks_need_no_gpu(lib):
    class Dev(ctypes.Structure):
        _fields_ = [(n, ctypes.c_int32) for n in ("a", "b", "c", "d", "e", "f")]

    lib.rm_occupancy.restype = ctypes.c_int
    bad = Dev(108, 2048, 32, 65536, 167936, 0)       # warp size 0
    assert lib.rm_occupancy(ctypes.byref(bad), ctypes.c_int64(4), *([None] * 11)) == 1
    good = Dev(108, 2048, 32, 65536, 167936, 32)
    assert lib.rm_occupancy(ctypes.byref(good), ctypes.c_int64(0), *([None] * 11)) == 0
    assert lib.rm_occupancy(ctypes.byref(good), ctypes.c_int64(4), *([None] * 11)) == 1
    lib.rm_place.restype = ctypes.c_int
    lib.rm_place.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                             ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                             ctypes.c_int32, ctypes.c_void_p, ctypes.c_double, ctypes.c_int32,
                             ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    nul = None
    assert lib.rm_place(4, nul, nul, nul, 65, 4, nul, nul, 0, nul, 0.5, 0, nul, nul, nul, nul) == 3
    assert lib.rm_place(4, nul, nul, nul, 4, 9, nul, nul, 0, nul, 0.5, 0, nul, nul, nul, nul) == 3
    assert lib.rm_place(4, nul, nul, nul, 4, 4, nul, nul, 0, nul, float("nan"), 0, nul, nul,
                        nul, nul) == 1


def _gfx950_code_objects(path):
    """The gfx950 code objects bundled into the library's .hip_fatbin
    section (one offload bundle per compiled source)."""
    import struct
    import subprocess
    import tempfile
    objcopy = "/opt/rocm/llvm/bin/llvm-objcopy"
    if not os.path.exists(objcopy):
        pytest.skip("llvm-objcopy not available")
    with tempfile.TemporaryDirectory() as d:
        fat = os.path.join(d, "fatbin")
        subprocess.run([objcopy, "--dump-section=.hip_fatbin=" + fat, path, os.devnull],
                       check=True, capture_output=True)
        data = open(fat, "rb").read()
    magic = b"__CLANG_OFFLOAD_BUNDLE__"
    out, pos = [], 0
    while True:
        at = data.find(magic, pos)
        if at < 0:
            return out
        (count,) = struct.unpack_from("<Q", data, at + len(magic))
        off = at + len(magic) + 8
        for _ in range(count):
            o, size, tlen = struct.unpack_from("<QQQ", data, off)
            off += 24
            triple = data[off:off + tlen].decode()
            off += tlen
            if "gfx950" in triple:
                out.append(data[at + o:at + o + size])
        pos = at + 1


def _static_lds_per_kernel(code_objects):
    """{kernel symbol: group_segment_fixed_size} from the code objects'
    AMDGPU metadata notes."""
    import subprocess
    import tempfile
    readelf = "/opt/rocm/llvm/bin/llvm-readelf"
    if not os.path.exists(readelf):
        pytest.skip("llvm-readelf not available")
    sizes = {}
    with tempfile.TemporaryDirectory() as d:
        for n, co in enumerate(code_objects):
            f = os.path.join(d, f"co{n}.elf")
            open(f, "wb").write(co)
            notes = subprocess.run([readelf, "--notes", f], check=True, capture_output=True,
                                   text=True).stdout
            for entry in re.split(r"\n\s+- \.", notes):
                name = re.search(r"\.name:\s+(\S+)", entry)
                lds = re.search(r"group_segment_fixed_size:\s+(\d+)", entry)
                if name and lds and not name.group(1).endswith(".kd"):
                    sizes[name.group(1)] = int(lds.group(1))
    return sizes


def test_byte_addressed_sweeps_declare_no_static_lds(lib):
    # The FIRST, OFFSETS and sampled sweep kernels address LDS by byte
    # addresses from 0, which needs their dynamic allocation to start at 0,
    # i.e. no static LDS.  rm_pair_slowdown_matrix checks the same property
    # at run time (hipFuncGetAttributes) and returns RM_EUNSUPPORTED without
    # it; here it is read from the built code object.
    # FIRST has one kernel per tile shape (rows, columns, waves per pair).
    sizes = _static_lds_per_kernel(_gfx950_code_objects(LIB))
    families = ("sweep_first_kernel", "sweep_offsets_kernel", "sweep_sampled_kernel")
    found = {k: v for k, v in sizes.items() if any(s in k for s in families)}
    for fam in families:
        assert any(fam in k for k in found), (fam, sorted(sizes))
    assert sum("sweep_first_kernel" in k for k in found) == 6, sorted(found)
    assert all(v == 0 for v in found.values()), found
