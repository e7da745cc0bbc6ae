"""The x-packed and head-major KV transforms' index maps, emulated on the CPU (no GPU).

tests/cpp/xpacked_emu.cpp runs one wave of the dummy-task kernel's x-packed
transform over the kernel's own index maps (mma_xpacked.h): it checks that every
global access stays inside the piece, every LDS access inside the wave's tile,
and that every destination byte is written exactly once; the result is compared
here with the oracle (oracle.kv.piece_to_block / block_to_piece). The tile
capacities are the runtime's (the larger of 16 KiB and one head's tile in each
staging order) and the smallest one that fits a head.
"""
import ctypes
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import kv as okv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
XP = okv.LAYOUT_XPACKED


@pytest.fixture(scope="module")
def emu(tmp_path_factory):
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("no C++ compiler")
    out = str(tmp_path_factory.mktemp("xp") / "libxpemu.so")
    # The emulator checks every access itself before making it (no sanitizer runtime in
    # a library loaded into python).
    cmd = [cxx, "-std=c++17", "-O1", "-g", "-shared", "-fPIC", "-Wall",
           f"-I{os.path.join(ROOT, 'paper_2512_16056_amd', 'csrc')}",
           os.path.join(ROOT, "tests", "cpp", "xpacked_emu.cpp"), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    lib = ctypes.CDLL(out)
    f = lib.emu_xpacked
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int] + [ctypes.c_uint32] * 5
    h = lib.emu_hnd
    h.restype = ctypes.c_int
    h.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int] + [ctypes.c_uint32] * 3
    f.hnd = h
    return f


def _caps(B, H, D, E):
    R = D * E
    need = max(B * (R + 16), (R // 16) * (B * 16 + 16), (R // E) * (B * E + 16))
    return sorted({need, max(need, 16 * 1024), 36 * 1024} - {c for c in (36 * 1024,) if c < need})


SHAPES = [(16, 8, 128, 2), (16, 8, 64, 2), (16, 1, 128, 2), (32, 8, 128, 1), (16, 4, 64, 4), (8, 3, 16, 2),
          (2, 5, 8, 8), (16, 2, 32, 1), (4, 8, 16, 4), (64, 2, 128, 1)]


@pytest.mark.parametrize("shape", SHAPES)
def test_xpacked_index_maps_match_oracle(emu, shape):
    B, H, D, E = shape
    r = np.random.default_rng(sum(shape))
    piece = np.ascontiguousarray(r.integers(0, 256, B * H * D * E, dtype=np.uint8))
    for cap in _caps(B, H, D, E):
        for k in (0, 1):
            want = okv.piece_to_block(piece, k, XP, (B, H, D, E))
            got = np.zeros_like(piece)
            rc = emu(piece.ctypes.data, got.ctypes.data, 1, k, B, H, D * E, E, cap)
            assert rc == 0, (shape, cap, k, "to_block", rc)
            assert np.array_equal(got, want), (shape, cap, k, "to_block")
            back = np.zeros_like(piece)
            rc = emu(want.ctypes.data, back.ctypes.data, 0, k, B, H, D * E, E, cap)
            assert rc == 0, (shape, cap, k, "from_block", rc)
            assert np.array_equal(back, piece), (shape, cap, k, "from_block")


def test_emulator_catches_a_wrong_map(emu):
    # a tile too small for one head makes the maps step outside it: the emulator reports it
    B, H, D, E = 16, 2, 128, 2
    piece = np.zeros(B * H * D * E, np.uint8)
    got = np.zeros_like(piece)
    assert emu(piece.ctypes.data, got.ctypes.data, 1, 1, B, H, D * E, E, 1024) != 0


HND_SHAPES = [(16, 8, 128, 2), (16, 8, 64, 2), (16, 1, 128, 2), (1, 8, 128, 2), (32, 8, 128, 1), (8, 3, 16, 2),
              (2, 5, 8, 8), (64, 2, 128, 1), (3, 7, 16, 4)]


@pytest.mark.parametrize("shape", HND_SHAPES)
def test_hnd_index_map_matches_oracle(emu, shape):
    """The head-major map: every access inside the piece, every byte written once, and the
    result equal to the oracle's, in both directions."""
    B, H, D, E = shape
    r = np.random.default_rng(sum(shape) + 1)
    piece = np.ascontiguousarray(r.integers(0, 256, B * H * D * E, dtype=np.uint8))
    blk = np.zeros_like(piece)
    assert emu.hnd(piece.ctypes.data, blk.ctypes.data, 1, B, H, D * E) == 0
    assert np.array_equal(blk, okv.piece_to_block(piece, 0, okv.LAYOUT_HND, (B, H, D, E)))
    back = np.zeros_like(piece)
    assert emu.hnd(blk.ctypes.data, back.ctypes.data, 0, B, H, D * E) == 0
    assert np.array_equal(back, piece)
