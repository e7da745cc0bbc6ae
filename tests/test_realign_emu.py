"""The CU path's copy of relatively misaligned ranges, emulated on the CPU (no GPU).

tests/cpp/realign_emu.cpp runs one wave of the dummy-task kernel's realigning copy
(aligned 16-byte source units shifted into aligned destination units in registers,
neighbouring units taken across lanes) with the kernel's batch shape, clamps and
predicates. It checks every load against the aligned units the source range
touches, every store against the destination range, exactly-once writes, and the
result against the source, at every relatively misaligned pair of offsets modulo 16.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def emu(tmp_path_factory):
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("no C++ compiler")
    out = str(tmp_path_factory.mktemp("realign") / "realign_emu")
    cmd = [cxx, "-std=c++17", "-O2", "-Wall", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           os.path.join(ROOT, "tests", "cpp", "realign_emu.cpp"), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return out


def test_realign_small_sizes(emu):
    # every size up to one batch and a bit: heads, tails, partial rows, the extra unit
    r = subprocess.run([emu, "1100", "1"], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("ok"), r.stdout


def test_realign_batch_boundaries(emu):
    # around one and several 16 KiB batches (the extra unit of a batch is the next batch's first)
    sizes = ["16383", "16384", "16385", "16399", "16400", "16415", "32768", "32783", "49153", "65536", "100013"]
    r = subprocess.run([emu, "0", "1", *sizes], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("ok"), r.stdout
