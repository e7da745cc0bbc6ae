"""Host-side checks of the C ABI (no GPU needed): symbol exports, one HIP runtime
in the process, the planner and table validation against the oracle."""
import itertools
import os
import re

import numpy as np
import pytest

import workloads as W
from oracle import kv as okv
from oracle import plan as oplan

mma = pytest.importorskip("paper_2512_16056_amd")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "mma.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:mma_status_t|const char\*)\s+(mma_\w+)\s*\(", src, flags=re.M)))


def test_every_declared_symbol_is_exported():
    names = _declared_functions()
    assert len(names) >= 20
    for n in names:
        assert hasattr(mma.lib, n), n
        assert n in mma._SIGNATURES, f"binding lacks {n}"


def test_single_hip_runtime_in_process():
    maps = open("/proc/self/maps").read()
    hips = {line.split()[-1] for line in maps.splitlines() if "libamdhip64" in line}
    assert len(hips) == 1, hips


def test_status_strings_and_defaults():
    assert mma.mma_status_str(0) == "MMA_OK"
    assert mma.mma_status_str(-3) == "MMA_ERR_NOT_PINNED"
    c = mma.mma_config_default()
    assert c.chunk_bytes == 2 << 20 and c.queue_depth == 2 and c.cu_sub_bytes == 64 << 10
    assert c.small_bytes == 64 << 10 and c.cu_workgroups > 0 and c.watchdog_ms > 0
    assert c.control == mma.MMA_CONTROL_HOST  # the engine thread drives transfers unless asked otherwise
    assert c.engine_nap_us == 50  # and naps between rounds while every path has work queued


def test_calls_before_init_fail_cleanly():
    with pytest.raises(mma.MMAError) as e:
        mma.mma_memcpy_async(0, 0, 16, mma.MMA_H2D, 0)
    assert e.value.name == "MMA_ERR_NOT_INITIALIZED"
    with pytest.raises(mma.MMAError):
        mma.mma_get_stats()


@pytest.mark.skipif(os.path.exists("/dev/kfd") and os.access("/dev/kfd", os.R_OK), reason="GPU present")
def test_init_without_gpu_reports_error():
    with pytest.raises(mma.MMAError) as e:
        mma.mma_init(0)
    assert e.value.name == "MMA_ERR_INVALID_ARG"


def _as_oracle_list(entries):
    return [(i, o, b, bool(f & mma.MMA_TASK_CU_ONLY)) for i, o, b, f in entries]


@pytest.mark.parametrize("chunk,fallback,small", [(16, 32, 8), (7, 7, 1), (64, 200, 64), (4096, 8192, 1000)])
def test_plan_list_matches_oracle(chunk, fallback, small):
    r = np.random.default_rng(chunk)
    for _ in range(30):
        sizes = [int(x) for x in r.integers(0, 600, r.integers(1, 12))]
        got = _as_oracle_list(mma.mma_plan_list(sizes, chunk, fallback, small))
        assert got == oplan.plan_list(sizes, chunk, fallback, small)


def test_plan_workload_counts_match_oracle():
    M, K = W.MiB, W.KiB
    sizes = W.weight_tensor_bytes()
    for chunk in (2 * M, 256 * K, 5 * 1000 * 1000):
        got = mma.mma_plan_list(sizes, chunk, 2 * chunk, 64 * K)
        want = oplan.plan_list(sizes, chunk, 2 * chunk, 64 * K)
        assert _as_oracle_list(got) == want
    s = W.KV64K
    for chunk in (2 * M, 256 * K, 100 * K, 16 * K):
        got = mma.mma_plan_kv(4096, s.pieces_per_block, s.piece_bytes, chunk)
        assert [(i, o, b) for i, o, b, _ in got] == oplan.plan_kv(4096, s.pieces_per_block, s.piece_bytes, chunk)
        assert oplan.kv_covers_exactly_once([(i, o, b) for i, o, b, _ in got], 4096, s.pieces_per_block)


def test_plan_linear_covers_exactly_once():
    for n in list(range(0, 70)) + [4095, 4096, 4097, 1 << 20, (1 << 20) + 13]:
        for chunk in (16, 48, 4096):
            got = mma.mma_plan_list([n], chunk, 2 * chunk, 0)
            assert (n == 0 and got == []) or oplan.covers_exactly_once([(o, b) for _, o, b, _ in got], n)


def test_plan_limits():
    """Plans too large for memory fail at once with MMA_ERR_NO_MEMORY (a count computed before any
    item is stored), and a tensor whose last chunk ends at 2^64 - 1 is split without wrapping."""
    for call in (lambda: mma.mma_plan_list([1 << 60], 1, 2, 1),
                 lambda: mma.mma_plan_kv(1 << 62, 64, 1, 1)):
        with pytest.raises(mma.MMAError) as e:
            call()
        assert e.value.name == "MMA_ERR_NO_MEMORY"
    top = (1 << 64) - 1
    assert mma.mma_plan_list([top], 1 << 63, 2, 1) == [(0, 0, 1 << 63, 0), (0, 1 << 63, top - (1 << 63), 0)]
    assert mma.mma_status_str(-11) == "MMA_ERR_INTERNAL" and mma.mma_status_str(-8) == "MMA_ERR_NO_MEMORY"


def test_validate_tables_matches_oracle():
    r = np.random.default_rng(4)
    for _ in range(300):
        n = int(r.integers(0, 8))
        sc, dc = int(r.integers(1, 8)), int(r.integers(1, 8))
        src = r.integers(-1, sc + 1, n)
        dst = r.integers(-1, dc + 1, n)
        assert mma.mma_validate_kv_tables(src, sc, dst, dc) == okv.validate_tables(src, sc, dst, dc)
    for perm in itertools.permutations(range(4)):
        assert mma.mma_validate_kv_tables([0, 1, 2, 3], 4, perm, 4)
    # short tables against large destination counts (the sorted check) and long ones (the bitmap)
    for _ in range(200):
        dc = int(r.choice([1000, 100_000, 5_000_000]))
        n = int(r.integers(2, 40)) if r.random() < 0.7 else int(r.integers(dc // 64, dc // 64 + 50))
        dst = r.choice(dc, n, replace=False) if dc <= 100_000 else r.permutation(np.unique(r.integers(0, dc, 2 * n)))[:n]
        n = len(dst)
        if r.random() < 0.5:
            dst[int(r.integers(1, n))] = dst[int(r.integers(0, n))]  # a duplicate (or, rarely, the same slot)
        if r.random() < 0.1:
            dst[int(r.integers(0, n))] = dc  # out of range
        src = r.integers(0, 8, n)
        assert mma.mma_validate_kv_tables(src, 8, dst, dc) == okv.validate_tables(src, 8, dst, dc), (dc, n)


def test_kv_layout_sizes():
    """The sizes a KV layout implies, and the rejection of layouts whose sizes wrap 64 bits (the KV
    calls apply the same check before any range check)."""
    def sizes(*f):
        return mma.mma_kv_layout_sizes(mma.kv_layout(*f))

    # the 64k-token workload: 16 tokens x 8 heads x 128 x bf16 pieces, 32 layers, 4096 slots, 4352 GPU blocks
    assert sizes(32, 16, 8, 128, 2, 4352, 4096) == {"piece": 32768, "slot": 2 << 20, "pool": 8 << 30,
                                                    "layer": 285212672}
    for s in (W.small_kv_shape(), W.KVShape(layers=3, block_tokens=1, kv_heads=1, head_dim=5, elem_bytes=2,
                                            gpu_num_blocks=50, host_num_slots=40, n_blocks=37)):
        got = sizes(s.layers, s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes, s.gpu_num_blocks,
                    s.host_num_slots)
        assert got == {"piece": s.piece_bytes, "slot": s.slot_bytes, "pool": s.slot_bytes * s.host_num_slots,
                       "layer": s.layer_bytes}
    # a 4 GiB piece is the largest accepted
    assert sizes(1, 1 << 16, 1 << 16, 1, 1, 1, 1) == {"piece": 1 << 32, "slot": 1 << 33, "pool": 1 << 33,
                                                       "layer": 1 << 33}
    # 256 layers of 4 GiB pieces: a 2 TiB slot; 2^23 - 1 slots fit 64 bits, 2^23 wrap to 0
    assert sizes(256, 1 << 16, 1 << 16, 1, 1, 1, (1 << 23) - 1)["pool"] == (1 << 64) - (1 << 41)
    # a layer of 2^31 - 1 blocks of two 4 GiB pieces fits, 2^31 blocks wrap to 0
    assert sizes(1, 1 << 16, 1 << 16, 1, 1, (1 << 31) - 1, 1)["layer"] == (1 << 64) - (1 << 33)
    assert sizes(256, 1, 1, 1, 1, 1, 1)["slot"] == 512
    bad = [(256, 1 << 16, 1 << 16, 1, 1, 1, 1 << 23),       # pool size wraps to 0
           (1, 1 << 16, 1 << 16, 1, 1, 1 << 31, 1),          # layer size wraps to 0
           (1, 1 << 16, 1 << 16, 1 << 16, 1 << 16, 1, 1),    # piece wraps to 0
           (1, 1 << 16, (1 << 16) + 1, 1, 1, 1, 1),          # piece above 4 GiB
           (1, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 16, 1, 1),  # piece product beyond 64 bits
           (257, 1, 1, 1, 1, 1, 1)]                          # more layers than a call takes
    bad += [tuple(0 if k == z else 1 for k in range(7)) for z in range(7)]  # each field 0 in turn
    for f in bad:
        with pytest.raises(mma.MMAError) as e:
            sizes(*f)
        assert e.value.name == "MMA_ERR_INVALID_ARG", f
    out = (mma._U64 * 1)(7)
    assert mma.lib.mma_kv_layout_sizes(None, out, None, None, None) == mma.MMA_ERR_INVALID_ARG and out[0] == 7
    assert mma.lib.mma_kv_layout_sizes(mma.kv_layout(*bad[0]), out, None, None, None) == mma.MMA_ERR_INVALID_ARG
    assert out[0] == 7  # nothing written on rejection


def test_struct_layouts_match_header(tmp_path):
    """Every ctypes mirror has the size and field offsets that a C compiler gives the header's struct."""
    import ctypes
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    structs = ["mma_config_t", "mma_stats_t", "mma_copy_desc_t", "mma_kv_layout_t", "mma_trace_rec_t",
               "mma_plan_entry_t"]
    lines = ['#include "mma.h"', "#include <stdio.h>", "#include <stddef.h>", "int main(void) {"]
    want = []
    for sname in structs:
        cls = getattr(mma, sname)
        lines.append(f'  printf("%zu\\n", sizeof({sname}));')
        want.append(ctypes.sizeof(cls))
        for fname, _ in cls._fields_:
            lines.append(f'  printf("%zu\\n", offsetof({sname}, {fname}));')
            want.append(getattr(cls, fname).offset)
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run([cc, "-std=c99", f"-I{os.path.join(ROOT, 'include')}", str(src), "-o", str(exe)], check=True)
    got = [int(v) for v in subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split()]
    assert got == want


def test_interposer_exports_and_links_no_runtime():
    """libmma_interpose.so exports the three intercepted HIP copies and links neither the HIP
    runtime nor libmma.so (both are resolved inside the process at the first call)."""
    import subprocess
    lib = os.path.join(ROOT, "paper_2512_16056_amd", "libmma_interpose.so")
    if not os.path.exists(lib):
        pytest.skip("interposer not built")
    syms = subprocess.run(["nm", "-D", "--defined-only", lib], capture_output=True, text=True).stdout
    for name in ("hipMemcpyAsync", "hipMemcpy", "hipMemcpyWithStream"):
        assert re.search(rf"\bT {name}$", syms, flags=re.M), name
    needed = subprocess.run(["readelf", "-d", lib], capture_output=True, text=True).stdout
    assert "libamdhip64" not in needed and "libmma.so" not in needed


def test_layer_table_addresses_and_reuse():
    """The KV calls' layer array: one address per layer in order, and a table built once is
    passed through unchanged (no per-call rebuild)."""
    import ctypes
    import torch
    ts = [torch.empty(64, dtype=torch.uint8) for _ in range(5)]
    lt = mma.layer_table(ts)
    assert [lt[i] for i in range(5)] == [t.data_ptr() for t in ts]
    assert mma.layer_table(lt) is lt
    assert list(mma.layer_table([7, 0x1000])) == [7, 0x1000]
    assert isinstance(mma.layer_table([]), ctypes.Array)
