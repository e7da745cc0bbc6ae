"""Both directions at once (Section 5.1.2, concurrent flows): while one direction moves, the other
pulls only from its duplex paths.

A 2 GiB host->device copy runs on stream A. On stream B, issued after it, a paged-KV offload
(copy-engine share through staging) and a device->host tensor list with one tensor below the
CU-only size. Every result is compared with the oracle. The trace shows which paths carried the
device->host transfers: under the default configuration only engines 2-5, plus the CU path for
the micro-tasks that only it may carry, while the host->device copy moved. Two streams can share
a hardware queue, and then B's work starts only after A's. So the test takes the first of a few
stream pairs that ran side by side, by the trace's timestamps.
"""
import time

import numpy as np
import pytest
import torch

import workloads as W
from oracle import copy as ocopy
from oracle import kv as okv

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2512_16056_amd as mma  # noqa: E402
from gpu_helpers import device_bytes, log, session, to_host  # noqa: E402

SHAPE = W.KVShape(layers=8, block_tokens=16, kv_heads=8, head_dim=128, elem_bytes=2,
                  gpu_num_blocks=1024, host_num_slots=1024, n_blocks=512)  # 512 KiB slots, 256 MiB offload
H2D_BYTES = 2 << 30
LIST_SIZES = [(24 << 20) + 5, 4096, 16 << 20]  # the 4 KiB tensor is below small_bytes: CU path only
ENGINES_2_5 = 0x3C


def _layout(s):
    return mma.kv_layout(s.layers, s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes, s.gpu_num_blocks,
                         s.host_num_slots)


def test_duplex_defaults_follow_path_masks():
    with session("both") as cfg:
        d2h = cfg.duplex_paths_d2h
        if d2h & ENGINES_2_5 != ENGINES_2_5:
            pytest.skip(f"engines 2-5 not available for device->host (duplex set {d2h:#x})")
        assert d2h == ENGINES_2_5, hex(d2h)
        assert cfg.duplex_paths_h2d == cfg.path_mask_h2d & 0xFFFF, (hex(cfg.duplex_paths_h2d), hex(cfg.path_mask_h2d))
    # an explicit device->host mask keeps its own engines (without the CU path)
    with session("both", path_mask_d2h=mma.MMA_PATH_CU | 0x3) as cfg:
        assert cfg.duplex_paths_d2h == 0x3, hex(cfg.duplex_paths_d2h)
    with session("cu") as cfg:  # no engine: the direction keeps its CU path
        assert cfg.duplex_paths_d2h == mma.MMA_PATH_CU and cfg.duplex_paths_h2d == mma.MMA_PATH_CU
    with session("both", duplex_paths_h2d=mma.MMA_DUPLEX_UNCHANGED,
                 duplex_paths_d2h=mma.MMA_DUPLEX_UNCHANGED) as cfg:
        assert cfg.duplex_paths_h2d == cfg.path_mask_h2d and cfg.duplex_paths_d2h == cfg.path_mask_d2h


def test_duplex_paths_while_both_directions_move():
    s = SHAPE
    plan = W.kv_offload_plan(s, cfg=4)
    r = np.random.default_rng(11)

    def seeded(n):
        return np.frombuffer(r.bytes(n), np.uint8)

    h2d_src = mma.PinnedBuffer(H2D_BYTES)
    h2d_src.array[:] = seeded(H2D_BYTES)
    pool = mma.PinnedBuffer(s.host_num_slots * s.slot_bytes)
    pool.array[:] = seeded(pool.nbytes)
    pool_before = pool.array.copy()
    layers = []
    for l in range(s.layers):
        t = device_bytes(s.layer_bytes)
        t.copy_(torch.from_numpy(seeded(s.layer_bytes).copy()))
        layers.append(t)
    views = [to_host(t).reshape(2, s.gpu_num_blocks, s.piece_bytes) for t in layers]
    lsrc = [device_bytes(n) for n in LIST_SIZES]
    for t in lsrc:
        t.copy_(torch.from_numpy(seeded(t.numel()).copy()))
    ldst = mma.PinnedBuffer(sum(LIST_SIZES) + 64)
    h2d_dst = device_bytes(H2D_BYTES, W.GPU_POISON)
    trace, ran_side_by_side = None, False
    for attempt in range(6):
        sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
        log(f"duplex attempt {attempt}")
        ldst.array[:] = 0x5A
        pool.array[:] = pool_before
        with session("both", cu_whole_bytes=1, cu_whole_bytes_d2h=1):
            mma.mma_trace_enable(True)
            mma.mma_memcpy_async(h2d_dst, h2d_src, H2D_BYTES, mma.MMA_H2D, sa)
            # the host->device engine thread marks its direction as moving within microseconds of
            # the start; submissions in that window would still prefill CU-path entries
            time.sleep(0.002)
            mma.mma_kv_offload(_layout(s), pool, layers, plan.src_blocks, plan.dest, sb)
            offs = np.cumsum([0] + LIST_SIZES[:-1])
            mma.mma_weights_load([(ldst.ptr + int(o), t, n) for o, t, n in zip(offs, lsrc, LIST_SIZES)], mma.MMA_D2H,
                                 sb)
            torch.cuda.synchronize()
            mma.mma_synchronize()
            stats = mma.mma_get_stats()
            trace = mma.mma_trace_read()
            mma.mma_trace_enable(False)
        assert stats["failed_transfers"] == 0
        h = [x for x in trace if x["dir"] == mma.MMA_H2D]
        d = [x for x in trace if x["dir"] == mma.MMA_D2H]
        assert len(h) == 1 and len(d) == 2, trace
        # the device->host transfers started after the host->device copy had started and ended
        # before it completed: the whole of them ran while it moved
        ran_side_by_side = all(h[0]["t_started_ns"] < x["t_started_ns"] and x["t_last_task_ns"] < h[0]["t_last_task_ns"]
                               for x in d)
        if ran_side_by_side:
            break
    if not ran_side_by_side:
        pytest.skip("no stream pair of six ran both directions side by side")
    # bytes: every transfer against the oracle
    got = to_host(h2d_dst)
    assert np.array_equal(got, ocopy.memcpy(np.full(H2D_BYTES, W.GPU_POISON, np.uint8), 0, h2d_src.array, 0,
                                            H2D_BYTES))
    want_pool = okv.kv_offload(pool_before.reshape(s.host_num_slots, -1), views, plan.src_blocks, plan.dest)
    assert np.array_equal(pool.array.reshape(s.host_num_slots, -1), want_pool)
    want = np.full(sum(LIST_SIZES) + 64, 0x5A, np.uint8)
    for o, t, n in zip(np.cumsum([0] + LIST_SIZES[:-1]), lsrc, LIST_SIZES):
        want = ocopy.memcpy(want, int(o), to_host(t), 0, n)
    assert np.array_equal(ldst.array, want)
    # paths: the device->host transfers ran on engines 2-5, and on the CU path only what only it may carry
    kv, lst = (d[0], d[1]) if d[0]["kind"] == 2 else (d[1], d[0])
    for x, name in ((kv, "kv offload"), (lst, "list")):
        pt = x["path_tasks"]
        log(f"{name}: tasks per path {[(i, v) for i, v in enumerate(pt) if v]}")
        assert pt[0] == 0 and pt[1] == 0, (name, pt)
        assert sum(pt[2:6]) > 0, (name, pt)
    assert kv["path_tasks"][16] == 0, kv["path_tasks"]
    assert lst["path_tasks"][16] == 1, lst["path_tasks"]  # the 4 KiB tensor
    h2d_dst = None
