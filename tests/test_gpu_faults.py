"""Failure handling, with every fault forced from the host: kernels still exit
through their own bounded waits, nothing on the GPU faults or hangs."""
import time

import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2512_16056_amd as mma  # noqa: E402
from gpu_helpers import log, session, to_host  # noqa: E402


def _copy_and_check(n, paths="both", **cfg):
    src_np = np.ascontiguousarray(W.uniform_bytes(12, 0, n, n))
    src = mma.PinnedBuffer(n)
    src.array[:] = src_np
    dst = torch.full((n,), W.WEIGHT_POISON, dtype=torch.uint8, device="cuda")
    t0 = time.time()
    mma.mma_memcpy_async(dst, src, n, mma.MMA_H2D)
    torch.cuda.synchronize()
    dt = time.time() - t0
    assert np.array_equal(to_host(dst), src_np)
    src.free()
    return dt


def test_sdma_submit_failures_are_rerouted():
    with session("both", chunk_bytes=1 << 20):
        mma.mma_reset_stats()
        mma.mma_test_set_fault(mma.MMA_FAULT_SDMA_SUBMIT_FAIL, 3)
        _copy_and_check(32 << 20)
        mma.mma_synchronize()
        st = mma.mma_get_stats()
        mma.mma_test_set_fault(mma.MMA_FAULT_SDMA_SUBMIT_FAIL, 0)
    log(f"  submit failures={st['sdma_submit_failures']} path bytes={st['path_bytes'][:2]}+cu {st['path_bytes'][16]}")
    assert st["failed_transfers"] == 0
    assert 1 <= st["sdma_submit_failures"] <= 3


@pytest.mark.parametrize("layout", [mma.MMA_KV_LAYOUT_PIECE, mma.MMA_KV_LAYOUT_XPACKED])
def test_kv_sdma_submit_failures_are_rerouted(layout):
    """Refused copy-engine commands during a KV fetch (host -> staging) and a KV offload
    (staging -> host, after the CU gather into staging): the micro-tasks go back to the CU path
    and both results match the oracle; no transfer fails."""
    from oracle import kv as okv
    s = W.KVShape(layers=3, block_tokens=16, kv_heads=2, head_dim=64, elem_bytes=2, gpu_num_blocks=40,
                  host_num_slots=32, n_blocks=24)
    geom = (s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes)
    ol = okv.LAYOUT_XPACKED if layout else okv.LAYOUT_PIECE
    lay = mma.kv_layout(s.layers, s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes, s.gpu_num_blocks,
                        s.host_num_slots, layout)
    hs, gb = W.kv_fetch_tables(s, cfg=3)
    with session("sdma", chunk_bytes=4 * s.piece_bytes):
        pool = mma.PinnedBuffer(s.host_num_slots * s.slot_bytes)
        pool.array[:] = np.random.default_rng(3).integers(0, 256, pool.nbytes, dtype=np.uint8)
        pool_np = pool.array.reshape(s.host_num_slots, -1).copy()
        layers = [torch.full((s.layer_bytes,), W.GPU_POISON, dtype=torch.uint8, device="cuda") for _ in range(s.layers)]
        before = [to_host(t).reshape(2, s.gpu_num_blocks, s.piece_bytes) for t in layers]
        mma.mma_reset_stats()
        mma.mma_test_set_fault(mma.MMA_FAULT_SDMA_SUBMIT_FAIL, 3)
        try:
            mma.mma_kv_fetch(lay, pool, layers, hs, gb)
            torch.cuda.synchronize()
            mma.mma_synchronize()
        finally:
            mma.mma_test_set_fault(mma.MMA_FAULT_SDMA_SUBMIT_FAIL, 0)
        st_fetch = mma.mma_get_stats()
        want = okv.kv_fetch(pool_np, before, hs, gb, ol, geom)
        for l in range(s.layers):
            assert np.array_equal(to_host(layers[l]).reshape(want[l].shape), want[l]), l
        views = [to_host(t).reshape(2, s.gpu_num_blocks, s.piece_bytes) for t in layers]
        dest = np.roll(hs, 3).astype(np.int32)
        mma.mma_test_set_fault(mma.MMA_FAULT_SDMA_SUBMIT_FAIL, 3)
        try:
            mma.mma_kv_offload(lay, pool, layers, gb, dest)
            torch.cuda.synchronize()
            mma.mma_synchronize()
        finally:
            mma.mma_test_set_fault(mma.MMA_FAULT_SDMA_SUBMIT_FAIL, 0)
        st = mma.mma_get_stats()
        want = okv.kv_offload(pool_np, views, gb, dest, ol, geom)
        assert np.array_equal(pool.array.reshape(s.host_num_slots, -1), want)
        pool.free()
    log(f"  refused commands: fetch {st_fetch['sdma_submit_failures']}, total {st['sdma_submit_failures']}")
    assert st_fetch["sdma_submit_failures"] >= 1
    assert st["sdma_submit_failures"] > st_fetch["sdma_submit_failures"]
    assert st["failed_transfers"] == 0


def test_sdma_only_submit_failures_fall_back_to_cu():
    with session("sdma", chunk_bytes=1 << 20):
        mma.mma_test_set_fault(mma.MMA_FAULT_SDMA_SUBMIT_FAIL, 1000000)
        _copy_and_check(8 << 20)
        mma.mma_test_set_fault(mma.MMA_FAULT_SDMA_SUBMIT_FAIL, 0)
        mma.mma_synchronize()
        st = mma.mma_get_stats()
    assert st["path_bytes"][16] == 8 << 20


def test_engine_stall_keeps_stream_blocked():
    with session("both", chunk_bytes=1 << 20):
        mma.mma_test_set_fault(mma.MMA_FAULT_ENGINE_STALL_US, 200000)
        try:
            dt = _copy_and_check(16 << 20)
        finally:
            mma.mma_test_set_fault(mma.MMA_FAULT_ENGINE_STALL_US, 0)
        mma.mma_synchronize()
    log(f"  stalled copy took {dt * 1e3:.1f} ms")
    assert dt >= 0.15


def test_watchdog_releases_stream_and_error_is_sticky():
    n = 8 << 20
    with session("both", chunk_bytes=1 << 20, watchdog_ms=300):
        src = mma.PinnedBuffer(n)
        dst = torch.empty(n, dtype=torch.uint8, device="cuda")
        mma.mma_test_set_fault(mma.MMA_FAULT_ENGINE_IGNORE, 1)
        try:
            t0 = time.time()
            mma.mma_memcpy_async(dst, src, n, mma.MMA_H2D)
            torch.cuda.synchronize()            # must return: the wait kernel's watchdog ends it
            dt = time.time() - t0
            deadline = time.time() + 10
            while mma.mma_get_stats()["failed_transfers"] == 0 and time.time() < deadline:
                time.sleep(0.01)
        finally:
            mma.mma_test_set_fault(mma.MMA_FAULT_ENGINE_IGNORE, 0)
        log(f"  watchdog released the stream after {dt * 1e3:.0f} ms")
        assert mma.mma_get_stats()["failed_transfers"] == 1
        with pytest.raises(mma.MMAError) as e:
            mma.mma_memcpy_async(dst, src, n, mma.MMA_H2D)
        assert e.value.name == "MMA_ERR_TRANSFER_FAILED"
        mma.mma_clear_error()
        src.array[:] = 3
        mma.mma_memcpy_async(dst, src, n, mma.MMA_H2D)
        torch.cuda.synchronize()
        assert bool((dst == 3).all())
        mma.mma_synchronize()
        src.free()


@pytest.mark.parametrize("refused", [1, 2, 1000000])
def test_device_control_refused_commands_go_to_cu(refused):
    """Device control on an idle stream: copy-engine commands refused at submission move their
    micro-tasks to the CU path before the launch; the copy is exact and nothing fails."""
    n = (48 << 20) + 5
    src_np = np.ascontiguousarray(W.uniform_bytes(12, 1, n, n))
    stream = torch.cuda.Stream()
    with session("both", control=mma.MMA_CONTROL_DEVICE):
        src = mma.PinnedBuffer(n)
        src.array[:] = src_np
        dst = torch.full((n,), W.WEIGHT_POISON, dtype=torch.uint8, device="cuda")
        torch.cuda.synchronize()
        mma.mma_reset_stats()
        mma.mma_test_set_fault(mma.MMA_FAULT_SDMA_SUBMIT_FAIL, refused)
        try:
            mma.mma_memcpy_async(dst, src, n, mma.MMA_H2D, stream)
            stream.synchronize()
        finally:
            mma.mma_test_set_fault(mma.MMA_FAULT_SDMA_SUBMIT_FAIL, 0)
        mma.mma_synchronize()
        st = mma.mma_get_stats()
        assert np.array_equal(to_host(dst), src_np)
        src.free()
    log(f"  refused={st['sdma_submit_failures']} commands={st['sdma_commands']} cu bytes={st['path_bytes'][16]}")
    assert st["failed_transfers"] == 0
    assert 1 <= st["sdma_submit_failures"] <= refused
    if refused > 2:  # every command refused: the CU path carried everything
        assert st["path_bytes"][16] == n


def test_device_control_watchdog_releases_stream_and_error_is_sticky():
    """Device control on an idle stream with the copy engines' completion signal held one count
    above their commands: the kernel's last wave never sees them finish, its watchdog releases
    the stream, the transfer is reported failed and the error is sticky. The data itself has
    landed (every real command completed)."""
    n = (64 << 20) + 3
    src_np = np.ascontiguousarray(W.uniform_bytes(12, 2, n, n))
    stream = torch.cuda.Stream()
    with session("both", control=mma.MMA_CONTROL_DEVICE, watchdog_ms=300):
        src = mma.PinnedBuffer(n)
        src.array[:] = src_np
        dst = torch.full((n,), W.WEIGHT_POISON, dtype=torch.uint8, device="cuda")
        torch.cuda.synchronize()
        mma.mma_test_set_fault(mma.MMA_FAULT_DEVICE_SIGNAL_HOLD, 1)
        try:
            t0 = time.time()
            mma.mma_memcpy_async(dst, src, n, mma.MMA_H2D, stream)
            stream.synchronize()                # must return: the wait's watchdog ends it
            dt = time.time() - t0
        finally:
            mma.mma_test_set_fault(mma.MMA_FAULT_DEVICE_SIGNAL_HOLD, 0)
        deadline = time.time() + 10
        while mma.mma_get_stats()["failed_transfers"] == 0 and time.time() < deadline:
            time.sleep(0.01)
        log(f"  watchdog released the stream after {dt * 1e3:.0f} ms")
        assert dt >= 0.25
        assert mma.mma_get_stats()["failed_transfers"] == 1
        assert np.array_equal(to_host(dst), src_np)
        with pytest.raises(mma.MMAError) as e:
            mma.mma_memcpy_async(dst, src, n, mma.MMA_H2D, stream)
        assert e.value.name == "MMA_ERR_TRANSFER_FAILED"
        mma.mma_clear_error()
        # the record came back: later transfers run normally
        for _ in range(70):
            mma.mma_memcpy_async(dst, src, n, mma.MMA_H2D, stream)
        stream.synchronize()
        mma.mma_synchronize()
        assert mma.mma_get_stats()["failed_transfers"] == 1
        src.free()
