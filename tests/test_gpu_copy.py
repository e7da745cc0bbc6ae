"""GPU parity of single copies and tensor lists against the oracle (byte-exact).

Every case calls the library through the C ABI (via the ctypes binding) and
compares each destination byte -- inside and outside the copied ranges -- with
oracle.copy on the same seeded inputs.
"""
import time

import numpy as np
import pytest
import torch

import workloads as W
from oracle import copy as ocopy

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is gpu-marked
    pytest.skip("no GPU", allow_module_level=True)

import paper_2512_16056_amd as mma  # noqa: E402
from gpu_helpers import PATHS, device_bytes, from_host, log, session, to_host  # noqa: E402

SIZES = [0, 1, 2, 3, 15, 16, 17, 31, 32, 33, 63, 64, 65, 255, 256, 257, 1023, 1024, 1025, 4095, 4096]
SRC_OFFS = [0, 1, 2, 3, 4, 7, 8, 9, 15]
DST_OFFS = [0, 1, 7, 15]
REGION = 8192


def _cases():
    return [(n, so, do) for n in SIZES for so in SRC_OFFS for do in DST_OFFS]


@pytest.mark.parametrize("direction", [mma.MMA_H2D, mma.MMA_D2H])
@pytest.mark.parametrize("chunk", [16, 48, 4096])
@pytest.mark.parametrize("paths", list(PATHS))
def test_tiny_bruteforce(paths, chunk, direction):
    log(f"tiny bruteforce paths={paths} chunk={chunk} dir={direction}")
    cases = _cases()
    src_np = np.ascontiguousarray(W.uniform_bytes(0, 0, chunk, REGION + 64))
    poison = np.full(len(cases) * REGION, 0xFF, np.uint8)
    # small_bytes=1: even the tiny copies may ride an SDMA engine
    with session(paths, chunk_bytes=chunk, small_bytes=1):
        if direction == mma.MMA_H2D:
            src = mma.PinnedBuffer(src_np.size)
            src.array[:] = src_np
            dst = from_host(poison)
            for k, (n, so, do) in enumerate(cases):
                mma.mma_memcpy_async(dst.data_ptr() + k * REGION + do, src.ptr + so, n, direction)
            torch.cuda.synchronize()
            mma.mma_synchronize()
            got = to_host(dst)
        else:
            src = from_host(src_np)
            dst = mma.PinnedBuffer(poison.size)
            dst.array[:] = poison
            for k, (n, so, do) in enumerate(cases):
                mma.mma_memcpy_async(dst.ptr + k * REGION + do, src.data_ptr() + so, n, direction)
            torch.cuda.synchronize()
            mma.mma_synchronize()
            got = dst.array.copy()
        stats = mma.mma_get_stats()
    for k, (n, so, do) in enumerate(cases):
        want = ocopy.memcpy(poison[k * REGION:(k + 1) * REGION], do, src_np, so, n)
        assert np.array_equal(got[k * REGION:(k + 1) * REGION], want), (n, so, do)
    assert stats["failed_transfers"] == 0
    if paths == "cu":
        assert sum(stats["path_bytes"][:16]) == 0
    if paths == "sdma":
        assert stats["path_bytes"][16] == 0


@pytest.mark.parametrize("direction", [mma.MMA_H2D, mma.MMA_D2H])
@pytest.mark.parametrize("paths", list(PATHS))
def test_copy_64mib(paths, direction):
    """The 64 MiB workload: one host->GPU copy split into 2 MiB micro-transfers (and its reverse)."""
    log(f"64MiB copy paths={paths} dir={direction}")
    n = W.COPY64_BYTES
    src_np = np.ascontiguousarray(W.uniform_bytes(1, W.TAG_DATA, 0, n))
    with session(paths, chunk_bytes=W.COPY64_CHUNK):
        for rep in range(3):
            if direction == mma.MMA_H2D:
                src = mma.PinnedBuffer(n)
                src.array[:] = src_np
                dst = device_bytes(n, W.WEIGHT_POISON)
                mma.mma_memcpy_async(dst, src, n, direction)
                torch.cuda.synchronize()
                got = to_host(dst)
            else:
                src = from_host(src_np)
                dst = mma.PinnedBuffer(n)
                dst.array[:] = W.WEIGHT_POISON
                mma.mma_memcpy_async(dst, src, n, direction)
                torch.cuda.synchronize()
                got = dst.array.copy()
            assert np.array_equal(got, ocopy.memcpy(np.full(n, W.WEIGHT_POISON, np.uint8), 0, src_np, 0, n))
        mma.mma_synchronize()
        stats = mma.mma_get_stats()
    assert stats["failed_transfers"] == 0
    total = sum(stats["path_bytes"])
    assert total == 3 * n
    log(f"  path bytes: cu={stats['path_bytes'][16]} sdma={stats['path_bytes'][:4]}")


@pytest.mark.parametrize("nap", ["default", "off"])
def test_engine_naps(nap):
    """The engine thread naps between rounds while every path has work queued (Section 5.3, CPU
    overhead; engine_nap_us), or polls throughout (MMA_ENGINE_NAP_OFF). 1 GiB copies in both
    directions, three each, are the oracle's bytes either way; the statistics count the naps."""
    log(f"engine naps: {nap}")
    n = 1 << 30
    src_np = np.ascontiguousarray(W.uniform_bytes(1, W.TAG_DATA, 7, n))
    over = {} if nap == "default" else {"engine_nap_us": mma.MMA_ENGINE_NAP_OFF}
    with session("both", **over) as cfg:
        assert cfg.engine_nap_us == (50 if nap == "default" else mma.MMA_ENGINE_NAP_OFF)
        h = mma.PinnedBuffer(n)
        d = device_bytes(n)
        dsrc = from_host(src_np)
        for direction in (mma.MMA_H2D, mma.MMA_D2H):
            for rep in range(3):
                if direction == mma.MMA_H2D:
                    h.array[:] = src_np
                    d.fill_(W.WEIGHT_POISON)
                    mma.mma_memcpy_async(d, h, n, direction)
                    torch.cuda.synchronize()
                    got = to_host(d)
                else:
                    d.copy_(dsrc)
                    h.array[:] = W.WEIGHT_POISON
                    torch.cuda.synchronize()
                    mma.mma_memcpy_async(h, d, n, direction)
                    torch.cuda.synchronize()
                    got = h.array.copy()
                assert np.array_equal(got, ocopy.memcpy(np.full(n, W.WEIGHT_POISON, np.uint8), 0, src_np, 0, n)), \
                    (direction, rep)
        mma.mma_synchronize()
        stats = mma.mma_get_stats()
        h.free()
    assert stats["failed_transfers"] == 0
    log(f"  naps {stats['engine_naps']}, engine CPU {stats['engine_cpu_ns'] / 1e6:.1f} ms")
    if nap == "default":
        assert stats["engine_naps"] > 0
    else:
        assert stats["engine_naps"] == 0


@pytest.mark.parametrize("direction", [mma.MMA_H2D, mma.MMA_D2H])
def test_whole_transfers_on_cu_path(direction):
    """Default configuration around the size limit of transfers taken whole by the CU path
    (24 MiB host->device, 8 MiB device->host, and at most 48 CU entries): below it no copy
    engine takes part, above it they do; every byte matches the oracle, poison outside the
    destination stays."""
    limit = (24 << 20) if direction == mma.MMA_H2D else (8 << 20)
    cases = [(3 << 20) + 1, 4 << 20, limit - 5, limit, limit + 1]
    pad = 4096
    with session("both", cu_whole_bytes=0, cu_whole_bytes_d2h=0):  # 0: the default limits
        cfg = mma.mma_get_config()
        assert (cfg.cu_whole_bytes, cfg.cu_whole_bytes_d2h) == (24 << 20, 8 << 20)
        for n in cases:
            log(f"whole transfer n={n} dir={direction}")
            src_np = np.ascontiguousarray(W.uniform_bytes(13, direction, n, n + 16))
            mma.mma_synchronize()
            mma.mma_reset_stats()
            if direction == mma.MMA_H2D:
                src = mma.PinnedBuffer(n + 16)
                src.array[:] = src_np
                dst = device_bytes(n + 2 * pad, W.WEIGHT_POISON)
                mma.mma_memcpy_async(dst.data_ptr() + pad + 3, src.ptr + 3, n, direction)
                torch.cuda.synchronize()
                got = to_host(dst)
            else:
                src = from_host(src_np)
                dst = mma.PinnedBuffer(n + 2 * pad)
                dst.array[:] = W.WEIGHT_POISON
                mma.mma_memcpy_async(dst.ptr + pad + 3, src.data_ptr() + 3, n, direction)
                torch.cuda.synchronize()
                got = dst.array.copy()
            mma.mma_synchronize()
            st = mma.mma_get_stats()
            want = ocopy.memcpy(np.full(n + 2 * pad, W.WEIGHT_POISON, np.uint8), pad + 3, src_np, 3, n)
            assert np.array_equal(got, want), n
            assert st["failed_transfers"] == 0
            if n <= limit:
                assert st["sdma_commands"] == 0 and st["path_bytes"][16] == n, (n, st["path_bytes"])
            else:
                assert st["sdma_commands"] > 0, n
            if direction == mma.MMA_D2H:
                dst.free()
            else:
                src.free()
        # tensor lists: 48 tensors fit one launch, 49 do not
        for count in (48, 49):
            sizes = [100 * 1024 + 16 * k for k in range(count)]
            offs, total = W.arena_offsets(sizes, 256)
            host = mma.PinnedBuffer(total)
            host.array[:] = W.uniform_bytes(14, count, direction, total)
            devs = [device_bytes(z + 64, W.WEIGHT_POISON) for z in sizes]
            mma.mma_synchronize()
            mma.mma_reset_stats()
            if direction == mma.MMA_H2D:
                mma.mma_weights_load([(devs[t], host.ptr + offs[t], z) for t, z in enumerate(sizes)], direction)
            else:
                for t, z in enumerate(sizes):
                    devs[t][:z] = torch.from_numpy(host.array[offs[t]:offs[t] + z].copy()).cuda()
                back = mma.PinnedBuffer(total)
                back.array[:] = W.WEIGHT_POISON
                mma.mma_weights_load([(back.ptr + offs[t], devs[t], z) for t, z in enumerate(sizes)], direction)
            torch.cuda.synchronize()
            mma.mma_synchronize()
            st = mma.mma_get_stats()
            for t, z in enumerate(sizes):
                if direction == mma.MMA_H2D:
                    got = to_host(devs[t])
                    want = ocopy.memcpy(np.full(z + 64, W.WEIGHT_POISON, np.uint8), 0, host.array, offs[t], z)
                else:
                    got = back.array[offs[t]:offs[t] + z]
                    want = host.array[offs[t]:offs[t] + z]
                assert np.array_equal(got, want), (count, t)
            assert (st["sdma_commands"] == 0) == (count == 48), (count, st["sdma_commands"])
            host.free()
            if direction == mma.MMA_D2H:
                back.free()


def test_deep_queue_does_not_wait_for_the_stream():
    """600 small copies queued on a stream held by a long-running kernel: they take light slots
    (a whole self-contained launch needs no transfer record), so the calls return while the
    stream is still held -- as hipMemcpyAsync would -- and every copy lands afterwards."""
    n, sz = 600, 64 << 10
    with session("both", cu_whole_bytes=0, cu_whole_bytes_d2h=0):
        st = torch.cuda.Stream()
        # a spin kernel of about 0.5 s holds the stream (calibrated on this GPU's clock)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(st)
        with torch.cuda.stream(st):
            torch.cuda._sleep(10_000_000)
        b.record(st)
        b.synchronize()
        cycles = int(10_000_000 * 500.0 / max(a.elapsed_time(b), 1e-3))
        src_np = np.ascontiguousarray(W.uniform_bytes(15, 0, 0, n * sz))
        src = mma.PinnedBuffer(n * sz)
        src.array[:] = src_np
        dst = device_bytes(n * sz, W.WEIGHT_POISON)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        with torch.cuda.stream(st):
            torch.cuda._sleep(cycles)
        e1.record(st)
        t0 = time.perf_counter()
        for i in range(n):
            mma.mma_memcpy_async(dst.data_ptr() + i * sz, src.ptr + i * sz, sz, mma.MMA_H2D, st)
        t_submit = time.perf_counter() - t0
        held = not e1.query()  # the spin kernel is still running
        st.synchronize()
        spin_ms = e0.elapsed_time(e1)
        log(f"  {n} submissions took {t_submit * 1e3:.1f} ms behind a {spin_ms:.0f} ms spin kernel")
        assert held and t_submit * 1e3 < 0.5 * spin_ms, (t_submit, spin_ms)
        assert np.array_equal(to_host(dst), src_np)
        mma.mma_synchronize()
        assert mma.mma_get_stats()["failed_transfers"] == 0
        src.free()


def _ragged_list(seed, count, max_size):
    r = np.random.default_rng(seed)
    sizes = [int(x) for x in r.integers(0, max_size, count)]
    sizes[0] = 0
    sizes[1] = 1
    sizes[2] = 64 * 1024 - 1   # just below the CU-only threshold
    sizes[3] = 64 * 1024       # at the threshold
    return sizes


@pytest.mark.parametrize("stream", ["legacy", "idle"])
@pytest.mark.parametrize("direction", [mma.MMA_H2D, mma.MMA_D2H])
@pytest.mark.parametrize("paths", list(PATHS))
def test_tensor_list_ragged(paths, direction, stream):
    """A ragged list of 40 tensors up to 3 MiB, on the legacy default stream and on a stream of its
    own with nothing pending (where the copy engines may start before the kernel launch)."""
    log(f"tensor list paths={paths} dir={direction} stream={stream}")
    st = torch.cuda.Stream() if stream == "idle" else None
    sizes = _ragged_list(7 + direction, 40, 3 * 1024 * 1024)
    src_offs, total = W.arena_offsets(sizes, 16)
    # destinations interleaved with untouched 4 KiB gaps, some misaligned by 16 B
    dst_offs, cur = [], 4096
    for s in sizes:
        dst_offs.append(cur)
        cur += s + 4096 + 16
    dtotal = cur
    src_np = np.ascontiguousarray(W.uniform_bytes(2, W.TAG_DATA, 99, total))
    poison = np.full(dtotal, W.WEIGHT_POISON, np.uint8)
    with session(paths, chunk_bytes=256 * 1024):
        if direction == mma.MMA_H2D:
            src = mma.PinnedBuffer(total)
            src.array[:] = src_np
            dst = from_host(poison)
            torch.cuda.synchronize()
            mma.mma_weights_load([(dst.data_ptr() + d, src.ptr + s, n) for d, s, n in zip(dst_offs, src_offs, sizes)],
                                 direction, st)
            torch.cuda.synchronize()
            got = to_host(dst)
        else:
            src = from_host(src_np)
            dst = mma.PinnedBuffer(dtotal)
            dst.array[:] = poison
            torch.cuda.synchronize()
            mma.mma_weights_load([(dst.ptr + d, src.data_ptr() + s, n) for d, s, n in zip(dst_offs, src_offs, sizes)],
                                 direction, st)
            torch.cuda.synchronize()
            got = dst.array.copy()
        mma.mma_synchronize()
    want = ocopy.tensor_list(poison, src_np, list(zip(dst_offs, src_offs, sizes)))
    assert np.array_equal(got, want)


@pytest.mark.parametrize("direction", [mma.MMA_H2D, mma.MMA_D2H])
@pytest.mark.parametrize("merge", [1, 0, 5])
def test_sdma_command_merging(merge, direction):
    """Micro-tasks that follow each other in both address spaces go to a copy engine as one
    command (at most sdma_merge_tasks of them; 0 = default). The bytes must not depend on it: a
    ragged linear copy and a list of tensors packed back to back on both sides (so runs cross
    tensor boundaries), on the SDMA engines only, against the oracle."""
    log(f"sdma merging merge={merge} dir={direction}")
    chunk = 256 << 10
    n = 37 * chunk + 12345
    sizes = _ragged_list(21 + direction, 24, 3 * chunk)
    offs, ltotal = W.arena_offsets(sizes, 1)
    src_np = np.ascontiguousarray(W.uniform_bytes(2, W.TAG_DATA, 123, n + ltotal))
    with session("sdma", chunk_bytes=chunk, sdma_merge_tasks=merge, small_bytes=1):
        mma.mma_reset_stats()
        if direction == mma.MMA_H2D:
            src = mma.PinnedBuffer(n + ltotal)
            src.array[:] = src_np
            dst = device_bytes(n + ltotal, W.WEIGHT_POISON)
            mma.mma_memcpy_async(dst, src, n, direction)
            mma.mma_weights_load([(dst.data_ptr() + n + o, src.ptr + n + o, k) for o, k in zip(offs, sizes)],
                                 direction)
            torch.cuda.synchronize()
            got = to_host(dst)
        else:
            src = from_host(src_np)
            dst = mma.PinnedBuffer(n + ltotal)
            dst.array[:] = W.WEIGHT_POISON
            mma.mma_memcpy_async(dst, src, n, direction)
            mma.mma_weights_load([(dst.ptr + n + o, src.data_ptr() + n + o, k) for o, k in zip(offs, sizes)],
                                 direction)
            torch.cuda.synchronize()
            got = dst.array.copy()
        mma.mma_synchronize()
        stats = mma.mma_get_stats()
    poison = np.full(n + ltotal, W.WEIGHT_POISON, np.uint8)
    want = ocopy.tensor_list(ocopy.memcpy(poison, 0, src_np, 0, n), src_np,
                             [(n + o, n + o, k) for o, k in zip(offs, sizes)])
    assert np.array_equal(got, want)
    assert stats["failed_transfers"] == 0
    sdma_tasks = sum(stats["path_tasks"][:16])
    log(f"  sdma tasks={sdma_tasks} commands={stats['sdma_commands']} cu tasks={stats['path_tasks'][16]}")
    assert sdma_tasks > 0
    if merge == 1:
        assert stats["sdma_commands"] == sdma_tasks
    else:
        assert stats["sdma_commands"] < sdma_tasks


def test_rejects_bad_arguments():
    with session("both"):
        src = mma.PinnedBuffer(4096)
        dst = device_bytes(4096)
        pageable = np.zeros(4096, np.uint8)
        with pytest.raises(mma.MMAError) as e:
            mma.mma_memcpy_async(dst, pageable, 4096, mma.MMA_H2D)
        assert e.value.name == "MMA_ERR_NOT_PINNED"
        with pytest.raises(mma.MMAError) as e:
            mma.mma_memcpy_async(dst, src, 4096, 7)
        assert e.value.name == "MMA_ERR_INVALID_ARG"
        with pytest.raises(mma.MMAError) as e:          # host range runs past the allocation
            mma.mma_memcpy_async(dst, src, 8192, mma.MMA_H2D)
        assert e.value.name in ("MMA_ERR_NOT_PINNED", "MMA_ERR_INVALID_ARG")
        with pytest.raises(mma.MMAError) as e:          # device pointer where host memory is expected
            mma.mma_memcpy_async(dst, dst, 16, mma.MMA_H2D)
        assert e.value.name == "MMA_ERR_INVALID_ARG"
        with pytest.raises(mma.MMAError) as e:          # overlapping destinations
            mma.mma_weights_load([(dst, src, 64), (dst.data_ptr() + 32, src, 64)], mma.MMA_H2D)
        assert e.value.name == "MMA_ERR_INVALID_ARG"
        # sizes whose range wraps the address space (a negative length cast to unsigned, or one that
        # ends just past 2^64), from inside allocations that earlier calls validated and cached
        mma.mma_memcpy_async(dst, src, 4096, mma.MMA_H2D)
        mma.mma_memcpy_async(src, dst, 4096, mma.MMA_D2H)
        torch.cuda.synchronize()
        h, d = src.ptr + 64, dst.data_ptr() + 64
        for n in ((1 << 64) - 1, (1 << 64) - h + 16, (1 << 64) - d + 16):
            for dr, a, b in ((mma.MMA_H2D, d, h), (mma.MMA_D2H, h, d)):
                with pytest.raises(mma.MMAError) as e:
                    mma.mma_memcpy_async(a, b, n, dr)
                assert e.value.name in ("MMA_ERR_NOT_PINNED", "MMA_ERR_INVALID_ARG"), (n, dr)
            with pytest.raises(mma.MMAError) as e:
                mma.mma_digest_u32(d, n & ~3, device_bytes(8, 0))
            assert e.value.name == "MMA_ERR_INVALID_ARG", n
        mma.mma_memcpy_async(dst, src, 0, mma.MMA_H2D)   # zero bytes: no-op
        mma.mma_weights_load([], mma.MMA_H2D)
        torch.cuda.synchronize()
        assert mma.mma_get_stats()["failed_transfers"] == 0
        src.free()


@pytest.mark.parametrize("direction", [mma.MMA_H2D, mma.MMA_D2H])
def test_sync_memcpy(direction):
    """mma_memcpy returns only once the data has arrived, ordered after earlier work on the default
    stream: a producer kernel on the default stream writes the source right before a D2H copy."""
    with session("both", chunk_bytes=1 << 20):
        for n in (0, 1, 4095, 1 << 20, (9 << 20) + 5):
            src_np = np.ascontiguousarray(W.uniform_bytes(33, direction, n, n))
            if direction == mma.MMA_H2D:
                src = mma.PinnedBuffer(n)
                src.array[:] = src_np
                dst = device_bytes(n, W.WEIGHT_POISON)
                mma.mma_memcpy(dst, src, n, direction)
                got = to_host(dst)[:n]  # synchronising read; the copy itself already returned
            else:
                src = device_bytes(n, 0)
                dev = device_bytes(n, 0)
                if n:
                    src[:n].copy_(torch.from_numpy(src_np.copy()))
                    torch.cuda.synchronize()
                    dev[:n].copy_(src[:n])  # producer on the default stream, not synchronised
                dst = mma.PinnedBuffer(n)
                dst.array[:] = W.WEIGHT_POISON
                mma.mma_memcpy(dst, dev, n, direction)
                got = dst.array[:n].copy()  # no synchronisation: mma_memcpy must have finished
            assert np.array_equal(got, src_np), n
        mma.mma_synchronize()


HIP_STREAM_PER_THREAD = 2  # hipStreamPerThread


@pytest.mark.parametrize("kind", ["idle", "busy", "per_thread", "legacy"])
@pytest.mark.parametrize("control", [mma.MMA_CONTROL_HOST, mma.MMA_CONTROL_DEVICE])
@pytest.mark.parametrize("direction", [mma.MMA_H2D, mma.MMA_D2H])
def test_sync_memcpy_stream(direction, control, kind):
    """mma_memcpy_stream returns MMA_COPY_RETIRED once the data has arrived, on
    - idle: a stream of its own with nothing pending. Above the whole-launch limit the copy engines
      are handed the copy before the kernel is launched (the idle-stream early start); the call
      must still be told when it retires, rather than fail at its time limit;
    - busy: the same stream behind a spin kernel; device to host, the source is written on that
      stream after the spin, right before the call, so the copy must be ordered after it;
    - per_thread: hipStreamPerThread; legacy: the legacy default stream.
    An engine-driven copy, a whole launch, a one-byte and a zero-byte copy each; every byte against
    the oracle, read without further synchronisation."""
    sizes = [(40 << 20) + 3, (3 << 20) + 5, 1, 0]
    top = max(sizes)
    src_np = np.ascontiguousarray(W.uniform_bytes(41, direction, 0, top))
    side = torch.cuda.Stream()
    stream = {"idle": side, "busy": side, "per_thread": HIP_STREAM_PER_THREAD, "legacy": 0}[kind]
    with session("both", cu_whole_bytes=0, cu_whole_bytes_d2h=0, control=control):
        if direction == mma.MMA_H2D:
            src = mma.PinnedBuffer(top)
            src.array[:] = src_np
        else:
            fresh = from_host(src_np)
            src = device_bytes(top, 0)
        for n in sizes:
            for rep in range(2):
                log(f"sync stream kind={kind} control={control} dir={direction} n={n} rep={rep}")
                if direction == mma.MMA_H2D:
                    dst = device_bytes(top, W.WEIGHT_POISON)
                    dptr, sptr = dst.data_ptr(), src.ptr
                else:
                    dst = mma.PinnedBuffer(top)
                    dst.array[:] = W.WEIGHT_POISON
                    dptr, sptr = dst.ptr, src.data_ptr()
                    src.zero_()
                    if kind != "busy":
                        src.copy_(fresh)
                torch.cuda.synchronize()  # every stream has nothing pending
                if kind == "busy":
                    with torch.cuda.stream(side):
                        torch.cuda._sleep(1_000_000)
                        if direction == mma.MMA_D2H:
                            src.copy_(fresh)  # the producer, on the copy's stream
                t0 = time.perf_counter()
                outcome = mma.mma_memcpy_stream(dptr, sptr, n, direction, stream)
                dt = time.perf_counter() - t0
                got = to_host(dst) if direction == mma.MMA_H2D else dst.array.copy()
                if direction == mma.MMA_D2H:
                    dst.free()
                assert outcome == mma.MMA_COPY_RETIRED, (n, outcome)
                assert dt < 2.0, (n, dt)
                want = ocopy.memcpy(np.full(top, W.WEIGHT_POISON, np.uint8), 0, src_np, 0, n)
                assert np.array_equal(got, want), n
        torch.cuda.synchronize()
        mma.mma_synchronize()
        assert mma.mma_get_stats()["failed_transfers"] == 0
        if direction == mma.MMA_H2D:
            src.free()


MISALIGNED = [(1, 0), (0, 1), (5, 9), (15, 2)]  # (source, destination) offsets modulo 16


@pytest.mark.parametrize("direction", [mma.MMA_H2D, mma.MMA_D2H])
@pytest.mark.parametrize("paths", ["default", *PATHS])
def test_misaligned_large(paths, direction):
    """Copies whose ends differ in alignment modulo 16, 1-40 MiB: whole CU-path launches below
    the size limit and multipath transfers above it (default paths), and each path set alone.
    The CU path realigns in registers; every byte matches the oracle and the poison around the
    destination stays."""
    sizes = [(1 << 20) + 3, (8 << 20) - 1, (24 << 20) - 7, (40 << 20) + 11]
    pad = 4096
    top = max(sizes) + 2 * pad
    src_np = np.ascontiguousarray(W.uniform_bytes(14, direction, 0, top))
    opts = {} if paths == "default" else PATHS[paths]
    with session("both", **{"cu_whole_bytes": 0, "cu_whole_bytes_d2h": 0, **opts}):
        if direction == mma.MMA_H2D:
            src = mma.PinnedBuffer(top)
            src.array[:] = src_np
        else:
            src = from_host(src_np)
        for n in sizes:
            for so, do in MISALIGNED:
                log(f"misaligned paths={paths} dir={direction} n={n} src+{so} dst+{do}")
                if direction == mma.MMA_H2D:
                    dst = device_bytes(top, W.WEIGHT_POISON)
                    mma.mma_memcpy_async(dst.data_ptr() + pad + do, src.ptr + so, n, direction)
                    torch.cuda.synchronize()
                    got = to_host(dst)
                else:
                    dst = mma.PinnedBuffer(top)
                    dst.array[:] = W.WEIGHT_POISON
                    mma.mma_memcpy_async(dst.ptr + pad + do, src.data_ptr() + so, n, direction)
                    torch.cuda.synchronize()
                    got = dst.array.copy()
                    dst.free()
                want = ocopy.memcpy(np.full(top, W.WEIGHT_POISON, np.uint8), pad + do, src_np, so, n)
                assert np.array_equal(got, want), (n, so, do)
        mma.mma_synchronize()
        st = mma.mma_get_stats()
    assert st["failed_transfers"] == 0
    if paths == "cu":
        assert sum(st["path_bytes"][:16]) == 0
    if paths == "sdma":
        assert st["path_bytes"][16] == 0
