"""GPU parity of transfers under device control (control = MMA_CONTROL_DEVICE) against the oracle.

Under device control the calling thread plans the whole transfer at submission and the
dummy-task kernel alone tracks its completion: the CU path's entries are all published before
the launch, the copy engines get a fixed share of a linear transfer when the stream has nothing
pending, and the kernel's last wave polls their completion signal. These tests check, byte for
byte against oracle.copy / oracle.kv on seeded inputs:
  - single copies of ragged sizes in both directions, on an idle stream (copy engines and CU
    path) and on a busy one (CU path only), with poison outside the destination untouched;
  - a tensor list with tensors below the CU-only size;
  - paged-KV fetch and offload in both GPU block layouts (CU path only);
  - stream ordering: a dependent kernel on the stream sees every byte of the copy, including
    the copy engines' share;
  - more transfers than there are records, the blocking mma_memcpy, a tensor list with more
    micro-tasks than a ring holds (planned again at a larger chunk, still under device control),
    and a KV transfer with more (handed to the engine thread).
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import copy as ocopy
from oracle import digest as odigest
from oracle import kv as okv

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2512_16056_amd as mma  # noqa: E402
from gpu_helpers import device_bytes, from_host, log, session, to_host  # noqa: E402

DEVICE = dict(control=mma.MMA_CONTROL_DEVICE)
SIZES = [1, 4095, (64 << 10) + 3, (3 << 20) + 1, (24 << 20) + 5, 64 << 20, (200 << 20) + 7]
PAD = 4096


def _busy(stream, ms=2.0):
    """Keep `stream` busy for about `ms` milliseconds (a GPU sleep kernel)."""
    with torch.cuda.stream(stream):
        torch.cuda._sleep(int(ms * 1e6))  # about 1 GHz cycles


def _copy(direction, n, src_np, stream, idle):
    """One copy of n bytes with PAD bytes of poison on each side of the destination; returns
    the destination region as numpy."""
    poison = np.full(n + 2 * PAD, W.WEIGHT_POISON, np.uint8)
    torch.cuda.synchronize()
    if direction == mma.MMA_H2D:
        src = mma.PinnedBuffer(n)
        src.array[:] = src_np
        dst = from_host(poison)
        torch.cuda.synchronize()
        if not idle:
            _busy(stream)
        mma.mma_memcpy_async(dst.data_ptr() + PAD, src.ptr, n, direction, stream)
        stream.synchronize()
        return to_host(dst)
    src = from_host(src_np)
    dst = mma.PinnedBuffer(poison.size)
    dst.array[:] = poison
    torch.cuda.synchronize()
    if not idle:
        _busy(stream)
    mma.mma_memcpy_async(dst.ptr + PAD, src.data_ptr(), n, direction, stream)
    stream.synchronize()
    return dst.array.copy()


@pytest.mark.parametrize("idle", [True, False])
@pytest.mark.parametrize("direction", [mma.MMA_H2D, mma.MMA_D2H])
@pytest.mark.parametrize("whole", ["default", "off"])
def test_device_copy(whole, direction, idle):
    """Ragged copies from 1 B to 200 MiB. whole='off' keeps even the small ones on a record
    (cu_whole_bytes=1) instead of a self-contained launch."""
    extra = dict(cu_whole_bytes=1, cu_whole_bytes_d2h=1) if whole == "off" else {}
    stream = torch.cuda.Stream()
    engine_bytes = 0
    with session("both", **DEVICE, **extra):
        assert mma.mma_get_config().control == mma.MMA_CONTROL_DEVICE
        for n in SIZES:
            log(f"device copy whole={whole} dir={direction} idle={idle} n={n}")
            src_np = np.ascontiguousarray(W.uniform_bytes(21, direction, n, n))
            before = mma.mma_get_stats()
            got = _copy(direction, n, src_np, stream, idle)
            mma.mma_synchronize()
            after = mma.mma_get_stats()
            want = ocopy.memcpy(np.full(n + 2 * PAD, W.WEIGHT_POISON, np.uint8), PAD, src_np, 0, n)
            assert np.array_equal(got, want), n
            eng = sum(after["path_bytes"][:16]) - sum(before["path_bytes"][:16])
            assert sum(after["path_bytes"]) - sum(before["path_bytes"]) == n
            assert after["failed_transfers"] == before["failed_transfers"]
            if not idle:
                assert eng == 0, "copy engines took part on a stream with work pending"
            engine_bytes += eng
    log(f"  copy-engine bytes over the sizes: {engine_bytes}")
    if idle:
        assert engine_bytes > 0, "the copy engines never took part on an idle stream"


def test_device_tensor_list():
    """A list with tensors below and above the CU-only size, on an idle stream."""
    sizes = [5, 8 << 10, 3 << 20, (64 << 10) - 1, 100, 17 << 20, (2 << 20) + 9, 1 << 10, 40 << 20]
    stream = torch.cuda.Stream()
    offs, off = [], 0
    for z in sizes:
        offs.append(off)
        off += (z + 255) // 256 * 256
    total = off
    src_np = np.ascontiguousarray(W.uniform_bytes(22, 0, 0, total))
    with session("both", **DEVICE):
        src = mma.PinnedBuffer(total)
        src.array[:] = src_np
        dsts = [device_bytes(z, W.WEIGHT_POISON) for z in sizes]
        torch.cuda.synchronize()
        mma.mma_weights_load([(d, src.ptr + o, z) for d, o, z in zip(dsts, offs, sizes)], mma.MMA_H2D, stream)
        stream.synchronize()
        mma.mma_synchronize()
        stats = mma.mma_get_stats()
        for d, o, z in zip(dsts, offs, sizes):
            assert np.array_equal(to_host(d)[:z], src_np[o:o + z]), z
    assert stats["failed_transfers"] == 0
    assert sum(stats["path_bytes"]) == sum(sizes)


KV_SHAPES = {
    "piece": (W.KVShape(layers=4, block_tokens=16, kv_heads=2, head_dim=64, elem_bytes=2,
                        gpu_num_blocks=300, host_num_slots=256, n_blocks=200), okv.LAYOUT_PIECE),
    "xpacked": (W.KVShape(layers=4, block_tokens=16, kv_heads=8, head_dim=128, elem_bytes=2,
                          gpu_num_blocks=300, host_num_slots=256, n_blocks=200), okv.LAYOUT_XPACKED),
    "hnd": (W.KVShape(layers=4, block_tokens=16, kv_heads=8, head_dim=128, elem_bytes=2,
                      gpu_num_blocks=300, host_num_slots=256, n_blocks=200), okv.LAYOUT_HND),
}


def _kv_layout(s, layout):
    gl = {okv.LAYOUT_PIECE: mma.MMA_KV_LAYOUT_PIECE, okv.LAYOUT_XPACKED: mma.MMA_KV_LAYOUT_XPACKED,
          okv.LAYOUT_HND: mma.MMA_KV_LAYOUT_HND}[layout]
    return mma.kv_layout(s.layers, s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes, s.gpu_num_blocks,
                         s.host_num_slots, gl)


@pytest.mark.parametrize("chunk", [4096, 1 << 21])
@pytest.mark.parametrize("shape", list(KV_SHAPES))
def test_device_kv_roundtrip(shape, chunk):
    """Fetch then offload (into other slots) on an idle stream: CU path only, byte-exact."""
    s, layout = KV_SHAPES[shape]
    geom = (s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes)
    hs, gb = W.kv_fetch_tables(s, cfg=3)
    plan = W.kv_offload_plan(s, cfg=4)
    stream = torch.cuda.Stream()
    log(f"device kv shape={shape} chunk={chunk}")
    with session("both", chunk_bytes=chunk, **DEVICE):
        r = np.random.default_rng(31)
        pool = mma.PinnedBuffer(s.host_num_slots * s.slot_bytes)
        pool.array[:] = r.integers(0, 256, pool.nbytes, dtype=np.uint8)
        layers = [device_bytes(s.layer_bytes, W.GPU_POISON) for _ in range(s.layers)]
        before = [to_host(t).reshape(2, s.gpu_num_blocks, s.piece_bytes) for t in layers]
        torch.cuda.synchronize()
        mma.mma_kv_fetch(_kv_layout(s, layout), pool, layers, hs, gb, stream)
        stream.synchronize()
        pool_v = pool.array.reshape(s.host_num_slots, s.slot_bytes)
        for l in range(s.layers):
            want = okv.kv_fetch_layer(pool_v, before[l], l, s.layers, hs, gb, layout, geom)
            got = to_host(layers[l]).reshape(2, s.gpu_num_blocks, s.piece_bytes)
            assert np.array_equal(got, want), f"layer {l}"
        views = [to_host(t).reshape(2, s.gpu_num_blocks, s.piece_bytes) for t in layers]
        pool_before = pool.array.copy()
        mma.mma_kv_offload(_kv_layout(s, layout), pool, layers, plan.src_blocks, plan.dest, stream)
        stream.synchronize()
        want = okv.kv_offload(pool_before.reshape(s.host_num_slots, -1), views, plan.src_blocks, plan.dest,
                              layout, geom)
        assert np.array_equal(pool.array.reshape(s.host_num_slots, -1), want)
        mma.mma_synchronize()
        stats = mma.mma_get_stats()
    assert stats["failed_transfers"] == 0
    assert sum(stats["path_bytes"][:16]) == 0, "copy engines took part in a KV transfer under device control"


@pytest.mark.parametrize("shape", list(KV_SHAPES))
def test_device_kv_hbm_pool(shape):
    """A KV pool in HBM (the CU path gathers and scatters within HBM): fetch, then offload the
    same blocks into other slots, both against the oracle."""
    s, layout = KV_SHAPES[shape]
    geom = (s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes)
    hs, gb = W.kv_fetch_tables(s, cfg=3)
    plan = W.kv_offload_plan(s, cfg=4)
    stream = torch.cuda.Stream()
    with session("both", chunk_bytes=1 << 20, **DEVICE):
        r = np.random.default_rng(33)
        pool_np = r.integers(0, 256, s.host_num_slots * s.slot_bytes, dtype=np.uint8)
        dpool = torch.from_numpy(pool_np.copy()).cuda()
        layers = [device_bytes(s.layer_bytes, W.GPU_POISON) for _ in range(s.layers)]
        before = [to_host(t).reshape(2, s.gpu_num_blocks, s.piece_bytes) for t in layers]
        torch.cuda.synchronize()
        mma.mma_kv_fetch(_kv_layout(s, layout), dpool, layers, hs, gb, stream)
        stream.synchronize()
        pool_v = pool_np.reshape(s.host_num_slots, s.slot_bytes)
        for l in range(s.layers):
            want = okv.kv_fetch_layer(pool_v, before[l], l, s.layers, hs, gb, layout, geom)
            assert np.array_equal(to_host(layers[l]).reshape(2, s.gpu_num_blocks, s.piece_bytes), want), l
        views = [to_host(t).reshape(2, s.gpu_num_blocks, s.piece_bytes) for t in layers]
        mma.mma_kv_offload(_kv_layout(s, layout), dpool, layers, plan.src_blocks, plan.dest, stream)
        stream.synchronize()
        want = okv.kv_offload(pool_v, views, plan.src_blocks, plan.dest, layout, geom)
        assert np.array_equal(to_host(dpool).reshape(s.host_num_slots, -1), want)
        mma.mma_synchronize()
        assert mma.mma_get_stats()["failed_transfers"] == 0


@pytest.mark.parametrize("rep", range(3))
def test_device_stream_ordering(rep):
    """A 256 MiB host->device copy on an idle stream (the copy engines carry their share), then
    the digest kernel on the same stream: its digest equals the oracle's digest of the source,
    so the stream waited for every path. Then the reverse: a kernel writes the source and the
    device->host copy follows on the stream, queued behind it or after it has finished (then the
    copy engines take part); either way it must see the kernel's bytes."""
    n = 256 << 20
    src_np = np.ascontiguousarray(W.uniform_bytes(23, rep, 0, n))
    stream = torch.cuda.Stream()
    with session("both", **DEVICE):
        src = mma.PinnedBuffer(n)
        src.array[:] = src_np
        dst = device_bytes(n, W.WEIGHT_POISON)
        out = torch.zeros(1, dtype=torch.int64, device="cuda")
        torch.cuda.synchronize()
        before = mma.mma_get_stats()
        mma.mma_memcpy_async(dst, src, n, mma.MMA_H2D, stream)
        mma.mma_digest_u32(dst.data_ptr(), n, out.data_ptr(), stream)
        stream.synchronize()
        got = int(out.cpu().numpy().view(np.uint64)[0])
        assert got == odigest.digest(src_np)
        mid = mma.mma_get_stats()
        log(f"  h2d copy-engine bytes {sum(mid['path_bytes'][:16]) - sum(before['path_bytes'][:16])}")
        # device -> host after a kernel that wrote the source on the same stream: queued right
        # behind it (CU path), and after it has finished (idle stream: the copy engines read
        # what the kernel wrote)
        host = mma.PinnedBuffer(n)
        for idle, val in ((False, 0x3C), (True, 0xC3)):
            host.array[:] = W.WEIGHT_POISON
            torch.cuda.synchronize()
            with torch.cuda.stream(stream):
                dst.fill_(val)
            if idle:
                stream.synchronize()
            b0 = mma.mma_get_stats()
            mma.mma_memcpy_async(host, dst, n, mma.MMA_D2H, stream)
            stream.synchronize()
            mma.mma_synchronize()
            b1 = mma.mma_get_stats()
            assert np.all(host.array == val), idle
            log(f"  d2h idle={idle} copy-engine bytes {sum(b1['path_bytes'][:16]) - sum(b0['path_bytes'][:16])}")
        assert mma.mma_get_stats()["failed_transfers"] == 0


def test_device_many_transfers_and_sync_copy():
    """Three times as many transfers as records, some on an idle stream and some queued behind
    others (both directions); then the blocking mma_memcpy. Every byte against the oracle."""
    n = (1 << 20) + 48
    count = 192
    src_np = np.ascontiguousarray(W.uniform_bytes(24, 0, 0, n * count))
    stream = torch.cuda.Stream()
    with session("both", **DEVICE, cu_whole_bytes=1, cu_whole_bytes_d2h=1):
        hsrc = mma.PinnedBuffer(n * count)
        hsrc.array[:] = src_np
        dmid = device_bytes(n * count, 0)
        hback = mma.PinnedBuffer(n * count)
        hback.array[:] = 0
        torch.cuda.synchronize()
        for i in range(count):
            if i % 8 == 0:
                stream.synchronize()  # idle: the copy engines take part
            mma.mma_memcpy_async(dmid.data_ptr() + i * n, hsrc.ptr + i * n, n, mma.MMA_H2D, stream)
        for i in range(count):
            mma.mma_memcpy_async(hback.ptr + i * n, dmid.data_ptr() + i * n, n, mma.MMA_D2H, stream)
        stream.synchronize()
        mma.mma_synchronize()
        assert np.array_equal(hback.array, src_np)
        stats = mma.mma_get_stats()
        assert stats["transfers"] >= 2 * count and stats["failed_transfers"] == 0
        # blocking copy
        m = (5 << 20) + 3
        back = mma.PinnedBuffer(m)
        back.array[:] = 0
        mma.mma_memcpy(back.ptr, dmid.data_ptr() + 7, m, mma.MMA_D2H)
        assert np.array_equal(back.array, src_np[7:7 + m])


@pytest.mark.parametrize("idle", [True, False])
def test_device_list_beyond_ring_replanned(idle):
    """A tensor list with more micro-tasks than a ring holds (10 x 481 at 64 KiB chunks) is planned
    again at twice the chunk size and stays under device control: byte-exact, copy engines
    included on an idle stream, and the engine thread never takes it."""
    sizes = [(30 << 20) + 1 + 4096 * k for k in range(10)]
    stream = torch.cuda.Stream()
    offs, off = [], 0
    for z in sizes:
        offs.append(off)
        off += (z + 255) // 256 * 256
    src_np = np.ascontiguousarray(W.uniform_bytes(23, 0, int(idle), off))
    with session("both", chunk_bytes=64 << 10, **DEVICE):
        src = mma.PinnedBuffer(off)
        src.array[:] = src_np
        dsts = [device_bytes(z, W.WEIGHT_POISON) for z in sizes]
        torch.cuda.synchronize()
        busy0 = mma.mma_get_stats()["engine_wall_busy_ns"]
        if not idle:
            _busy(stream)
        mma.mma_weights_load([(d, src.ptr + o, z) for d, o, z in zip(dsts, offs, sizes)], mma.MMA_H2D, stream)
        stream.synchronize()
        mma.mma_synchronize()
        stats = mma.mma_get_stats()
        for d, o, z in zip(dsts, offs, sizes):
            assert np.array_equal(to_host(d)[:z], ocopy.memcpy(np.full(z, W.WEIGHT_POISON, np.uint8), 0,
                                                                src_np[o:o + z], 0, z)), z
    assert stats["failed_transfers"] == 0
    assert sum(stats["path_bytes"]) == sum(sizes)
    assert stats["engine_wall_busy_ns"] == busy0, "the engine thread took the transfer"
    if idle:
        assert sum(stats["path_bytes"][:16]) > 0, "the copy engines took no share on an idle stream"
    else:
        assert sum(stats["path_bytes"][:16]) == 0


def test_device_beyond_ring_goes_to_engine_thread():
    """A KV fetch with more micro-tasks than a ring has entries (4400 single-piece tasks) is
    handed to the engine thread; byte-exact either way."""
    s = W.KVShape(layers=2, block_tokens=16, kv_heads=8, head_dim=128, elem_bytes=2,
                  gpu_num_blocks=1200, host_num_slots=1100, n_blocks=1100)
    hs, gb = W.kv_fetch_tables(s, cfg=3)
    stream = torch.cuda.Stream()
    with session("both", chunk_bytes=s.piece_bytes, **DEVICE):
        r = np.random.default_rng(32)
        pool = mma.PinnedBuffer(s.host_num_slots * s.slot_bytes)
        pool.array[:] = r.integers(0, 256, pool.nbytes, dtype=np.uint8)
        layers = [device_bytes(s.layer_bytes, W.GPU_POISON) for _ in range(s.layers)]
        before = [to_host(t).reshape(2, s.gpu_num_blocks, s.piece_bytes) for t in layers]
        torch.cuda.synchronize()
        busy0 = mma.mma_get_stats()["engine_wall_busy_ns"]
        mma.mma_kv_fetch(_kv_layout(s, okv.LAYOUT_PIECE), pool, layers, hs, gb, stream)
        stream.synchronize()
        mma.mma_synchronize()
        stats = mma.mma_get_stats()
        pool_v = pool.array.reshape(s.host_num_slots, s.slot_bytes)
        for l in range(s.layers):
            want = okv.kv_fetch_layer(pool_v, before[l], l, s.layers, hs, gb)
            assert np.array_equal(to_host(layers[l]).reshape(2, s.gpu_num_blocks, s.piece_bytes), want)
    assert stats["failed_transfers"] == 0
    assert stats["engine_wall_busy_ns"] > busy0, "the engine thread did not take the transfer"


@pytest.mark.parametrize("direction", [mma.MMA_H2D, mma.MMA_D2H])
def test_device_list_of_more_tensors_than_a_ring(direction):
    """A tensor list of 5000 small tensors has more micro-tasks than a ring at any chunk size (one
    per tensor): after the re-planning gives up it goes to the engine thread; byte-exact, gaps
    between destinations untouched."""
    sizes = [4096 + (k % 7) * 3 for k in range(5000)]
    src_offs, total = W.arena_offsets(sizes, 16)
    dst_offs, cur = [], 0
    for z in sizes:
        dst_offs.append(cur)
        cur += z + 48
    dtotal = cur
    src_np = np.ascontiguousarray(W.uniform_bytes(61, direction, 0, total))
    poison = np.full(dtotal, W.WEIGHT_POISON, np.uint8)
    stream = torch.cuda.Stream()
    with session("both", **DEVICE):
        torch.cuda.synchronize()
        busy0 = mma.mma_get_stats()["engine_wall_busy_ns"]
        if direction == mma.MMA_H2D:
            src = mma.PinnedBuffer(total)
            src.array[:] = src_np
            dst = from_host(poison)
            torch.cuda.synchronize()
            mma.mma_weights_load([(dst.data_ptr() + d, src.ptr + o, z) for d, o, z in zip(dst_offs, src_offs, sizes)],
                                 direction, stream)
            stream.synchronize()
            got = to_host(dst)
        else:
            src = from_host(src_np)
            dst = mma.PinnedBuffer(dtotal)
            dst.array[:] = poison
            torch.cuda.synchronize()
            mma.mma_weights_load([(dst.ptr + d, src.data_ptr() + o, z) for d, o, z in zip(dst_offs, src_offs, sizes)],
                                 direction, stream)
            stream.synchronize()
            got = dst.array.copy()
        mma.mma_synchronize()
        stats = mma.mma_get_stats()
    want = ocopy.tensor_list(poison, src_np, list(zip(dst_offs, src_offs, sizes)))
    assert np.array_equal(got, want)
    assert stats["failed_transfers"] == 0
    assert stats["engine_wall_busy_ns"] > busy0, "the engine thread did not take the transfer"
