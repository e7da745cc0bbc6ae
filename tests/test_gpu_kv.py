"""GPU parity of paged-KV fetch and offload against oracle.kv (byte-exact).

Small shapes cover several micro-tasks, CU sub-entries and SDMA staging slots,
ragged pieces (not a multiple of 16 bytes), every permutation of 4-entry tables,
and both paths; the full 64k-token workloads are checked layer by layer / over the
whole host pool.
"""
import itertools
import time

import numpy as np
import pytest
import torch

import workloads as W
from oracle import kv as okv

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2512_16056_amd as mma  # noqa: E402
from gpu_helpers import PATHS, device_bytes, log, session, to_host  # noqa: E402


def layout_of(s: W.KVShape):
    return mma.kv_layout(s.layers, s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes, s.gpu_num_blocks,
                         s.host_num_slots)


def _pool(s: W.KVShape, seed: int):
    buf = mma.PinnedBuffer(s.host_num_slots * s.slot_bytes)
    r = np.random.default_rng(seed)
    buf.array[:] = r.integers(0, 256, buf.nbytes, dtype=np.uint8)
    return buf


def _layers(s: W.KVShape, fill=None, seed=None):
    out = []
    for l in range(s.layers):
        t = device_bytes(s.layer_bytes, fill)
        if seed is not None:
            r = np.random.default_rng(seed + l)
            t.copy_(torch.from_numpy(r.integers(0, 256, s.layer_bytes, dtype=np.uint8)))
        out.append(t)
    return out


def _layer_views(s, layers):
    return [to_host(t).reshape(2, s.gpu_num_blocks, s.piece_bytes) for t in layers]


def check_fetch(s, pool, layers_before, layers_after, hs, gb):
    pool_v = pool.array.reshape(s.host_num_slots, s.slot_bytes)
    for l in range(s.layers):
        want = okv.kv_fetch_layer(pool_v, layers_before[l], l, s.layers, hs, gb)
        got = to_host(layers_after[l]).reshape(2, s.gpu_num_blocks, s.piece_bytes)
        assert np.array_equal(got, want), f"layer {l}"


SHAPES = {
    "small": W.small_kv_shape(),
    "ragged": W.KVShape(layers=3, block_tokens=1, kv_heads=1, head_dim=5, elem_bytes=2,
                        gpu_num_blocks=50, host_num_slots=40, n_blocks=37),
    "medium": W.KVShape(layers=4, block_tokens=16, kv_heads=2, head_dim=64, elem_bytes=2,
                        gpu_num_blocks=300, host_num_slots=256, n_blocks=200),
}


def _stream_of(kind):
    """None: the legacy default stream; else a stream of its own, on which nothing is pending once
    the caller has synchronised (the copy engines may then start before the kernel launch)."""
    return torch.cuda.Stream() if kind == "idle" else None


@pytest.mark.parametrize("stream", ["legacy", "idle"])
@pytest.mark.parametrize("chunk", [4096, 65536])
@pytest.mark.parametrize("shape", list(SHAPES))
@pytest.mark.parametrize("paths", list(PATHS))
def test_kv_fetch_small(paths, shape, chunk, stream):
    s = SHAPES[shape]
    log(f"kv fetch paths={paths} shape={shape} chunk={chunk} stream={stream}")
    hs, gb = W.kv_fetch_tables(s, cfg=3)
    st = _stream_of(stream)
    with session(paths, chunk_bytes=chunk, cu_sub_bytes=1024):
        pool = _pool(s, 1)
        layers = _layers(s, W.GPU_POISON)
        before = _layer_views(s, layers)
        torch.cuda.synchronize()
        mma.mma_kv_fetch(layout_of(s), pool, layers, hs, gb, st)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        stats = mma.mma_get_stats()
        check_fetch(s, pool, before, layers, hs, gb)
    assert stats["failed_transfers"] == 0
    assert sum(stats["path_bytes"]) == s.n_blocks * s.slot_bytes


@pytest.mark.parametrize("stream", ["legacy", "idle"])
@pytest.mark.parametrize("chunk", [4096, 65536])
@pytest.mark.parametrize("shape", list(SHAPES))
@pytest.mark.parametrize("paths", list(PATHS))
def test_kv_offload_small(paths, shape, chunk, stream):
    s = SHAPES[shape]
    log(f"kv offload paths={paths} shape={shape} chunk={chunk} stream={stream}")
    plan = W.kv_offload_plan(s, cfg=4)
    st = _stream_of(stream)
    with session(paths, chunk_bytes=chunk, cu_sub_bytes=1024):
        pool = _pool(s, 2)
        before = pool.array.copy()
        layers = _layers(s, seed=100)
        views = _layer_views(s, layers)
        torch.cuda.synchronize()
        mma.mma_kv_offload(layout_of(s), pool, layers, plan.src_blocks, plan.dest, st)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        want = okv.kv_offload(before.reshape(s.host_num_slots, -1), views, plan.src_blocks, plan.dest)
        assert np.array_equal(pool.array.reshape(s.host_num_slots, -1), want)


@pytest.mark.parametrize("merge", [1, 0])
def test_kv_sdma_merges_block_runs(merge):
    """With micro-tasks smaller than a block, one copy-engine command carries a block's run of
    consecutive pieces through staging (fetch) and back (offload); results stay byte-exact."""
    s = SHAPES["medium"]
    log(f"kv sdma merge={merge}")
    hs, gb = W.kv_fetch_tables(s, cfg=3)
    plan = W.kv_offload_plan(s, cfg=4)
    with session("sdma", chunk_bytes=2 * s.piece_bytes, cu_sub_bytes=1024, sdma_merge_tasks=merge):
        mma.mma_reset_stats()
        pool = _pool(s, 5)
        layers = _layers(s, W.GPU_POISON)
        before = _layer_views(s, layers)
        mma.mma_kv_fetch(layout_of(s), pool, layers, hs, gb)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        check_fetch(s, pool, before, layers, hs, gb)
        pool_before = pool.array.copy()
        views = _layer_views(s, layers)
        mma.mma_kv_offload(layout_of(s), pool, layers, plan.src_blocks, plan.dest)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        want = okv.kv_offload(pool_before.reshape(s.host_num_slots, -1), views, plan.src_blocks, plan.dest)
        assert np.array_equal(pool.array.reshape(s.host_num_slots, -1), want)
        stats = mma.mma_get_stats()
    sdma_tasks = sum(stats["path_tasks"][:16])
    log(f"  sdma tasks={sdma_tasks} commands={stats['sdma_commands']}")
    assert stats["failed_transfers"] == 0 and sdma_tasks > 0
    if merge == 1:
        assert stats["sdma_commands"] == sdma_tasks
    else:
        assert stats["sdma_commands"] < sdma_tasks


@pytest.mark.parametrize("paths", list(PATHS))
def test_kv_all_permutations(paths):
    s = W.KVShape(layers=2, block_tokens=2, kv_heads=1, head_dim=8, elem_bytes=2,
                  gpu_num_blocks=6, host_num_slots=4, n_blocks=4)
    with session(paths, chunk_bytes=64, cu_sub_bytes=256):
        pool = _pool(s, 3)
        src_layers = _layers(s, seed=7)
        src_views = _layer_views(s, src_layers)
        for perm in itertools.permutations(range(4)):
            hs = list(perm)
            gb = [5, 0, 3, 1]
            layers = _layers(s, W.GPU_POISON)
            before = _layer_views(s, layers)
            mma.mma_kv_fetch(layout_of(s), pool, layers, hs, gb)
            torch.cuda.synchronize()
            check_fetch(s, pool, before, layers, hs, gb)
            host = mma.PinnedBuffer(s.host_num_slots * s.slot_bytes)
            host.array[:] = W.HOST_FREE_POISON
            mma.mma_kv_offload(layout_of(s), host, src_layers, [2, 4, 0, 5], hs)
            torch.cuda.synchronize()
            want = okv.kv_offload(np.full((s.host_num_slots, s.slot_bytes), W.HOST_FREE_POISON, np.uint8),
                                  src_views, [2, 4, 0, 5], hs)
            assert np.array_equal(host.array.reshape(s.host_num_slots, -1), want), perm
            host.free()
        mma.mma_synchronize()


POOL_SHAPES = {
    **SHAPES,
    # pieces of 8 KiB + 48 bytes: one full span of the pool kernel and a short one
    "span_tail": W.KVShape(layers=2, block_tokens=16, kv_heads=1, head_dim=515, elem_bytes=1,
                           gpu_num_blocks=90, host_num_slots=80, n_blocks=70),
    # 32 KiB pieces, 3000 blocks: the launch's full 8192 workgroups, 12 spans each, so waves
    # move several spans and cross from one block into the next
    "wide": W.KVShape(layers=4, block_tokens=16, kv_heads=8, head_dim=128, elem_bytes=2,
                      gpu_num_blocks=3300, host_num_slots=3072, n_blocks=3000),
}


@pytest.mark.parametrize("route", ["pool", "ring"])
@pytest.mark.parametrize("shape", ["small", "ragged", "medium", "span_tail", "wide"])
def test_kv_device_pool(shape, route):
    """A pool in device memory: the same gather/scatter runs HBM -> HBM on the CU path -- one
    pool-kernel launch per transfer in the piece layout, or, when the pool kernel's table arena
    has no room (forced from the host), the transfer kernel's ring path."""
    s = POOL_SHAPES[shape]
    log(f"device pool {shape} route={route}: {s}")
    hs, gb = W.kv_fetch_tables(s, cfg=3)
    plan = W.kv_offload_plan(s, cfg=4)
    with session("both", chunk_bytes=4096):
        mma.mma_test_set_fault(mma.MMA_FAULT_POOL_NO_TABLE, 1 if route == "ring" else 0)
        r = np.random.default_rng(9)
        pool_np = r.integers(0, 256, s.host_num_slots * s.slot_bytes, dtype=np.uint8)
        pool = torch.from_numpy(pool_np.copy()).cuda()
        layers = _layers(s, W.GPU_POISON)
        before = _layer_views(s, layers)
        mma.mma_kv_fetch(layout_of(s), pool, layers, hs, gb)
        torch.cuda.synchronize()
        pv = pool_np.reshape(s.host_num_slots, s.slot_bytes)
        for l in range(s.layers):
            want = okv.kv_fetch_layer(pv, before[l], l, s.layers, hs, gb)
            assert np.array_equal(to_host(layers[l]).reshape(want.shape), want), l
        # offload back into the device pool
        src = _layers(s, seed=500)
        views = _layer_views(s, src)
        mma.mma_kv_offload(layout_of(s), pool, src, plan.src_blocks, plan.dest)
        torch.cuda.synchronize()
        want = okv.kv_offload(pv, views, plan.src_blocks, plan.dest)
        assert np.array_equal(to_host(pool).reshape(s.host_num_slots, -1), want)
        mma.mma_synchronize()
        st = mma.mma_get_stats()
        mma.mma_test_set_fault(mma.MMA_FAULT_POOL_NO_TABLE, 0)
    assert sum(st["path_bytes"][:16]) == 0 and st["failed_transfers"] == 0
    assert st["transfers"] == 2 and st["pool_launches"] == (2 if route == "pool" else 0), st


def test_kv_device_pool_queued_launches():
    """Pool launches queued back to back on two streams, with no synchronisation between them:
    each stream's fetches land in order (the last one wins) and every launch retires."""
    s = POOL_SHAPES["span_tail"]
    lay = layout_of(s)
    with session("both"):
        r = np.random.default_rng(21)
        pools = [r.integers(0, 256, s.host_num_slots * s.slot_bytes, dtype=np.uint8) for _ in range(3)]
        dpools = [torch.from_numpy(p.copy()).cuda() for p in pools]
        streams = [torch.cuda.Stream(), torch.cuda.Stream()]
        hs, gb = W.kv_fetch_tables(s, cfg=3)
        outs = []
        for k, st in enumerate(streams):
            layers = _layers(s, W.GPU_POISON)
            before = _layer_views(s, layers)
            torch.cuda.synchronize()
            lt = mma.layer_table(layers)
            for rep in range(6):  # pools 0, 1, 2, 0, 1, 2 (k = 0) or 1, 2, 0, ... (k = 1)
                mma.mma_kv_fetch(lay, dpools[(rep + k) % 3], lt, hs, gb, st)
            outs.append((layers, before, (5 + k) % 3))
        torch.cuda.synchronize()
        for layers, before, last in outs:
            pv = pools[last].reshape(s.host_num_slots, s.slot_bytes)
            for l in range(s.layers):
                want = okv.kv_fetch_layer(pv, before[l], l, s.layers, hs, gb)
                assert np.array_equal(to_host(layers[l]).reshape(want.shape), want), l
        mma.mma_synchronize()
        st = mma.mma_get_stats()
    assert st["transfers"] == 12 and st["failed_transfers"] == 0


def test_kv_rejects_bad_tables():
    s = SHAPES["small"]
    with session("both"):
        pool = _pool(s, 1)
        layers = _layers(s, 0)
        lay = layout_of(s)
        for hs, gb in [([0, 1], [3, 3]), ([0, s.host_num_slots], [0, 1]), ([0, 1], [0, s.gpu_num_blocks]),
                       ([-1, 1], [0, 1])]:
            with pytest.raises(mma.MMAError) as e:
                mma.mma_kv_fetch(lay, pool, layers, hs, gb)
            assert e.value.name == "MMA_ERR_INVALID_ARG"
        with pytest.raises(mma.MMAError):  # duplicate destination slot on offload
            mma.mma_kv_offload(lay, pool, layers, [0, 1], [2, 2])
        # layouts whose pool or layer size wraps 64 bits (to 0, which every range check would pass):
        # rejected before anything else, with tables that are in range
        for f in [(256, 1 << 16, 1 << 16, 1, 1, 1, 1 << 23), (1, 1 << 16, 1 << 16, 1, 1, 1 << 31, 1)]:
            for call in (mma.mma_kv_fetch, mma.mma_kv_offload, mma.mma_kv_fetch_noalloc):
                with pytest.raises(mma.MMAError) as e:
                    call(mma.kv_layout(*f), pool, [layers[0]] * f[0], [0], [0])
                assert e.value.name == "MMA_ERR_INVALID_ARG", (f, call)
        mma.mma_kv_fetch(lay, pool, layers, [], [])  # empty: no-op
        torch.cuda.synchronize()


# ----------------------------------------------------------------------------- x-packed GPU block layout
XP = okv.LAYOUT_XPACKED
XP_SHAPES = {
    # block_tokens * elem_bytes and head_dim * elem_bytes are multiples of 16
    "bf16": W.KVShape(layers=2, block_tokens=16, kv_heads=2, head_dim=16, elem_bytes=2,
                      gpu_num_blocks=40, host_num_slots=32, n_blocks=24),
    "fp8": W.KVShape(layers=3, block_tokens=16, kv_heads=3, head_dim=32, elem_bytes=1,
                     gpu_num_blocks=50, host_num_slots=40, n_blocks=30),
    "fp32": W.KVShape(layers=2, block_tokens=8, kv_heads=5, head_dim=16, elem_bytes=4,
                      gpu_num_blocks=33, host_num_slots=30, n_blocks=29),
    "fp64": W.KVShape(layers=1, block_tokens=2, kv_heads=3, head_dim=8, elem_bytes=8,
                      gpu_num_blocks=20, host_num_slots=20, n_blocks=17),
    "llama": W.KVShape(layers=4, block_tokens=16, kv_heads=8, head_dim=128, elem_bytes=2,
                       gpu_num_blocks=300, host_num_slots=256, n_blocks=200),
}


def xp_layout_of(s: W.KVShape):
    return mma.kv_layout(s.layers, s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes, s.gpu_num_blocks,
                         s.host_num_slots, mma.MMA_KV_LAYOUT_XPACKED)


def _geom(s: W.KVShape):
    return (s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes)


@pytest.mark.parametrize("chunk", [4096, 1 << 21])
@pytest.mark.parametrize("shape", list(XP_SHAPES))
@pytest.mark.parametrize("paths", list(PATHS))
def test_kv_xpacked_fetch(paths, shape, chunk):
    s = XP_SHAPES[shape]
    log(f"kv fetch x-packed paths={paths} shape={shape} chunk={chunk}")
    hs, gb = W.kv_fetch_tables(s, cfg=3)
    with session(paths, chunk_bytes=chunk, cu_sub_bytes=1024):
        pool = _pool(s, 5)
        layers = _layers(s, W.GPU_POISON)
        before = _layer_views(s, layers)
        mma.mma_kv_fetch(xp_layout_of(s), pool, layers, hs, gb)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        stats = mma.mma_get_stats()
        pool_v = pool.array.reshape(s.host_num_slots, s.slot_bytes)
        for l in range(s.layers):
            want = okv.kv_fetch_layer(pool_v, before[l], l, s.layers, hs, gb, XP, _geom(s))
            got = to_host(layers[l]).reshape(2, s.gpu_num_blocks, s.piece_bytes)
            assert np.array_equal(got, want), f"layer {l}"
    assert stats["failed_transfers"] == 0
    assert sum(stats["path_bytes"]) == s.n_blocks * s.slot_bytes


@pytest.mark.parametrize("chunk", [4096, 1 << 21])
@pytest.mark.parametrize("shape", list(XP_SHAPES))
@pytest.mark.parametrize("paths", list(PATHS))
def test_kv_xpacked_offload(paths, shape, chunk):
    s = XP_SHAPES[shape]
    log(f"kv offload x-packed paths={paths} shape={shape} chunk={chunk}")
    plan = W.kv_offload_plan(s, cfg=4)
    with session(paths, chunk_bytes=chunk, cu_sub_bytes=1024):
        pool = _pool(s, 6)
        before = pool.array.copy()
        layers = _layers(s, seed=200)
        views = _layer_views(s, layers)
        mma.mma_kv_offload(xp_layout_of(s), pool, layers, plan.src_blocks, plan.dest)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        want = okv.kv_offload(before.reshape(s.host_num_slots, -1), views, plan.src_blocks, plan.dest, XP, _geom(s))
        assert np.array_equal(pool.array.reshape(s.host_num_slots, -1), want)


@pytest.mark.parametrize("shape", ["bf16", "llama"])
def test_kv_xpacked_device_pool_roundtrip(shape):
    """An HBM-resident pool (CU gather/scatter in HBM) with the x-packed layout: fetch, then offload
    the same blocks into other slots; both against the oracle."""
    s = XP_SHAPES[shape]
    hs, gb = W.kv_fetch_tables(s, cfg=3)
    with session("both", chunk_bytes=4096):
        r = np.random.default_rng(8)
        pool_np = r.integers(0, 256, s.host_num_slots * s.slot_bytes, dtype=np.uint8)
        dpool = torch.from_numpy(pool_np.copy()).cuda()
        layers = _layers(s, W.GPU_POISON)
        before = _layer_views(s, layers)
        mma.mma_kv_fetch(xp_layout_of(s), dpool, layers, hs, gb)
        torch.cuda.synchronize()
        pv = pool_np.reshape(s.host_num_slots, s.slot_bytes)
        for l in range(s.layers):
            want = okv.kv_fetch_layer(pv, before[l], l, s.layers, hs, gb, XP, _geom(s))
            assert np.array_equal(to_host(layers[l]).reshape(2, s.gpu_num_blocks, s.piece_bytes), want), l
        dest = np.roll(hs, 1).astype(np.int32)
        views = _layer_views(s, layers)
        mma.mma_kv_offload(xp_layout_of(s), dpool, layers, gb, dest)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        want = okv.kv_offload(pv, views, gb, dest, XP, _geom(s))
        assert np.array_equal(to_host(dpool).reshape(s.host_num_slots, -1), want)


def test_kv_xpacked_rejects_unsupported_geometry():
    with session("both"):
        for s in [W.KVShape(layers=1, block_tokens=16, kv_heads=1, head_dim=12, elem_bytes=2,
                            gpu_num_blocks=4, host_num_slots=4, n_blocks=2),   # head row of 24 bytes
                  W.KVShape(layers=1, block_tokens=4, kv_heads=1, head_dim=16, elem_bytes=2,
                            gpu_num_blocks=4, host_num_slots=4, n_blocks=2),   # 8-byte token column
                  W.KVShape(layers=1, block_tokens=16, kv_heads=1, head_dim=24, elem_bytes=3,
                            gpu_num_blocks=4, host_num_slots=4, n_blocks=2),   # 3-byte elements
                  W.KVShape(layers=1, block_tokens=256, kv_heads=1, head_dim=128, elem_bytes=2,
                            gpu_num_blocks=4, host_num_slots=4, n_blocks=2)]:  # one head > the LDS tile
            pool = _pool(s, 1)
            layers = _layers(s, 0)
            with pytest.raises(mma.MMAError) as e:
                mma.mma_kv_fetch(xp_layout_of(s), pool, layers, [0, 1], [0, 1])
            assert e.value.name == "MMA_ERR_INVALID_ARG"
            pool.free()
        s = XP_SHAPES["bf16"]
        pool = _pool(s, 1)
        layers = _layers(s, 0)
        bad = mma.kv_layout(s.layers, s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes, s.gpu_num_blocks,
                            s.host_num_slots, 7)
        with pytest.raises(mma.MMAError) as e:
            mma.mma_kv_fetch(bad, pool, layers, [0], [0])
        assert e.value.name == "MMA_ERR_INVALID_ARG"
        torch.cuda.synchronize()


# ----------------------------------------------------------------------------- head-major GPU block layout
HND = okv.LAYOUT_HND
HND_SHAPES = {
    # head_dim * elem_bytes is a multiple of 16; any token count
    "bf16": W.KVShape(layers=2, block_tokens=16, kv_heads=2, head_dim=16, elem_bytes=2,
                      gpu_num_blocks=40, host_num_slots=32, n_blocks=24),
    "fp8": W.KVShape(layers=3, block_tokens=16, kv_heads=3, head_dim=32, elem_bytes=1,
                     gpu_num_blocks=50, host_num_slots=40, n_blocks=30),
    "fp32_5tok": W.KVShape(layers=2, block_tokens=5, kv_heads=3, head_dim=4, elem_bytes=4,
                           gpu_num_blocks=33, host_num_slots=30, n_blocks=29),
    "one_head": W.KVShape(layers=2, block_tokens=16, kv_heads=1, head_dim=64, elem_bytes=2,
                          gpu_num_blocks=20, host_num_slots=20, n_blocks=17),
    "llama": W.KVShape(layers=4, block_tokens=16, kv_heads=8, head_dim=128, elem_bytes=2,
                       gpu_num_blocks=300, host_num_slots=256, n_blocks=200),
}


def hnd_layout_of(s: W.KVShape):
    return mma.kv_layout(s.layers, s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes, s.gpu_num_blocks,
                         s.host_num_slots, mma.MMA_KV_LAYOUT_HND)


@pytest.mark.parametrize("chunk", [4096, 1 << 21])
@pytest.mark.parametrize("shape", list(HND_SHAPES))
@pytest.mark.parametrize("paths", list(PATHS))
def test_kv_hnd_fetch(paths, shape, chunk):
    s = HND_SHAPES[shape]
    log(f"kv fetch head-major paths={paths} shape={shape} chunk={chunk}")
    hs, gb = W.kv_fetch_tables(s, cfg=3)
    with session(paths, chunk_bytes=chunk, cu_sub_bytes=1024):
        pool = _pool(s, 9)
        layers = _layers(s, W.GPU_POISON)
        before = _layer_views(s, layers)
        mma.mma_kv_fetch(hnd_layout_of(s), pool, layers, hs, gb)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        stats = mma.mma_get_stats()
        pool_v = pool.array.reshape(s.host_num_slots, s.slot_bytes)
        for l in range(s.layers):
            want = okv.kv_fetch_layer(pool_v, before[l], l, s.layers, hs, gb, HND, _geom(s))
            got = to_host(layers[l]).reshape(2, s.gpu_num_blocks, s.piece_bytes)
            assert np.array_equal(got, want), f"layer {l}"
    assert stats["failed_transfers"] == 0
    assert sum(stats["path_bytes"]) == s.n_blocks * s.slot_bytes


@pytest.mark.parametrize("chunk", [4096, 1 << 21])
@pytest.mark.parametrize("shape", list(HND_SHAPES))
@pytest.mark.parametrize("paths", list(PATHS))
def test_kv_hnd_offload(paths, shape, chunk):
    s = HND_SHAPES[shape]
    log(f"kv offload head-major paths={paths} shape={shape} chunk={chunk}")
    plan = W.kv_offload_plan(s, cfg=4)
    with session(paths, chunk_bytes=chunk, cu_sub_bytes=1024):
        pool = _pool(s, 10)
        before = pool.array.copy()
        layers = _layers(s, seed=300)
        views = _layer_views(s, layers)
        mma.mma_kv_offload(hnd_layout_of(s), pool, layers, plan.src_blocks, plan.dest)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        want = okv.kv_offload(before.reshape(s.host_num_slots, -1), views, plan.src_blocks, plan.dest, HND, _geom(s))
        assert np.array_equal(pool.array.reshape(s.host_num_slots, -1), want)


HND_POOL_SHAPES = {
    **HND_SHAPES,
    # 9000 blocks of 512-byte pieces: a pool launch of 7200 workgroups with 5 pieces each, so
    # waves move several pieces and cross from one block into the next
    "many_small": W.KVShape(layers=2, block_tokens=16, kv_heads=1, head_dim=16, elem_bytes=2,
                            gpu_num_blocks=9500, host_num_slots=9216, n_blocks=9000),
}


@pytest.mark.parametrize("route", ["pool", "ring"])
@pytest.mark.parametrize("shape", ["fp32_5tok", "llama", "many_small"])
def test_kv_hnd_device_pool_roundtrip(shape, route):
    """An HBM-resident pool with the head-major layout (one pool-kernel launch per call, or the
    ring path when the table arena has no room, forced from the host): fetch, then offload the
    same blocks into other slots; both against the oracle."""
    s = HND_POOL_SHAPES[shape]
    log(f"head-major device pool {shape} route={route}")
    hs, gb = W.kv_fetch_tables(s, cfg=3)
    with session("both", chunk_bytes=4096):
        mma.mma_test_set_fault(mma.MMA_FAULT_POOL_NO_TABLE, 1 if route == "ring" else 0)
        r = np.random.default_rng(18)
        pool_np = r.integers(0, 256, s.host_num_slots * s.slot_bytes, dtype=np.uint8)
        dpool = torch.from_numpy(pool_np.copy()).cuda()
        layers = _layers(s, W.GPU_POISON)
        before = _layer_views(s, layers)
        mma.mma_kv_fetch(hnd_layout_of(s), dpool, layers, hs, gb)
        torch.cuda.synchronize()
        pv = pool_np.reshape(s.host_num_slots, s.slot_bytes)
        for l in range(s.layers):
            want = okv.kv_fetch_layer(pv, before[l], l, s.layers, hs, gb, HND, _geom(s))
            assert np.array_equal(to_host(layers[l]).reshape(2, s.gpu_num_blocks, s.piece_bytes), want), l
        dest = np.roll(hs, 1).astype(np.int32)
        views = _layer_views(s, layers)
        mma.mma_kv_offload(hnd_layout_of(s), dpool, layers, gb, dest)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        want = okv.kv_offload(pv, views, gb, dest, HND, _geom(s))
        assert np.array_equal(to_host(dpool).reshape(s.host_num_slots, -1), want)
        st = mma.mma_get_stats()
        mma.mma_test_set_fault(mma.MMA_FAULT_POOL_NO_TABLE, 0)
    assert st["failed_transfers"] == 0
    assert st["transfers"] == 2 and st["pool_launches"] == (2 if route == "pool" else 0), st


def test_kv_hnd_rejects_unsupported_geometry():
    with session("both"):
        s = W.KVShape(layers=1, block_tokens=16, kv_heads=2, head_dim=12, elem_bytes=2,
                      gpu_num_blocks=4, host_num_slots=4, n_blocks=2)  # head row of 24 bytes
        pool = _pool(s, 1)
        layers = _layers(s, 0)
        with pytest.raises(mma.MMAError) as e:
            mma.mma_kv_fetch(hnd_layout_of(s), pool, layers, [0, 1], [0, 1])
        assert e.value.name == "MMA_ERR_INVALID_ARG"
        pool.free()
        s = HND_SHAPES["bf16"]
        big = mma.PinnedBuffer(s.host_num_slots * s.slot_bytes + 64)  # a pool 8 bytes off alignment
        layers = _layers(s, 0)
        with pytest.raises(mma.MMAError) as e:
            mma.mma_kv_fetch(hnd_layout_of(s), big.ptr + 8, layers, [0], [0])
        assert e.value.name == "MMA_ERR_INVALID_ARG"
        big.free()
        torch.cuda.synchronize()


@pytest.mark.parametrize("gpu_layout", [0, 1, 2])
def test_kv_whole_transfers(gpu_layout):
    """Default size limits: KV fetches of up to 24 MiB (12 blocks of the 64k workload's shape) and
    offloads of up to 8 MiB (4 blocks) are taken whole by the CU path -- one self-contained launch,
    no copy engine -- and larger ones use every path; all three GPU block layouts, every byte
    against the oracle."""
    LAYOUTS = (okv.LAYOUT_PIECE, okv.LAYOUT_XPACKED, okv.LAYOUT_HND)
    base = W.KV64K
    with session("both", cu_whole_bytes=0, cu_whole_bytes_d2h=0):  # 0: the default limits
        for n in (1, 4, 5, 12, 13):
            s = W.KVShape(layers=base.layers, block_tokens=base.block_tokens, kv_heads=base.kv_heads,
                          head_dim=base.head_dim, elem_bytes=base.elem_bytes, gpu_num_blocks=20,
                          host_num_slots=16, n_blocks=n)
            log(f"whole kv layout={gpu_layout} blocks={n}")
            geom = _geom(s)
            lay = mma.kv_layout(s.layers, s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes, s.gpu_num_blocks,
                                s.host_num_slots, gpu_layout)
            r = np.random.default_rng(60 + n)
            hs = r.permutation(s.host_num_slots)[:n].astype(np.int32)
            gb = r.permutation(s.gpu_num_blocks)[:n].astype(np.int32)
            pool = _pool(s, 70 + n)
            layers = _layers(s, W.GPU_POISON)
            before = _layer_views(s, layers)
            mma.mma_synchronize()
            st0 = mma.mma_get_stats()
            mma.mma_kv_fetch(lay, pool, layers, hs, gb)
            torch.cuda.synchronize()
            mma.mma_synchronize()
            st1 = mma.mma_get_stats()
            pool_v = pool.array.reshape(s.host_num_slots, s.slot_bytes)
            for l in range(s.layers):
                want = okv.kv_fetch_layer(pool_v, before[l], l, s.layers, hs, gb, LAYOUTS[gpu_layout], geom)
                got = to_host(layers[l]).reshape(2, s.gpu_num_blocks, s.piece_bytes)
                assert np.array_equal(got, want), (n, l)
            eng = sum(st1["path_bytes"][:16]) - sum(st0["path_bytes"][:16])
            assert (eng == 0) == (n <= 12), (n, eng)
            dest = np.roll(hs, 1).astype(np.int32)
            views = _layer_views(s, layers)
            pool_before = pool.array.copy()
            mma.mma_kv_offload(lay, pool, layers, gb, dest)
            torch.cuda.synchronize()
            mma.mma_synchronize()
            st2 = mma.mma_get_stats()
            want = okv.kv_offload(pool_before.reshape(s.host_num_slots, -1), views, gb, dest, LAYOUTS[gpu_layout],
                                  geom)
            assert np.array_equal(pool.array.reshape(s.host_num_slots, -1), want), n
            eng = sum(st2["path_bytes"][:16]) - sum(st1["path_bytes"][:16])
            assert (eng == 0) == (n <= 4), (n, eng)
            assert st2["failed_transfers"] == 0
            pool.free()


def _fill_pool_c3(pool: np.ndarray, s: W.KVShape, hs: np.ndarray):
    v = pool.reshape(s.host_num_slots, s.slot_bytes)
    for i in range(s.n_blocks):
        v[hs[i]] = W.kv_block_bytes(3, i, s)


@pytest.mark.slow
def test_kv_fetch_64k_full():
    """The 64k-token KV fetch workload (8 GiB), in the configuration the benchmark times."""
    s = W.KV64K
    hs, gb = W.kv_fetch_tables(s, cfg=3)
    with session("both"):
        pool = mma.PinnedBuffer(s.host_num_slots * s.slot_bytes)
        t0 = time.time()
        _fill_pool_c3(pool.array, s, hs)
        log(f"  pool generated in {time.time() - t0:.1f}s")
        layers = _layers(s, W.GPU_POISON)
        poison = np.full((2, s.gpu_num_blocks, s.piece_bytes), W.GPU_POISON, np.uint8)
        mma.mma_kv_fetch(layout_of(s), pool, layers, hs, gb)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        stats = mma.mma_get_stats()
        log(f"  path bytes: cu={stats['path_bytes'][16]} sdma={stats['path_bytes'][:4]}")
        pool_v = pool.array.reshape(s.host_num_slots, s.slot_bytes)
        for l in range(s.layers):
            want = okv.kv_fetch_layer(pool_v, poison, l, s.layers, hs, gb)
            got = to_host(layers[l]).reshape(2, s.gpu_num_blocks, s.piece_bytes)
            assert np.array_equal(got, want), f"layer {l}"
        pool.free()
    assert stats["failed_transfers"] == 0


@pytest.mark.slow
def test_kv_offload_64k_full():
    """KV offload of a 50% dirty subset (4 GiB) into free host slots; the whole 8 GiB pool is verified."""
    s = W.KV64K
    plan = W.kv_offload_plan(s, cfg=4)
    with session("both"):
        pool = mma.PinnedBuffer(s.host_num_slots * s.slot_bytes)
        pv = pool.array.reshape(s.host_num_slots, s.slot_bytes)
        for slot in plan.occupied:
            pv[slot] = W.kv_occupied_bytes(4, int(slot), s)
        pv[plan.free] = W.HOST_FREE_POISON
        before = pv.copy()
        layers = _layers(s, W.GPU_POISON)
        # logical block i lives at GPU block gpu_blocks_all[i]
        blocks = np.empty((s.n_blocks, s.layers, 2, s.piece_bytes), np.uint8)
        for i in range(s.n_blocks):
            blocks[i] = W.kv_block_bytes(4, i, s).reshape(s.layers, 2, s.piece_bytes)
        for l in range(s.layers):
            lay_np = np.full((2, s.gpu_num_blocks, s.piece_bytes), W.GPU_POISON, np.uint8)
            lay_np[:, plan.gpu_blocks_all] = blocks[:, l].transpose(1, 0, 2)
            layers[l].copy_(torch.from_numpy(lay_np.reshape(-1)))
        del blocks
        views = _layer_views(s, layers)
        mma.mma_kv_offload(layout_of(s), pool, layers, plan.src_blocks, plan.dest)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        want = okv.kv_offload(before, views, plan.src_blocks, plan.dest)
        assert np.array_equal(pv, want)
        pool.free()


@pytest.mark.slow
@pytest.mark.parametrize("gpu_layout", ["xpacked", "hnd"])
def test_kv_xpacked_fetch_offload_64k(gpu_layout):
    """The 64k-token KV fetch (8 GiB) into the x-packed or head-major GPU layout, in the
    configuration the benchmark times, then the offload of every fetched block into the host slots
    in reverse order (a poisoned pool). Every layer of the GPU cache (all 4096 fetched blocks and the
    untouched ones) and the whole 8 GiB pool after the offload are compared with the oracle."""
    LAY, GL = ((XP, mma.MMA_KV_LAYOUT_XPACKED) if gpu_layout == "xpacked"
               else (okv.LAYOUT_HND, mma.MMA_KV_LAYOUT_HND))
    s = W.KV64K
    hs, gb = W.kv_fetch_tables(s, cfg=3)
    geom = _geom(s)
    with session("both", cu_whole_bytes=0):
        pool = mma.PinnedBuffer(s.host_num_slots * s.slot_bytes)
        _fill_pool_c3(pool.array, s, hs)
        layers = _layers(s, W.GPU_POISON)
        lay = mma.kv_layout(s.layers, s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes, s.gpu_num_blocks,
                            s.host_num_slots, GL)
        mma.mma_kv_fetch(lay, pool, layers, hs, gb)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        pool_v = pool.array.reshape(s.host_num_slots, s.slot_bytes)
        poison = np.full((2, s.gpu_num_blocks, s.piece_bytes), W.GPU_POISON, np.uint8)
        for l in range(s.layers):
            want = okv.kv_fetch_layer(pool_v, poison, l, s.layers, hs, gb, LAY, geom)
            got = to_host(layers[l]).reshape(2, s.gpu_num_blocks, s.piece_bytes)
            assert np.array_equal(got, want), l
            if l % 8 == 7:
                log(f"  {gpu_layout} fetch: layers 0..{l} match the oracle")
        views = _layer_views(s, layers)
        dest = hs[::-1].copy()
        pool.array[:] = W.HOST_FREE_POISON
        before = np.full((s.host_num_slots, s.slot_bytes), W.HOST_FREE_POISON, np.uint8)
        mma.mma_kv_offload(lay, pool, layers, gb, dest)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        want = okv.kv_offload(before, views, gb, dest, LAY, geom)
        del before, views
        assert np.array_equal(pool_v, want)
        log(f"  {gpu_layout} offload: the whole pool matches the oracle")
        del want
        st = mma.mma_get_stats()
        pool.free()
    assert st["failed_transfers"] == 0
