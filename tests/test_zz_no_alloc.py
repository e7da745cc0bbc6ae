"""The KV fetch that allocates nothing (mma_kv_fetch_noalloc), through the C ABI.

Its output is compared byte for byte with mma_kv_fetch's on the same inputs, and
both with the oracle, on two calls in a row, the second with fewer blocks (the
scratch array keeps the first call's table and counter; the second must not see
them), in each GPU block layout. Sizes beyond its fixed table are refused with
nothing enqueued.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import kv as okv

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2512_16056_amd as mma  # noqa: E402
from gpu_helpers import device_bytes, log, session, to_host  # noqa: E402

LAYOUTS = {"piece": okv.LAYOUT_PIECE, "hnd": okv.LAYOUT_HND, "xpacked": okv.LAYOUT_XPACKED}
# 1000 blocks: three table chunks (448 entries each), the last one ragged
SHAPE = W.KVShape(layers=4, block_tokens=16, kv_heads=2, head_dim=64, elem_bytes=2,
                  gpu_num_blocks=1200, host_num_slots=1100, n_blocks=1000)


def _tables(s: W.KVShape, n: int, cfg: int):
    hs = W.rng(cfg, W.TAG_HOST_PERM, 0).permutation(s.host_num_slots)[:n].astype(np.int32)
    gb = W.rng(cfg, W.TAG_GPU_PERM, 0).permutation(s.gpu_num_blocks)[:n].astype(np.int32)
    return hs, gb


@pytest.mark.parametrize("layout", list(LAYOUTS))
def test_noalloc_fetch_matches_kv_fetch(layout):
    s = SHAPE
    lay_id = LAYOUTS[layout]
    geom = (s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes)
    with session("both", cu_whole_bytes=0, cu_whole_bytes_d2h=0):
        lay = mma.kv_layout(s.layers, s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes, s.gpu_num_blocks,
                            s.host_num_slots, lay_id)
        pool = mma.PinnedBuffer(s.host_num_slots * s.slot_bytes)
        pool.array[:] = np.frombuffer(W.rng(17, W.TAG_DATA, lay_id).bytes(pool.nbytes), dtype=np.uint8)
        pv = pool.array.reshape(s.host_num_slots, s.slot_bytes)
        poison = np.full((2, s.gpu_num_blocks, s.piece_bytes), W.GPU_POISON, np.uint8)
        for call, n in enumerate((s.n_blocks, 7)):  # the second call is smaller
            log(f"noalloc fetch layout={layout} call={call} blocks={n}")
            hs, gb = _tables(s, n, cfg=20 + call)
            ref = [device_bytes(s.layer_bytes, W.GPU_POISON) for _ in range(s.layers)]
            got = [device_bytes(s.layer_bytes, W.GPU_POISON) for _ in range(s.layers)]
            mma.mma_kv_fetch(lay, pool, ref, hs, gb)
            mma.mma_kv_fetch_noalloc(lay, pool, got, hs, gb)
            torch.cuda.synchronize()
            mma.mma_synchronize()
            for l in range(s.layers):
                r = to_host(ref[l])
                g = to_host(got[l])
                assert np.array_equal(g, r), f"layer {l}: no-alloc fetch differs from mma_kv_fetch"
                want = okv.kv_fetch_layer(pv, poison, l, s.layers, hs, gb, layout=lay_id, geom=geom)
                assert np.array_equal(g.reshape(want.shape), want), f"layer {l}: differs from the oracle"
        pool.free()


def test_noalloc_fetch_limits():
    s = W.KVShape(layers=1, block_tokens=1, kv_heads=1, head_dim=8, elem_bytes=2,
                  gpu_num_blocks=70000, host_num_slots=70000, n_blocks=65537)
    with session("both"):
        lay = mma.kv_layout(s.layers, s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes, s.gpu_num_blocks,
                            s.host_num_slots)
        pool = mma.PinnedBuffer(s.host_num_slots * s.slot_bytes)
        pool.array[:] = 7
        layers = [device_bytes(s.layer_bytes, W.GPU_POISON)]
        hs = np.arange(s.n_blocks, dtype=np.int32)
        with pytest.raises(mma.MMAError) as e:  # one block past the fixed table
            mma.mma_kv_fetch_noalloc(lay, pool, layers, hs, hs)
        assert e.value.status == mma.MMA_ERR_INVALID_ARG
        with pytest.raises(mma.MMAError) as e:  # a duplicate destination, as for mma_kv_fetch
            mma.mma_kv_fetch_noalloc(lay, pool, layers, np.array([1, 2], np.int32), np.array([5, 5], np.int32))
        assert e.value.status == mma.MMA_ERR_INVALID_ARG
        torch.cuda.synchronize()
        assert np.all(to_host(layers[0]) == W.GPU_POISON)  # nothing was enqueued
        # the largest call it takes: 65536 one-token blocks
        hs = W.rng(21, W.TAG_HOST_PERM, 0).permutation(s.host_num_slots)[:65536].astype(np.int32)
        gb = W.rng(21, W.TAG_GPU_PERM, 0).permutation(s.gpu_num_blocks)[:65536].astype(np.int32)
        mma.mma_kv_fetch_noalloc(lay, pool, layers, hs, gb)
        torch.cuda.synchronize()
        pv = pool.array.reshape(s.host_num_slots, s.slot_bytes)
        want = okv.kv_fetch_layer(pv, np.full((2, s.gpu_num_blocks, s.piece_bytes), W.GPU_POISON, np.uint8),
                                  0, 1, hs, gb)
        assert np.array_equal(to_host(layers[0]).reshape(want.shape), want)
        pool.free()
