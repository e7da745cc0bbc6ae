"""Seeded random mixes of every transfer kind in flight at once, checked against the oracle.

One schedule of ~150 operations is drawn from a seed: single copies and tensor lists in both
directions (1 byte to 12 MiB, odd offsets, self-contained launches, whole-CU transfers, early
starts on idle streams, multipath transfers with merged copy-engine commands) and paged-KV
fetches and offloads in all three GPU block layouts, a third of them with the pool in HBM (pool
launches in the piece and head-major layouts, the ring for x-packed), issued in random order over four streams
(including the legacy default stream). Every operation writes its own destination range and
reads a read-only source, so the final state is unique whatever the interleaving; each
destination (and the poison around it) is compared byte-exact with oracle.copy / oracle.kv.
"""
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
from gpu_helpers import log, session, to_host  # noqa: E402

POISON = 0xEE
KV_SHAPES = [
    W.KVShape(layers=2, block_tokens=16, kv_heads=2, head_dim=64, elem_bytes=2, gpu_num_blocks=24, host_num_slots=20,
              n_blocks=12),
    W.KVShape(layers=3, block_tokens=16, kv_heads=4, head_dim=32, elem_bytes=1, gpu_num_blocks=30, host_num_slots=30,
              n_blocks=25),
    W.KVShape(layers=1, block_tokens=8, kv_heads=1, head_dim=16, elem_bytes=4, gpu_num_blocks=9, host_num_slots=7,
              n_blocks=7),
]


class Bump:
    """Disjoint 256-byte-aligned ranges of one buffer."""

    def __init__(self, size):
        self.size, self.at = size, 0

    def take(self, n):
        o = self.at
        self.at = (self.at + n + 255 + 64) & ~255  # 64 bytes of untouched poison between ranges
        assert self.at <= self.size, "schedule larger than the arena"
        return o


def _size(r):
    # log-uniform from 1 B to 12 MiB, with extra weight on the boundaries of the whole-CU limits
    if r.random() < 0.15:
        return int(r.choice([(8 << 20) - 1, 8 << 20, (8 << 20) + 1, 3 << 20, (3 << 20) + 16, 48 * 16384]))
    return int(np.exp(r.uniform(0, np.log(12 << 20))))


@pytest.mark.parametrize("control", [mma.MMA_CONTROL_HOST, mma.MMA_CONTROL_DEVICE])
@pytest.mark.parametrize("seed", [1, 2])
def test_random_mixed_schedule(seed, control):
    r = np.random.default_rng(seed)
    HOST, DEV = 256 << 20, 256 << 20
    with session("both", cu_whole_bytes=0, cu_whole_bytes_d2h=0, chunk_bytes=1 << 20, control=control):
        src_h = mma.PinnedBuffer(32 << 20)                   # read-only host source
        src_h.array[:] = r.integers(0, 256, src_h.nbytes, dtype=np.uint8)
        src_d_np = r.integers(0, 256, 32 << 20, dtype=np.uint8)
        src_d = torch.from_numpy(src_d_np.copy()).cuda()      # read-only device source
        dst_h = mma.PinnedBuffer(HOST)
        dst_h.array[:] = POISON
        dst_d = torch.full((DEV,), POISON, dtype=torch.uint8, device="cuda")
        bh, bd = Bump(HOST), Bump(DEV)
        streams = [torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream(), None]  # None: legacy default
        expect = []  # (side, destination offset, source offset, bytes)
        kv_jobs = []
        torch.cuda.synchronize()
        n_ops = 150
        for op in range(n_ops):
            st = streams[int(r.integers(len(streams)))]
            kind = r.choice(["copy", "copy", "list", "kv"], p=[0.35, 0.25, 0.25, 0.15])
            d2h = bool(r.integers(2))
            if kind == "copy":
                n = _size(r)
                so = int(r.integers(0, (32 << 20) - n)) if n < (32 << 20) else 0
                if d2h:
                    do = bh.take(n) + int(r.integers(0, 16))
                    mma.mma_memcpy_async(dst_h.ptr + do, src_d.data_ptr() + so, n, mma.MMA_D2H, st)
                    expect.append(("h", do, so, n))
                else:
                    do = bd.take(n) + int(r.integers(0, 16))
                    mma.mma_memcpy_async(dst_d.data_ptr() + do, src_h.ptr + so, n, mma.MMA_H2D, st)
                    expect.append(("d", do, so, n))
            elif kind == "list":
                cnt = int(r.integers(2, 61))
                items = []
                for _ in range(cnt):
                    n = _size(r) // 8 + int(r.integers(0, 3))
                    so = int(r.integers(0, (32 << 20) - n))
                    do = (bh if d2h else bd).take(n) + int(r.integers(0, 16))
                    items.append((do, so, n))
                if d2h:
                    mma.mma_weights_load([(dst_h.ptr + do, src_d.data_ptr() + so, n) for do, so, n in items],
                                         mma.MMA_D2H, st)
                else:
                    mma.mma_weights_load([(dst_d.data_ptr() + do, src_h.ptr + so, n) for do, so, n in items],
                                         mma.MMA_H2D, st)
                expect += [("h" if d2h else "d", do, so, n) for do, so, n in items]
            else:
                s = KV_SHAPES[int(r.integers(len(KV_SHAPES)))]
                xp = int(r.integers(3))  # GPU block layout: 0 piece, 1 x-packed, 2 head-major
                lay = mma.kv_layout(s.layers, s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes, s.gpu_num_blocks,
                                    s.host_num_slots, xp)
                pool_np = r.integers(0, 256, (s.host_num_slots, s.slot_bytes), dtype=np.uint8)
                if r.integers(3) == 0:  # a pool in HBM: one pool-kernel launch (piece, head-major) or the ring
                    pool = torch.from_numpy(pool_np.reshape(-1).copy()).cuda()
                else:
                    pool = mma.PinnedBuffer(pool_np.size)
                    pool.array[:] = pool_np.reshape(-1)
                layers_np = [r.integers(0, 256, (2, s.gpu_num_blocks, s.piece_bytes), dtype=np.uint8)
                             for _ in range(s.layers)]
                layers = [torch.from_numpy(x.reshape(-1).copy()).cuda() for x in layers_np]
                a = r.permutation(s.host_num_slots)[:s.n_blocks].astype(np.int32)
                b = r.permutation(s.gpu_num_blocks)[:s.n_blocks].astype(np.int32)
                torch.cuda.synchronize()  # the per-job inputs were written by torch on its own stream
                if d2h:
                    mma.mma_kv_offload(lay, pool, layers, b, a, st)
                else:
                    mma.mma_kv_fetch(lay, pool, layers, a, b, st)
                kv_jobs.append((s, xp, d2h, pool, pool_np, layers, layers_np, a, b))
        torch.cuda.synchronize()
        mma.mma_synchronize()
        stats = mma.mma_get_stats()
        log(f"  seed {seed}: {len(expect)} ranges, {len(kv_jobs)} KV jobs, transfers {stats['transfers']}, "
            f"cu bytes {stats['path_bytes'][16]}, sdma bytes {sum(stats['path_bytes'][:16])}, "
            f"commands {stats['sdma_commands']}")
        got = {"h": dst_h.array.copy(), "d": to_host(dst_d)}
        src = {"h": src_d_np, "d": src_h.array}
        covered = {"h": np.zeros(HOST, bool), "d": np.zeros(DEV, bool)}
        # Each range with 32 bytes of its poison margin on both sides (ranges are at least 48 bytes
        # apart), against the oracle; then every byte outside all ranges must still be poison.
        for side, do, so, n in expect:
            w0, w1 = max(0, do - 32), do + n + 32
            want = ocopy.memcpy(np.full(w1 - w0, POISON, np.uint8), do - w0, src[side], so, n)
            assert np.array_equal(got[side][w0:w1], want), (side, do, so, n)
            covered[side][do:do + n] = True
        for side in ("h", "d"):
            assert np.all(got[side][~covered[side]] == POISON), side
        for s, xp, d2h, pool, pool_np, layers, layers_np, a, b in kv_jobs:
            geom = (s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes)
            layout = (okv.LAYOUT_PIECE, okv.LAYOUT_XPACKED, okv.LAYOUT_HND)[xp]
            on_dev = isinstance(pool, torch.Tensor)
            if d2h:
                want = okv.kv_offload(pool_np, layers_np, b, a, layout, geom)
                got_pool = to_host(pool) if on_dev else pool.array
                assert np.array_equal(got_pool.reshape(s.host_num_slots, -1), want), (xp, on_dev)
            else:
                want = okv.kv_fetch(pool_np, layers_np, a, b, layout, geom)
                for l in range(s.layers):
                    assert np.array_equal(to_host(layers[l]).reshape(want[l].shape), want[l]), (l, xp, on_dev)
            if not on_dev:
                pool.free()
        src_h.free()
        dst_h.free()
    assert stats["failed_transfers"] == 0
