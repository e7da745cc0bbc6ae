"""Full-size parity of the model wake-up, fall-asleep and mixed-contention workloads.

Model wake-up: 291 Llama-3-8B-shaped bf16 tensors (16,060,522,496 B) from one pinned
arena into separate device tensors as one logical transfer; every destination byte
is compared with its source (oracle.copy: dst = src) and with oracle.digest. Fall
asleep: the same list from device tensors back into a pinned arena.

Mixed contention: the same kind of tensor list loaded on stream A as 34 groups,
each followed on A by the dependent digest kernel over that group, while a 50%-dirty
64k-token KV offload runs on stream B, with 256 KiB micro-transfers. The digests
must equal the oracle digests of the sources (stream ordering survived), the
weights must be byte-exact and the whole host pool must match oracle.kv.
"""
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import workloads as W
from oracle import digest as odigest
from oracle import kv as okv

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2512_16056_amd as mma  # noqa: E402
from gpu_helpers import log, session  # noqa: E402
from test_gpu_kv import layout_of  # noqa: E402

POOL = ThreadPoolExecutor(16)


def weights_arena(cfg: int):
    sizes = W.weight_tensor_bytes()
    offs, total = W.arena_offsets(sizes, 256)
    arena = mma.PinnedBuffer(total)

    def fill(t):
        arena.array[offs[t]:offs[t] + sizes[t]] = W.weight_values(cfg, t, sizes[t] // 2).view(np.uint8)

    list(POOL.map(fill, range(len(sizes))))
    return arena, sizes, offs


def test_weights_wakeup_full():
    t0 = time.time()
    with session("both"):
        arena, sizes, offs = weights_arena(2)
        assert sum(sizes) == 16060522496
        dst = [torch.full((n,), W.WEIGHT_POISON, dtype=torch.uint8, device="cuda") for n in sizes]
        log(f"  inputs ready in {time.time() - t0:.1f}s")
        stream = torch.cuda.Stream()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        mma.mma_weights_load([(dst[t], arena.ptr + offs[t], sizes[t]) for t in range(len(sizes))],
                             mma.MMA_H2D, stream)
        b.record(stream)
        stream.synchronize()
        mma.mma_synchronize()
        ms = a.elapsed_time(b)
        st = mma.mma_get_stats()
        log(f"  wake-up: {ms:.1f} ms, {sum(sizes) / ms / 1e6:.2f} GB/s; cu={st['path_bytes'][16]} "
            f"sdma={st['path_bytes'][:2]}")
        assert st["failed_transfers"] == 0

        def check(t):
            got = dst[t].cpu().numpy()
            src = arena.array[offs[t]:offs[t] + sizes[t]]
            return bool(np.array_equal(got, src)) and odigest.digest(got) == odigest.digest(src)

        bad = [t for t, ok in enumerate(map(check, range(len(sizes)))) if not ok]
        assert not bad, bad
        del dst
        arena.free()


def test_weights_sleep_full():
    """Model fall-asleep (Section 5.2.2, the other direction of a model switch): the same
    291-tensor list (16,060,522,496 B) from device tensors into a poisoned pinned arena as one
    logical device->host transfer. Each tensor's bytes must equal its source (oracle.copy:
    dst = src) and its digest the source's, and the alignment gaps between tensors in the arena
    must keep their poison."""
    t0 = time.time()
    with session("both"):
        src_arena, sizes, offs = weights_arena(2)
        # device tensors written by the runtime's copy, independent of this library
        dev = [torch.from_numpy(src_arena.array[offs[t]:offs[t] + sizes[t]]).to("cuda") for t in range(len(sizes))]
        dst_arena = mma.PinnedBuffer(src_arena.nbytes)
        dst_arena.array[:] = W.WEIGHT_POISON
        torch.cuda.synchronize()
        log(f"  inputs ready in {time.time() - t0:.1f}s")
        stream = torch.cuda.Stream()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        mma.mma_weights_load([(dst_arena.ptr + offs[t], dev[t], sizes[t]) for t in range(len(sizes))],
                             mma.MMA_D2H, stream)
        b.record(stream)
        stream.synchronize()
        mma.mma_synchronize()
        ms = a.elapsed_time(b)
        st = mma.mma_get_stats()
        log(f"  fall-asleep: {ms:.1f} ms, {sum(sizes) / ms / 1e6:.2f} GB/s; cu={st['path_bytes'][16]} "
            f"sdma={st['path_bytes'][:2]}")
        assert st["failed_transfers"] == 0 and sum(st["path_bytes"]) == sum(sizes)
        del dev

        def check(t):
            got = dst_arena.array[offs[t]:offs[t] + sizes[t]]
            want = src_arena.array[offs[t]:offs[t] + sizes[t]]
            gap_end = offs[t + 1] if t + 1 < len(sizes) else dst_arena.nbytes
            gap_ok = bool(np.all(dst_arena.array[offs[t] + sizes[t]:gap_end] == W.WEIGHT_POISON))
            return bool(np.array_equal(got, want)) and odigest.digest(got) == odigest.digest(want) and gap_ok

        bad = [t for t, ok in enumerate(POOL.map(check, range(len(sizes)))) if not ok]
        assert not bad, bad
        dst_arena.free()
        src_arena.free()


def test_mixed_contention_full():
    t0 = time.time()
    s = W.KV64K
    plan = W.kv_offload_plan(s, cfg=5)
    with session("both", chunk_bytes=256 << 10):
        arena, sizes, offs = weights_arena(5)
        groups = W.weight_groups()
        assert len(groups) == 34 and sum(len(g) for g in groups) == len(sizes)
        dst = [torch.full((n,), W.WEIGHT_POISON, dtype=torch.uint8, device="cuda") for n in sizes]
        digests = torch.zeros(len(sizes), dtype=torch.int64, device="cuda")

        pool = mma.PinnedBuffer(s.host_num_slots * s.slot_bytes)
        pv = pool.array.reshape(s.host_num_slots, s.slot_bytes)

        def fill_occ(slot):
            pv[slot] = W.kv_occupied_bytes(5, int(slot), s)

        list(POOL.map(fill_occ, plan.occupied))
        pv[plan.free] = W.HOST_FREE_POISON
        before = pv.copy()
        blocks = np.empty((s.n_blocks, s.layers, 2, s.piece_bytes), np.uint8)

        def fill_blk(i):
            blocks[i] = W.kv_block_bytes(5, i, s).reshape(s.layers, 2, s.piece_bytes)

        list(POOL.map(fill_blk, range(s.n_blocks)))
        layers = []
        for l in range(s.layers):
            lay_np = np.full((2, s.gpu_num_blocks, s.piece_bytes), W.GPU_POISON, np.uint8)
            lay_np[:, plan.gpu_blocks_all] = blocks[:, l].transpose(1, 0, 2)
            layers.append(torch.from_numpy(lay_np.reshape(-1)).cuda())
        del blocks
        torch.cuda.synchronize()
        log(f"  inputs ready in {time.time() - t0:.1f}s")

        sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
        ea, eb = [torch.cuda.Event(enable_timing=True) for _ in range(2)], \
            [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ea[0].record(sa)
        eb[0].record(sb)
        # stream B: the offload, enqueued first so it overlaps the whole weight load
        mma.mma_kv_offload(layout_of(s), pool, layers, plan.src_blocks, plan.dest, sb)
        eb[1].record(sb)
        for g in groups:
            mma.mma_weights_load([(dst[t], arena.ptr + offs[t], sizes[t]) for t in g], mma.MMA_H2D, sa)
            for t in g:  # dependent HBM-bound consumer of the group just loaded
                mma.mma_digest_u32(dst[t], sizes[t], digests.data_ptr() + 8 * t, sa)
        ea[1].record(sa)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        st = mma.mma_get_stats()
        log(f"  stream A (weights + digests): {ea[0].elapsed_time(ea[1]):.1f} ms; "
            f"stream B (offload): {eb[0].elapsed_time(eb[1]):.1f} ms; failed={st['failed_transfers']}")
        assert st["failed_transfers"] == 0

        got_d = digests.cpu().numpy().view(np.uint64)
        want_d = list(POOL.map(lambda t: odigest.digest(arena.array[offs[t]:offs[t] + sizes[t]]), range(len(sizes))))
        bad = [t for t in range(len(sizes)) if int(got_d[t]) != want_d[t]]
        assert not bad, f"digest mismatch (ordering) for tensors {bad[:10]}"
        for t in range(len(sizes)):
            assert np.array_equal(dst[t].cpu().numpy(), arena.array[offs[t]:offs[t] + sizes[t]]), t
        views = [t.cpu().numpy().reshape(2, s.gpu_num_blocks, s.piece_bytes) for t in layers]
        want = okv.kv_offload(before, views, plan.src_blocks, plan.dest)
        assert np.array_equal(pv, want)
        del dst, layers
        pool.free()
        arena.free()
