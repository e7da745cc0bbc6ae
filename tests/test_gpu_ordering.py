"""Stream-ordering checks of the dummy-task substitution (Section 3.3: downstream
work must not see a copy before all fragments land; upstream producers must be
complete before any byte is read).

Destinations start as poison and a dependent HBM-bound kernel (the library's
digest kernel) runs right after each transfer on the same stream; its digest is
compared with oracle.digest of the *source*. An early release reads poison and
fails. Producer kernels write device data right before an offload on the same
stream; a late start would ship stale bytes.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import digest as odigest
from oracle import kv as okv

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2512_16056_amd as mma  # noqa: E402
from gpu_helpers import PATHS, device_bytes, from_host, log, session, to_host  # noqa: E402
from test_gpu_kv import layout_of  # noqa: E402


def test_digest_kernel_matches_oracle():
    with session("both"):
        for n in (4, 8, 12, 1000, 4096, 65536 + 12, (1 << 22) + 4):
            src = np.ascontiguousarray(W.uniform_bytes(9, 0, n, n))
            d = from_host(src)
            out = torch.zeros(1, dtype=torch.int64, device="cuda")
            mma.mma_digest_u32(d, n, out)
            torch.cuda.synchronize()
            got = int(out.cpu().numpy().view(np.uint64)[0])
            assert got == odigest.digest(src), n
        # unaligned start (4-byte aligned only) and ragged tail
        src = np.ascontiguousarray(W.uniform_bytes(9, 1, 0, 4096))
        d = from_host(src)
        out = torch.zeros(1, dtype=torch.int64, device="cuda")
        mma.mma_digest_u32(d.data_ptr() + 4, 4000 + 3, out)
        torch.cuda.synchronize()
        assert int(out.cpu().numpy().view(np.uint64)[0]) == odigest.digest(src[4:4 + 4003])


@pytest.mark.parametrize("paths", list(PATHS))
def test_h2d_then_dependent_kernel(paths):
    log(f"h2d ordering paths={paths}")
    sizes = [64 << 20, 3 << 20, (5 << 20) + 123, 777, 64 << 10, 16 << 20]
    with session(paths, chunk_bytes=1 << 20):
        stream = torch.cuda.Stream()
        srcs, dsts, outs = [], [], []
        with torch.cuda.stream(stream):
            for rep in range(3):
                for k, n in enumerate(sizes):
                    src = mma.PinnedBuffer(n)
                    src.array[:] = W.uniform_bytes(7, rep, k, n)
                    dst = torch.empty(n, dtype=torch.uint8, device="cuda")
                    dst.fill_(W.WEIGHT_POISON)                      # producer of the old contents
                    out = torch.zeros(1, dtype=torch.int64, device="cuda")
                    mma.mma_memcpy_async(dst, src, n, mma.MMA_H2D, stream)
                    mma.mma_digest_u32(dst, n, out, stream)          # dependent consumer
                    srcs.append(src)
                    dsts.append(dst)
                    outs.append(out)
        stream.synchronize()
        for src, out in zip(srcs, outs):
            assert int(out.cpu().numpy().view(np.uint64)[0]) == odigest.digest(src.array)
        mma.mma_synchronize()


@pytest.mark.parametrize("paths", list(PATHS))
def test_producer_then_d2h(paths):
    log(f"d2h ordering paths={paths}")
    n = 24 << 20
    with session(paths, chunk_bytes=1 << 20):
        stream = torch.cuda.Stream()
        with torch.cuda.stream(stream):
            base = torch.arange(n // 4, dtype=torch.int32, device="cuda")
            hosts = []
            for rep in range(4):
                dev = torch.empty(n, dtype=torch.uint8, device="cuda")
                # producer kernel on the same stream, immediately before the offload
                dev.view(torch.int32).copy_(base * (2 * rep + 3) + 0x1234567)
                host = mma.PinnedBuffer(n)
                host.array[:] = W.HOST_FREE_POISON
                mma.mma_memcpy_async(host, dev, n, mma.MMA_D2H, stream)
                hosts.append((rep, host))
        stream.synchronize()
        idx = np.arange(n // 4, dtype=np.int64)
        for rep, host in hosts:
            want = ((idx * (2 * rep + 3) + 0x1234567) & 0xFFFFFFFF).astype(np.uint32).view(np.uint8)
            assert np.array_equal(host.array, want), rep
        mma.mma_synchronize()


@pytest.mark.parametrize("control", [mma.MMA_CONTROL_HOST, mma.MMA_CONTROL_DEVICE])
def test_two_streams_concurrent(control):
    """An H2D stream and a D2H stream with dependent work on each, interleaved."""
    n = 32 << 20
    with session("both", chunk_bytes=256 << 10, control=control):
        sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
        src = mma.PinnedBuffer(n)
        src.array[:] = W.uniform_bytes(11, 0, 0, n)
        dev_b = from_host(W.uniform_bytes(11, 0, 1, n))
        torch.cuda.synchronize()
        outs, hosts = [], []
        for rep in range(4):
            with torch.cuda.stream(sa):
                dst = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(0)
                out = torch.zeros(1, dtype=torch.int64, device="cuda")
                mma.mma_memcpy_async(dst, src, n, mma.MMA_H2D, sa)
                mma.mma_digest_u32(dst, n, out, sa)
                outs.append(out)
            with torch.cuda.stream(sb):
                host = mma.PinnedBuffer(n)
                mma.mma_memcpy_async(host, dev_b, n, mma.MMA_D2H, sb)
                hosts.append(host)
        torch.cuda.synchronize()
        want = odigest.digest(src.array)
        assert all(int(o.cpu().numpy().view(np.uint64)[0]) == want for o in outs)
        want_b = to_host(dev_b)
        assert all(np.array_equal(h.array, want_b) for h in hosts)
        mma.mma_synchronize()


def test_kv_fetch_then_dependent_kernel():
    s = W.KVShape(layers=4, block_tokens=16, kv_heads=2, head_dim=64, elem_bytes=2,
                  gpu_num_blocks=300, host_num_slots=256, n_blocks=200)
    hs, gb = W.kv_fetch_tables(s, cfg=3)
    with session("both", chunk_bytes=64 << 10, cu_sub_bytes=8 << 10):
        pool = mma.PinnedBuffer(s.host_num_slots * s.slot_bytes)
        pool.array[:] = np.random.default_rng(5).integers(0, 256, pool.nbytes, dtype=np.uint8)
        stream = torch.cuda.Stream()
        outs = []
        with torch.cuda.stream(stream):
            layers = [torch.empty(s.layer_bytes, dtype=torch.uint8, device="cuda").fill_(W.GPU_POISON)
                      for _ in range(s.layers)]
            mma.mma_kv_fetch(layout_of(s), pool, layers, hs, gb, stream)
            for l in range(s.layers):
                out = torch.zeros(1, dtype=torch.int64, device="cuda")
                mma.mma_digest_u32(layers[l], s.layer_bytes, out, stream)
                outs.append(out)
        stream.synchronize()
        poison = np.full((2, s.gpu_num_blocks, s.piece_bytes), W.GPU_POISON, np.uint8)
        pv = pool.array.reshape(s.host_num_slots, s.slot_bytes)
        for l in range(s.layers):
            want = okv.kv_fetch_layer(pv, poison, l, s.layers, hs, gb)
            assert int(outs[l].cpu().numpy().view(np.uint64)[0]) == odigest.digest(want), l
        mma.mma_synchronize()


@pytest.mark.parametrize("control", [mma.MMA_CONTROL_HOST, mma.MMA_CONTROL_DEVICE])
def test_concurrent_submitters(control):
    """Four host threads, each with its own stream, submit interleaved H2D copies, D2H copies and
    tensor lists of mixed sizes (self-contained, CU+SDMA and SDMA-merged ones) at the same time;
    each transfer is followed on its stream by the dependent digest kernel, and in the last round by
    a blocking device->host copy (mma_memcpy_stream) whose result is read at once. Every destination
    and every digest must equal the oracle's (submissions are serialised inside the library;
    streams are independent; each blocking caller waits for its own copy)."""
    from concurrent.futures import ThreadPoolExecutor
    sizes = [12345, 1 << 20, (3 << 20) + 17, 9 << 20, 64 << 10]
    with session("both", chunk_bytes=1 << 20, control=control):
        def worker(tid):
            stream = torch.cuda.Stream()
            with torch.cuda.stream(stream):  # torch's own allocations and fills go on this stream too
                return _submitter(tid, stream)

        def _submitter(tid, stream):
            results, bad = [], []
            for rep in range(3):
                for k, n in enumerate(sizes):
                    src_np = np.ascontiguousarray(W.uniform_bytes(40 + tid, rep, k, n))
                    h = mma.PinnedBuffer(n)
                    h.array[:] = src_np
                    d = torch.empty(n, dtype=torch.uint8, device="cuda")
                    out = torch.zeros(1, dtype=torch.int64, device="cuda")
                    back = mma.PinnedBuffer(n)
                    back.array[:] = W.WEIGHT_POISON
                    half = n // 2
                    if (rep + k) % 2:
                        mma.mma_memcpy_async(d, h, n, mma.MMA_H2D, stream)
                    else:
                        mma.mma_weights_load([(d.data_ptr(), h.ptr, half), (d.data_ptr() + half, h.ptr + half, n - half)],
                                             mma.MMA_H2D, stream)
                    mma.mma_digest_u32(d, n, out, stream)
                    mma.mma_memcpy_async(back, d, n, mma.MMA_D2H, stream)
                    results.append((src_np, h, d, out, back))
                    if rep == 2:  # a blocking copy behind that work, read at once
                        back2 = mma.PinnedBuffer(n)
                        back2.array[:] = W.WEIGHT_POISON
                        outcome = mma.mma_memcpy_stream(back2, d, n, mma.MMA_D2H, stream)
                        if outcome != mma.MMA_COPY_RETIRED or not np.array_equal(back2.array, src_np):
                            bad.append(("blocking", tid, k, outcome))
                        back2.free()
            stream.synchronize()
            for i, (src_np, h, d, out, back) in enumerate(results):
                if not np.array_equal(back.array, src_np):
                    bad.append(("d2h", i))
                if int(out.cpu().numpy().view(np.uint64)[0]) != odigest.digest(src_np):
                    bad.append(("digest", i))
                h.free()
                back.free()
            return bad

        with ThreadPoolExecutor(4) as ex:
            bad = [b for r in ex.map(worker, range(4)) for b in r]
        torch.cuda.synchronize()
        mma.mma_synchronize()
        st = mma.mma_get_stats()
    assert not bad, bad[:10]
    assert st["failed_transfers"] == 0
    log(f"  transfers={st['transfers']} sdma commands={st['sdma_commands']} cu bytes={st['path_bytes'][16]}")
