"""Benchmark of the multipath host->GPU path on one MI355X.

One step = one paged-KV fetch of a 64k-token prompt prefix (Llama-3-8B GQA shape:
32 layers x K,V x 8 kv heads x 128 dims, bf16, 16-token blocks -> 4096 blocks,
8 GiB) from a pinned host pool into the GPU's paged cache through
mma_kv_fetch. The step exercises every part of the path: planner, CU-path
gather, SDMA staging + HBM scatter, completion counters and the stream wait.
Inputs are resident (host pool filled, GPU cache allocated) before timing.

Printed: one JSON line (stdout) with the throughput, the KV fetch latency, the
roofline of the dummy-task kernel (PCIe-bound), the oracle's CPU throughput on
the same workload, native hipMemcpyAsync comparators, and the 64 MiB single-copy
workload.

Usage: python bench.py [--gpus 1] [--steps 10] [--warmup 2]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "host→GPU GB/s per copy (% of PCIe5 x16 peak); 64k-token KV fetch latency"
PCIE5_X16_GBS = 32e9 * 16 * 128 / 130 / 8 / 1e9   # 63.0 GB/s per direction after 128b/130b coding


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=int(os.environ.get("WORLD_SIZE", "1")))
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-extras", action="store_true", help="skip native comparators and the 64 MiB copy")
    p.add_argument("--cpu-seconds", type=float, default=10.0, help="minimum oracle timing window")
    p.add_argument("--calib", action="store_true",
                   help="only run plain kernels of known traffic (1 GiB fill, read, copy) for counter scaling")
    return p.parse_args()


def calibration_kernels():
    """Plain kernels of known HBM traffic, run under rocprofv3 --pmc to scale FETCH_SIZE/WRITE_SIZE:
    a torch fill (writes N), mma_digest_u32 (reads N) and a device-to-device copy (reads N, writes N)."""
    import torch

    import paper_2512_16056_amd as mma
    n = 1 << 30
    mma.mma_init(0)
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty(n, dtype=torch.uint8, device="cuda")
    out = torch.zeros(1, dtype=torch.int64, device="cuda")
    for _ in range(3):
        a.fill_(7)
        mma.mma_digest_u32(a, n, out)
        b.copy_(a)
    torch.cuda.synchronize()
    mma.mma_finalize()
    print(json.dumps({"calibration": {"bytes": n, "kernels": ["fill: write N", "mma_digest_kernel: read N",
                                                              "copyBuffer: read N + write N"]}}), flush=True)


def recorded_traffic(root: str):
    """HBM/EA bytes per launch of the transfer kernel from the committed rocprofv3 --pmc summary,
    valid only while the kernel source is the one that was profiled."""
    import hashlib
    path = os.path.join(root, "profiles", "mma_transfer_kernel__kv_fetch_64k.traffic.json")
    src = os.path.join(root, "paper_2512_16056_amd", "csrc", "mma_kernels.hip")
    try:
        rec = json.load(open(path))
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    except (OSError, ValueError):
        return None
    if rec.get("kernel_sha256") != sha:
        return None
    return rec.get("traffic_bytes_per_launch")


def main():
    args = parse()
    if args.calib:
        calibration_kernels()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the multipath path here is the single-GPU share (SDMA engines + "
              f"CU zero-copy over this GPU's own PCIe link); --gpus {args.gpus} is not supported.",
              file=sys.stderr)
        sys.exit(2)

    import ctypes

    import numpy as np
    import torch

    import paper_2512_16056_amd as mma
    import workloads as W

    torch.cuda.set_device(0)
    s = W.KV64K
    hs, gb = W.kv_fetch_tables(s, cfg=3)
    total = s.n_blocks * s.slot_bytes

    mma.mma_init(0)  # defaults, then MMA_* environment overrides
    cfg = mma.mma_get_config().as_dict()
    log("config:", cfg)

    # ---- inputs: pinned 8 GiB pool (seeded, block i at host_slots[i]) and the GPU paged cache
    t0 = time.time()
    pool = mma.PinnedBuffer(s.host_num_slots * s.slot_bytes)
    pv = pool.array.reshape(s.host_num_slots, s.slot_bytes)

    def fill(i):
        pv[hs[i]] = W.kv_block_bytes(3, i, s)

    with ThreadPoolExecutor(16) as ex:
        list(ex.map(fill, range(s.n_blocks)))
    layers = [torch.full((s.layer_bytes,), W.GPU_POISON, dtype=torch.uint8, device="cuda") for _ in range(s.layers)]
    lay = mma.kv_layout(s.layers, s.block_tokens, s.kv_heads, s.head_dim, s.elem_bytes, s.gpu_num_blocks,
                        s.host_num_slots)
    torch.cuda.synchronize()
    log(f"inputs ready in {time.time() - t0:.1f}s")

    stream = torch.cuda.Stream()
    for _ in range(args.warmup):
        mma.mma_kv_fetch(lay, pool, layers, hs, gb, stream)
    stream.synchronize()
    mma.mma_synchronize()
    mma.mma_reset_stats()

    # ---- timed region: exactly K steps, bracketed by synchronize on both sides
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for a, b in ev:
        a.record(stream)
        mma.mma_kv_fetch(lay, pool, layers, hs, gb, stream)
        b.record(stream)
    torch.cuda.synchronize()
    t_end = time.perf_counter()
    elapsed = t_end - t_start
    mma.mma_synchronize()
    stats = mma.mma_get_stats()
    kernel_ms = [a.elapsed_time(b) for a, b in ev]
    avg_kernel_ms = sum(kernel_ms) / len(kernel_ms)
    ms_per_step = elapsed * 1e3 / args.steps
    value = total * args.steps / elapsed / 1e9
    achieved = total / (avg_kernel_ms * 1e-3) / 1e9
    log(f"kv fetch: {ms_per_step:.2f} ms/step, {value:.2f} GB/s wall; kernel avg {avg_kernel_ms:.2f} ms "
        f"(min {min(kernel_ms):.2f}, max {max(kernel_ms):.2f}) = {achieved:.2f} GB/s")

    # ---- sampled parity against the oracle definition (full parity lives in the tests)
    r = np.random.default_rng(0)
    ok = True
    host = {}
    for _ in range(64):
        i, l, k = int(r.integers(s.n_blocks)), int(r.integers(s.layers)), int(r.integers(2))
        off = (k * s.gpu_num_blocks + int(gb[i])) * s.piece_bytes
        got = layers[l][off:off + s.piece_bytes].cpu().numpy()
        want = pv[hs[i]].reshape(s.layers, 2, s.piece_bytes)[l, k]
        ok &= bool(np.array_equal(got, want))
    log(f"sampled parity: {'ok' if ok else 'MISMATCH'}")

    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic",
        "config": {
            "workload": "kv_fetch_64k_tokens: 4096 blocks x 16 tokens, 32 layers x K,V x 8 kv heads x 128 dim bf16 "
                        "(8 GiB) pinned host pool -> paged GPU cache via block table",
            "bytes_per_step": total,
            "pieces_per_step": s.n_blocks * s.pieces_per_block,
            "chunk_bytes": cfg["chunk_bytes"],
            "paths_h2d": hex(cfg["path_mask_h2d"]),
            "cu_workgroups": cfg["cu_workgroups"],
            "parallelism": "1 GPU (SDMA engines + CU zero-copy on its own PCIe link)",
        },
        "kv_fetch_latency_ms": round(avg_kernel_ms, 3),
        "sampled_parity": ok,
        "path_bytes": {"cu": stats["path_bytes"][16],
                       **{f"sdma{e}": stats["path_bytes"][e] for e in range(16) if stats["path_bytes"][e]}},
        "engine_cpu_ms_per_step": round(stats["engine_cpu_ns"] / 1e6 / max(1, args.steps + args.warmup), 3),
        "roofline": {
            "kernel": "mma_transfer_kernel (dummy task: CU gather + stream wait)",
            "bound": "pcie",
            "achieved": round(achieved, 3),
            "peak": round(PCIE5_X16_GBS, 2),
            "unit": "GB/s",
            "frac": round(achieved / PCIE5_X16_GBS, 4),
            "traffic": recorded_traffic(ROOT),
        },
    }

    extras = {}
    if not args.no_extras:
        # measured link peak: native hipMemcpyAsync of 1 GiB from pinned memory
        n = 1 << 30
        hbuf = torch.empty(n, dtype=torch.uint8).pin_memory()
        dbuf = torch.empty(n, dtype=torch.uint8, device="cuda")
        times = []
        for _ in range(6):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            with torch.cuda.stream(stream):
                dbuf.copy_(hbuf, non_blocking=True)
            b.record(stream)
            b.synchronize()
            times.append(a.elapsed_time(b))
        link = n / (sorted(times[1:])[len(times[1:]) // 2] * 1e-3) / 1e9
        extras["measured_h2d_link_GBs"] = round(link, 2)
        out["roofline"]["measured_peak"] = round(link, 2)
        out["roofline"]["frac_of_measured"] = round(achieved / link, 4)
        del hbuf, dbuf

        # native per-piece hipMemcpyAsync KV fetch (262,144 copies)
        nat = ctypes.CDLL(os.path.join(ROOT, "paper_2512_16056_amd", "libmma_native.so"))
        lp = (ctypes.c_void_p * s.layers)(*[t.data_ptr() for t in layers])
        hs_c = hs.ctypes.data_as(ctypes.c_void_p)
        gb_c = gb.ctypes.data_as(ctypes.c_void_p)
        for fn_name in ("native_kv_fetch", "native_kv_fetch_batch"):
            fn = getattr(nat, fn_name)
            fn.restype = ctypes.c_int
            fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64,
                           ctypes.c_uint32, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p]
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            rc = fn(pool.ptr, lp, hs_c, gb_c, s.n_blocks, s.layers, s.piece_bytes, s.gpu_num_blocks,
                    stream.cuda_stream)
            stream.synchronize()
            dt = time.perf_counter() - t0
            if rc == 0:
                extras[f"{fn_name}_ms"] = round(dt * 1e3, 2)
            else:
                extras[f"{fn_name}_ms"] = None
        nat_ms = extras.get("native_kv_fetch_ms")
        if nat_ms:
            extras["kv_fetch_speedup_vs_native"] = round(nat_ms / ms_per_step, 2)

        # the 64 MiB single-copy workload: MMA vs one hipMemcpyAsync
        n = W.COPY64_BYTES
        src = mma.PinnedBuffer(n)
        src.array[:] = W.uniform_bytes(1, W.TAG_DATA, 0, n)
        dst = torch.empty(n, dtype=torch.uint8, device="cuda")
        srct = torch.from_numpy(src.array)  # pinned memory seen by torch as a CPU tensor

        def timed(fn, reps=50, warm=5):
            ts = []
            for _ in range(min(warm, reps)):
                fn()
            stream.synchronize()
            for _ in range(reps):
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(stream)
                fn()
                b.record(stream)
                b.synchronize()
                ts.append(a.elapsed_time(b))
            ts.sort()
            return ts[len(ts) // 2]

        mma_ms = timed(lambda: mma.mma_memcpy_async(dst, src, n, mma.MMA_H2D, stream))
        ok64 = bool(np.array_equal(dst.cpu().numpy(), src.array))

        def native():
            with torch.cuda.stream(stream):
                dst.copy_(srct, non_blocking=True)

        nat64 = timed(native)
        extras["copy64"] = {"mma_ms": round(mma_ms, 4), "mma_GBs": round(n / mma_ms / 1e6, 2),
                            "native_ms": round(nat64, 4), "native_GBs": round(n / nat64 / 1e6, 2),
                            "ratio_vs_native": round(nat64 / mma_ms, 3), "parity": ok64,
                            "frac_of_pcie5": round(n / mma_ms / 1e6 / PCIE5_X16_GBS, 4)}
        if "measured_h2d_link_GBs" in extras:
            extras["copy64"]["frac_of_measured"] = round(n / mma_ms / 1e6 / extras["measured_h2d_link_GBs"], 4)
        src.free()

        # KV offload (GPU -> host): the 50%-dirty subset of the cache just fetched, 2048 blocks (4 GiB),
        # into a permutation of host slots; against 131,072 per-piece hipMemcpyAsync D2H.
        plan = W.kv_offload_plan(s, cfg=4)
        src_blocks = gb[plan.dirty].astype(np.int32)
        off_bytes = len(plan.dirty) * s.slot_bytes

        def offload():
            mma.mma_kv_offload(lay, pool, layers, src_blocks, plan.dest, stream)

        off_ms = timed(offload, reps=5)
        fn = nat.native_kv_offload
        fn.restype = ctypes.c_int
        fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64,
                       ctypes.c_uint32, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        rc = fn(pool.ptr, lp, src_blocks.ctypes.data_as(ctypes.c_void_p), plan.dest.ctypes.data_as(ctypes.c_void_p),
                len(plan.dirty), s.layers, s.piece_bytes, s.gpu_num_blocks, stream.cuda_stream)
        stream.synchronize()
        nat_off = (time.perf_counter() - t0) * 1e3 if rc == 0 else None
        extras["kv_offload_2048_blocks"] = {"mma_ms": round(off_ms, 3), "mma_GBs": round(off_bytes / off_ms / 1e6, 2),
                                            "native_per_piece_ms": round(nat_off, 2) if nat_off else None,
                                            "speedup_vs_native": round(nat_off / off_ms, 2) if nat_off else None}

        # The same gather with the pool resident in HBM: the CU gather/scatter code alone, HBM-bound.
        dpool = torch.empty(s.host_num_slots * s.slot_bytes, dtype=torch.uint8, device="cuda")
        dpool.copy_(torch.from_numpy(pool.array))
        hbm_ms = timed(lambda: mma.mma_kv_fetch(lay, dpool, layers, hs, gb, stream), reps=5)
        ok_hbm = True
        for _ in range(16):
            i, l, k = int(r.integers(s.n_blocks)), int(r.integers(s.layers)), int(r.integers(2))
            off = (k * s.gpu_num_blocks + int(gb[i])) * s.piece_bytes
            ok_hbm &= bool(np.array_equal(layers[l][off:off + s.piece_bytes].cpu().numpy(),
                                          pool.array.reshape(s.host_num_slots, s.layers, 2, -1)[hs[i], l, k]))
        extras["kv_gather_hbm_pool"] = {"ms": round(hbm_ms, 3), "payload_GBs": round(total / hbm_ms / 1e6, 1),
                                        "hbm_GBs_read_plus_write": round(2 * total / hbm_ms / 1e6, 1),
                                        "frac_of_8TBs": round(2 * total / hbm_ms / 1e6 / 8000.0, 4),
                                        "sampled_parity": ok_hbm}
        del dpool

        # Model wake-up: 291 Llama-3-8B-shaped bf16 tensors (16.06 GB) as one list, against 291 hipMemcpyAsync.
        sizes = W.weight_tensor_bytes()
        offs, wtotal = W.arena_offsets(sizes, 256)
        arena = mma.PinnedBuffer(wtotal)
        arena.array[:] = 0x3C
        wdst = [torch.empty(n, dtype=torch.uint8, device="cuda") for n in sizes]
        lst = [(wdst[t], arena.ptr + offs[t], sizes[t]) for t in range(len(sizes))]
        w_ms = timed(lambda: mma.mma_weights_load(lst, mma.MMA_H2D, stream), reps=3)
        D = (ctypes.c_void_p * len(sizes))(*[t.data_ptr() for t in wdst])
        S = (ctypes.c_void_p * len(sizes))(*[arena.ptr + o for o in offs])
        Z = (ctypes.c_uint64 * len(sizes))(*sizes)
        nat.native_list.restype = ctypes.c_int
        w_nat = timed(lambda: nat.native_list(D, S, Z, ctypes.c_uint64(len(sizes)), 0,
                                              ctypes.c_void_p(stream.cuda_stream)), reps=3)
        extras["weights_wakeup_291"] = {"mma_ms": round(w_ms, 2), "mma_GBs": round(wtotal / w_ms / 1e6, 2),
                                        "native_ms": round(w_nat, 2), "ratio_vs_native": round(w_nat / w_ms, 3)}
        del wdst
        arena.free()
        log("extras:", extras)
    out["extras"] = extras

    if not args.no_cpu_baseline:
        from oracle import kv as okv
        poison = np.full((2, s.gpu_num_blocks, s.piece_bytes), W.GPU_POISON, np.uint8)
        reps, t0 = 0, time.perf_counter()
        while True:
            for l in range(s.layers):
                okv.kv_fetch_layer(pv, poison, l, s.layers, hs, gb)
            reps += 1
            if time.perf_counter() - t0 >= args.cpu_seconds:
                break
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": round(total * reps / dt / 1e9, 3), "unit": "GB/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"{reps} x the full 4096-block 64k-token KV fetch (oracle.kv.kv_fetch_layer "
                                         f"over 32 layers, numpy slice copies, one thread), {dt:.1f} s"}
    print(json.dumps(out), flush=True)
    pool.free()
    mma.mma_finalize()


if __name__ == "__main__":
    main()
