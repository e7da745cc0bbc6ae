"""Child process of test_gpu_interpose.py, run with libmma_interpose.so in LD_PRELOAD.

An unmodified torch program's copies, and direct calls of the interposed HIP functions
(hipMemcpyAsync, with an explicit kind and with hipMemcpyDefault, hipMemcpy and
hipMemcpyWithStream, the latter also on a stream of its own with nothing pending, resolved from the process's global scope, where the preloaded library
comes first), move seeded bytes in each direction on its own. Each result is compared with oracle.copy and read back over a route that stays
with the runtime (pageable host memory). Per call, the library's statistics tell whether
the copy went through it (and which paths carried it). With the argument "faults", the
failure handling is checked with host-forced faults instead, and with "defaults" which copies go
through the library when neither MMA_INTERPOSE_SYNC nor MMA_INTERPOSE_IDLE is set. Prints one JSON
line.
"""
import ctypes
import json
import os
import sys

import numpy as np
import torch

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
from oracle import copy as ocopy  # noqa: E402

H2D, D2H, DEFAULT = 1, 2, 4  # hipMemcpyKind (hipMemcpyDefault: the runtime infers the direction)
HIP_ERROR_UNKNOWN = 999
POISON = 0xA5
SIZES = [(3 << 20) + 5, (40 << 20) + 3, 4096]  # whole CU launch, multipath engine, below the threshold

_rt = ctypes.CDLL(None)  # the global scope: the interposer's exports come first
for _name, _args in (("hipMemcpy", [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]),
                     ("hipMemcpyAsync", [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int,
                                         ctypes.c_void_p]),
                     ("hipMemcpyWithStream", [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int,
                                              ctypes.c_void_p])):
    getattr(_rt, _name).argtypes = _args
    getattr(_rt, _name).restype = ctypes.c_int


def seeded(n, seed):
    return np.random.default_rng(seed).integers(0, 256, n, dtype=np.uint8)


def stats(mma):
    s = mma.mma_get_stats()
    return {"transfers": s["transfers"], "failed": s["failed_transfers"], "sdma": sum(s["path_bytes"][:16]),
            "cu": s["path_bytes"][16]}


def delta(a, b):
    return {k: b[k] - a[k] for k in a}


_SIDE = []


def _side_stream():
    if not _SIDE:
        _SIDE.append(torch.cuda.Stream())
    return _SIDE[0]


def call(route, dst, src, n, kind, stream):
    """One interposed copy; returns the HIP status."""
    if route == "torch_sync":  # copy_ with non_blocking=False: hipMemcpyWithStream in torch on ROCm
        dst.copy_(src, non_blocking=False)
        return 0
    if route == "torch_async":
        dst.copy_(src, non_blocking=True)
        torch.cuda.current_stream().synchronize()
        return 0
    d, s = dst.data_ptr(), src.data_ptr()
    if route == "hipMemcpy":
        return _rt.hipMemcpy(d, s, n, kind)
    if route == "hipMemcpyAsync/default":  # direction from the pointers' attributes
        rc = _rt.hipMemcpyAsync(d, s, n, DEFAULT, stream)
        torch.cuda.current_stream().synchronize()
        return rc
    if route == "hipMemcpyWithStream":
        return _rt.hipMemcpyWithStream(d, s, n, kind, stream)
    if route == "hipMemcpyWithStream/idle":  # a stream of its own with nothing pending: early start
        torch.cuda.synchronize()
        return _rt.hipMemcpyWithStream(d, s, n, kind, _side_stream().cuda_stream)
    rc = _rt.hipMemcpyAsync(d, s, n, kind, stream)
    torch.cuda.current_stream().synchronize()
    return rc


def routes(mma):
    out = {}
    stream = torch.cuda.current_stream().cuda_stream
    seed = 0
    for route in ("torch_async", "torch_sync", "hipMemcpyAsync", "hipMemcpyAsync/default", "hipMemcpy",
                  "hipMemcpyWithStream", "hipMemcpyWithStream/idle"):
        for n in SIZES:
            for kind in (H2D, D2H):
                seed += 1
                src_np = seeded(n, seed)
                before = stats(mma)
                if kind == H2D:
                    src = torch.from_numpy(src_np).pin_memory()
                    dst = torch.full((n,), POISON, dtype=torch.uint8, device="cuda")
                    rc = call(route, dst, src, n, kind, stream)
                    got = dst.cpu().numpy()  # pageable: read back by the runtime
                else:
                    src = torch.from_numpy(src_np).to("cuda")  # pageable: written by the runtime
                    dst = torch.full((n,), POISON, dtype=torch.uint8).pin_memory()
                    rc = call(route, dst, src, n, kind, stream)
                    got = dst.numpy().copy()
                torch.cuda.synchronize()
                mma.mma_synchronize()
                want = ocopy.memcpy(np.full(n, POISON, np.uint8), 0, src_np, 0, n)
                d = delta(before, stats(mma))
                out[f"{route}/{'h2d' if kind == H2D else 'd2h'}/{n}"] = {
                    "rc": rc, "exact": bool(np.array_equal(got, want)), **d}
    return out


def faults(mma):
    """Host control, engine threads told to ignore new transfers (the dummy task's watchdog then
    releases the stream): a blocking copy must still deliver its bytes (re-issued by the runtime
    once libmma has retired the failed copy), and an asynchronous copy's failure must be
    reported by the next interposed call, after which copies go through libmma again."""
    out = {}
    n = (40 << 20) + 3  # above the whole-launch limit: the engine thread drives it
    stream = torch.cuda.current_stream().cuda_stream
    src_np = seeded(n, 101)
    src = torch.from_numpy(src_np).pin_memory()
    want = ocopy.memcpy(np.full(n, POISON, np.uint8), 0, src_np, 0, n)

    mma.mma_test_set_fault(mma.MMA_FAULT_ENGINE_IGNORE, 1)
    before = stats(mma)
    dst = torch.full((n,), POISON, dtype=torch.uint8, device="cuda")
    print("faults: blocking hipMemcpy while the engine ignores transfers", file=sys.stderr, flush=True)
    rc = _rt.hipMemcpy(dst.data_ptr(), src.data_ptr(), n, H2D)
    out["sync_rc"] = rc
    out["sync_exact"] = bool(np.array_equal(dst.cpu().numpy(), want))
    out["sync"] = delta(before, stats(mma))

    before = stats(mma)
    dst2 = torch.full((n,), POISON, dtype=torch.uint8, device="cuda")
    print("faults: hipMemcpyAsync while the engine ignores transfers", file=sys.stderr, flush=True)
    out["async_rc"] = _rt.hipMemcpyAsync(dst2.data_ptr(), src.data_ptr(), n, H2D, stream)
    torch.cuda.synchronize()  # released by the watchdog
    mma.mma_test_set_fault(mma.MMA_FAULT_ENGINE_IGNORE, 0)
    # retire it; the sticky failure stays set (mma_synchronize reports it, and does not clear it)
    out["async_sync_status"] = mma.lib.mma_synchronize(20000)
    out["async"] = delta(before, stats(mma))
    small = (1 << 20) + 7
    dst3 = torch.full((small,), POISON, dtype=torch.uint8, device="cuda")
    print("faults: the next interposed call reports the failure", file=sys.stderr, flush=True)
    out["next_rc"] = _rt.hipMemcpyAsync(dst3.data_ptr(), src.data_ptr(), small, H2D, stream)
    torch.cuda.synchronize()
    out["next_untouched"] = bool(np.all(dst3.cpu().numpy() == POISON))  # the reporting call copied nothing
    before = stats(mma)
    out["after_rc"] = _rt.hipMemcpyAsync(dst3.data_ptr(), src.data_ptr(), small, H2D, stream)
    torch.cuda.synchronize()
    mma.mma_synchronize()
    out["after_exact"] = bool(np.array_equal(dst3.cpu().numpy(), src_np[:small]))
    out["after"] = delta(before, stats(mma))
    return out


def defaults(mma):
    """The interposer's defaults (MMA_INTERPOSE_SYNC and MMA_INTERPOSE_IDLE unset): an asynchronous
    pinned copy queued behind other work goes through the library, one on a stream with nothing
    pending and the blocking ones stay with the runtime; all exact. Then an asynchronous copy that
    fails in the library (host-forced: the engine thread ignores it, the watchdog releases the
    stream) is reported by the next call, a copy on an idle stream that copies nothing, and the
    one after that goes to the runtime again."""
    out = {}
    n = (40 << 20) + 3
    stream = torch.cuda.current_stream().cuda_stream
    src_np = seeded(n, 202)
    src = torch.from_numpy(src_np).pin_memory()

    def busy():  # about 50 ms of other work queued on the stream before the copy
        torch.cuda._sleep(int(2.4e9 * 0.05))

    for name, route, pre in (("hipMemcpyAsync/busy", "hipMemcpyAsync", busy),
                             ("hipMemcpyAsync/idle", "hipMemcpyAsync", None),
                             ("hipMemcpy", "hipMemcpy", None), ("hipMemcpyWithStream", "hipMemcpyWithStream", None)):
        dst = torch.full((n,), POISON, dtype=torch.uint8, device="cuda")
        torch.cuda.synchronize()
        before = stats(mma)
        if pre:
            pre()
        rc = call(route, dst, src, n, H2D, stream)
        torch.cuda.synchronize()
        mma.mma_synchronize()
        out[name] = {"rc": rc, "exact": bool(np.array_equal(dst.cpu().numpy(), src_np)), **delta(before, stats(mma))}

    rep = {}
    want = ocopy.memcpy(np.full(n, POISON, np.uint8), 0, src_np, 0, n)
    mma.mma_test_set_fault(mma.MMA_FAULT_ENGINE_IGNORE, 1)
    dst = torch.full((n,), POISON, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    before = stats(mma)
    print("defaults: hipMemcpyAsync behind other work while the engine ignores transfers", file=sys.stderr,
          flush=True)
    busy()
    rep["failed_rc"] = _rt.hipMemcpyAsync(dst.data_ptr(), src.data_ptr(), n, H2D, stream)
    torch.cuda.synchronize()  # released by the watchdog
    mma.mma_test_set_fault(mma.MMA_FAULT_ENGINE_IGNORE, 0)
    mma.lib.mma_synchronize(20000)  # retire it: the failure is now sticky
    rep["failed"] = delta(before, stats(mma))
    small = (1 << 20) + 7
    dst3 = torch.full((small,), POISON, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    print("defaults: the next interposed call, on an idle stream, reports the failure", file=sys.stderr, flush=True)
    rep["next_rc"] = _rt.hipMemcpyAsync(dst3.data_ptr(), src.data_ptr(), small, H2D, stream)
    torch.cuda.synchronize()
    rep["next_untouched"] = bool(np.all(dst3.cpu().numpy() == POISON))
    before = stats(mma)
    rep["after_rc"] = _rt.hipMemcpyAsync(dst3.data_ptr(), src.data_ptr(), small, H2D, stream)
    torch.cuda.synchronize()
    mma.mma_synchronize()
    rep["after_exact"] = bool(np.array_equal(dst3.cpu().numpy(), want[:small]))
    rep["after"] = delta(before, stats(mma))
    out["idle_report"] = rep
    return out


def main():
    torch.cuda.set_device(0)
    import paper_2512_16056_amd as mma  # the library the interposer loaded (same path, same instance)
    # the first interposed call initialises the library: make one before reading its statistics
    warm = torch.zeros(1 << 20, dtype=torch.uint8).pin_memory()
    torch.zeros(1 << 20, dtype=torch.uint8, device="cuda").copy_(warm, non_blocking=True)
    torch.cuda.synchronize()
    if len(sys.argv) > 1 and sys.argv[1] == "faults":
        res = faults(mma)
    elif len(sys.argv) > 1 and sys.argv[1] == "defaults":
        res = defaults(mma)
    else:
        res = routes(mma)
    print(json.dumps(res), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
