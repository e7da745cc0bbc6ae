"""Python binding of libmma.so -- multipath host<->GPU copies on one MI355X.

Argument marshalling only: every function forwards to the C entry point of the
same name in ``include/mma.h``; all data movement runs in the library's HIP
kernels and SDMA submissions. PyTorch provides device memory and streams.

``import torch`` happens before the library is loaded so that libmma.so binds to
the HIP runtime already in the process (one runtime, shared streams). If the
library has not been built this import fails loudly -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np
import torch  # noqa: F401  (loads the process's HIP runtime first)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmma.so")

MMA_OK = 0
MMA_ERR_NOT_INITIALIZED = -1
MMA_ERR_INVALID_ARG = -2
MMA_ERR_NOT_PINNED = -3
MMA_ERR_HIP = -4
MMA_ERR_TRANSFER_FAILED = -6
MMA_ERR_TIMEOUT = -10
MMA_ERR_NO_MEMORY = -8
MMA_ERR_INTERNAL = -11
MMA_H2D = 0
MMA_D2H = 1
MMA_PATH_CU = 0x80000000
MMA_DUPLEX_UNCHANGED = 0xFFFFFFFF  # duplex_paths_*: keep the direction's own paths
MMA_ENGINE_NAP_OFF = 0xFFFFFFFF  # engine_nap_us: the engine threads poll without sleeping
MMA_KV_LAYOUT_PIECE = 0
MMA_KV_LAYOUT_XPACKED = 1
MMA_KV_LAYOUT_HND = 2
MMA_CONTROL_HOST = 0
MMA_CONTROL_DEVICE = 1
MMA_NUM_PATHS = 17
MMA_FAULT_ENGINE_STALL_US = 1
MMA_FAULT_SDMA_SUBMIT_FAIL = 2
MMA_FAULT_ENGINE_IGNORE = 3
MMA_FAULT_DEVICE_SIGNAL_HOLD = 4
MMA_FAULT_POOL_NO_TABLE = 5
MMA_COPY_NOT_ENQUEUED = 0
MMA_COPY_RETIRED = 1
MMA_COPY_IN_FLIGHT = 2
MMA_TASK_CU_ONLY = 1
MMA_TASK_SDMA_ONLY = 2

STATUS = {
    0: "MMA_OK", -1: "MMA_ERR_NOT_INITIALIZED", -2: "MMA_ERR_INVALID_ARG", -3: "MMA_ERR_NOT_PINNED",
    -4: "MMA_ERR_HIP", -5: "MMA_ERR_HSA", -6: "MMA_ERR_TRANSFER_FAILED", -7: "MMA_ERR_ALREADY_INITIALIZED",
    -8: "MMA_ERR_NO_MEMORY", -9: "MMA_ERR_BUFFER_TOO_SMALL", -10: "MMA_ERR_TIMEOUT", -11: "MMA_ERR_INTERNAL",
}


class MMAError(RuntimeError):
    def __init__(self, status: int, func: str, detail: str):
        self.status = status
        self.name = STATUS.get(status, str(status))
        super().__init__(f"{func}: {self.name}: {detail}")


class mma_config_t(ctypes.Structure):
    _fields_ = [("chunk_bytes", ctypes.c_uint64), ("fallback_bytes", ctypes.c_uint64),
                ("small_bytes", ctypes.c_uint64), ("queue_depth", ctypes.c_uint32),
                ("cu_queue_depth", ctypes.c_uint32), ("backoff_depth", ctypes.c_uint32),
                ("path_mask_h2d", ctypes.c_uint32), ("path_mask_d2h", ctypes.c_uint32),
                ("cu_workgroups", ctypes.c_uint32), ("cu_sub_bytes", ctypes.c_uint32),
                ("watchdog_ms", ctypes.c_uint32), ("static_split", ctypes.c_uint32),
                ("static_cu_percent", ctypes.c_uint32), ("sdma_merge_tasks", ctypes.c_uint32),
                ("cu_whole_bytes", ctypes.c_uint32), ("cu_whole_bytes_d2h", ctypes.c_uint32),
                ("control", ctypes.c_uint32), ("duplex_paths_h2d", ctypes.c_uint32),
                ("duplex_paths_d2h", ctypes.c_uint32), ("engine_nap_us", ctypes.c_uint32)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class mma_copy_desc_t(ctypes.Structure):
    _fields_ = [("dst", ctypes.c_void_p), ("src", ctypes.c_void_p), ("bytes", ctypes.c_uint64)]


class mma_kv_layout_t(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_uint32), ("block_tokens", ctypes.c_uint32),
                ("kv_heads", ctypes.c_uint32), ("head_dim", ctypes.c_uint32),
                ("elem_bytes", ctypes.c_uint32), ("gpu_num_blocks", ctypes.c_uint32),
                ("host_num_slots", ctypes.c_uint32), ("gpu_layout", ctypes.c_uint32)]


class mma_stats_t(ctypes.Structure):
    _fields_ = [("transfers", ctypes.c_uint64), ("failed_transfers", ctypes.c_uint64),
                ("path_bytes", ctypes.c_uint64 * MMA_NUM_PATHS), ("path_tasks", ctypes.c_uint64 * MMA_NUM_PATHS),
                ("staging_bytes", ctypes.c_uint64), ("sdma_submit_failures", ctypes.c_uint64),
                ("engine_cpu_ns", ctypes.c_uint64), ("engine_wall_busy_ns", ctypes.c_uint64),
                ("sdma_foreign_busy_skips", ctypes.c_uint64), ("sdma_congestion_backoffs", ctypes.c_uint64),
                ("sdma_commands", ctypes.c_uint64),
                ("sdma_engines_h2d", ctypes.c_uint32), ("sdma_engines_d2h", ctypes.c_uint32),
                ("cu_path_enabled", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
                ("pool_launches", ctypes.c_uint64), ("engine_naps", ctypes.c_uint64)]

    def as_dict(self):
        d = {k: getattr(self, k) for k, _ in self._fields_ if k not in ("reserved", "path_bytes", "path_tasks")}
        d["path_bytes"] = list(self.path_bytes)
        d["path_tasks"] = list(self.path_tasks)
        return d


class mma_trace_rec_t(ctypes.Structure):
    _fields_ = [("seq", ctypes.c_uint64), ("dir", ctypes.c_int32), ("kind", ctypes.c_int32),
                ("bytes", ctypes.c_uint64), ("tasks", ctypes.c_uint64),
                ("t_api_ns", ctypes.c_uint64), ("t_submit_ns", ctypes.c_uint64), ("t_started_ns", ctypes.c_uint64),
                ("t_first_sdma_ns", ctypes.c_uint64), ("t_last_task_ns", ctypes.c_uint64),
                ("t_complete_ns", ctypes.c_uint64), ("t_retire_ns", ctypes.c_uint64),
                ("path_tasks", ctypes.c_uint64 * MMA_NUM_PATHS), ("failed", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]

    def as_dict(self):
        d = {k: getattr(self, k) for k, _ in self._fields_ if k not in ("reserved", "path_tasks")}
        d["path_tasks"] = list(self.path_tasks)
        return d


class mma_plan_entry_t(ctypes.Structure):
    _fields_ = [("item", ctypes.c_uint64), ("offset", ctypes.c_uint64), ("bytes", ctypes.c_uint64),
                ("flags", ctypes.c_uint32), ("reserved", ctypes.c_uint32)]


_P = ctypes.c_void_p
_U64 = ctypes.c_uint64
_I32 = ctypes.c_int32
_U32 = ctypes.c_uint32
_S = ctypes.c_int32

# name -> (argtypes, restype)
_SIGNATURES = {
    "mma_config_default": ([ctypes.POINTER(mma_config_t)], _S),
    "mma_init": ([ctypes.c_int, ctypes.POINTER(mma_config_t)], _S),
    "mma_finalize": ([], _S),
    "mma_get_config": ([ctypes.POINTER(mma_config_t)], _S),
    "mma_synchronize": ([_U32], _S),
    "mma_host_alloc": ([_U64, ctypes.POINTER(_P)], _S),
    "mma_host_free": ([_P], _S),
    "mma_memcpy_async": ([_P, _P, _U64, _I32, _P], _S),
    "mma_memcpy": ([_P, _P, _U64, _I32], _S),
    "mma_memcpy_stream": ([_P, _P, _U64, _I32, _P, ctypes.POINTER(_I32)], _S),
    "mma_weights_load": ([ctypes.POINTER(mma_copy_desc_t), _U64, _I32, _P], _S),
    # the layer array and the two tables go as plain addresses: a ctypes pointer cast costs
    # microseconds per call, as much as a small transfer's whole host-side set-up
    "mma_kv_fetch": ([ctypes.POINTER(mma_kv_layout_t), _P, _P, _P, _P, _U64, _P], _S),
    "mma_kv_offload": ([ctypes.POINTER(mma_kv_layout_t), _P, _P, _P, _P, _U64, _P], _S),
    "mma_kv_fetch_noalloc": ([ctypes.POINTER(mma_kv_layout_t), _P, _P, _P, _P, _U64, _P], _S),
    "mma_digest_u32": ([_P, _U64, _P, _P], _S),
    "mma_get_stats": ([ctypes.POINTER(mma_stats_t)], _S),
    "mma_reset_stats": ([], _S),
    "mma_status_str": ([_S], ctypes.c_char_p),
    "mma_last_error": ([], ctypes.c_char_p),
    "mma_clear_error": ([], _S),
    "mma_plan_list": ([ctypes.POINTER(_U64), _U64, _U64, _U64, _U64, ctypes.POINTER(mma_plan_entry_t), _U64,
                       ctypes.POINTER(_U64)], _S),
    "mma_plan_kv": ([_U64, _U32, _U64, _U64, ctypes.POINTER(mma_plan_entry_t), _U64, ctypes.POINTER(_U64)], _S),
    "mma_validate_kv_tables": ([ctypes.POINTER(_I32), _U32, ctypes.POINTER(_I32), _U32, _U64], _S),
    "mma_kv_layout_sizes": ([ctypes.POINTER(mma_kv_layout_t), ctypes.POINTER(_U64), ctypes.POINTER(_U64),
                             ctypes.POINTER(_U64), ctypes.POINTER(_U64)], _S),
    "mma_trace_enable": ([_I32], _S),
    "mma_trace_read": ([ctypes.POINTER(mma_trace_rec_t), _U64, ctypes.POINTER(_U64)], _S),
    "mma_test_set_fault": ([_I32, _U64], _S),
}


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python paper_2512_16056_amd/build.py`")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (args, res) in _SIGNATURES.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    return lib


lib = _load()


def _check(status: int, func: str) -> None:
    if status != MMA_OK:
        raise MMAError(status, func, lib.mma_last_error().decode(errors="replace"))


def _ptr(x) -> int:
    """Device/host address of an int, torch tensor, numpy array or PinnedBuffer."""
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    if isinstance(x, torch.Tensor):
        return x.data_ptr()
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    if isinstance(x, PinnedBuffer):
        return x.ptr
    raise TypeError(f"cannot take the address of {type(x)}")


def _stream(s) -> int:
    if s is None:
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else 0
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


# ------------------------------------------------------------------ lifecycle
def mma_config_default() -> mma_config_t:
    c = mma_config_t()
    _check(lib.mma_config_default(ctypes.byref(c)), "mma_config_default")
    return c


def mma_init(device: int = 0, cfg: Optional[mma_config_t] = None, **overrides) -> None:
    """Initialise on `device`. cfg=None and no overrides: defaults + MMA_* environment."""
    if overrides and cfg is None:
        cfg = mma_config_t()
    for k, v in overrides.items():
        setattr(cfg, k, v)
    _check(lib.mma_init(device, ctypes.byref(cfg) if cfg is not None else None), "mma_init")


def mma_finalize() -> None:
    _check(lib.mma_finalize(), "mma_finalize")


def mma_get_config() -> mma_config_t:
    c = mma_config_t()
    _check(lib.mma_get_config(ctypes.byref(c)), "mma_get_config")
    return c


def mma_synchronize(timeout_ms: int = 60000) -> None:
    _check(lib.mma_synchronize(timeout_ms), "mma_synchronize")


# ------------------------------------------------------------------ host memory
def mma_host_alloc(nbytes: int) -> int:
    p = ctypes.c_void_p()
    _check(lib.mma_host_alloc(nbytes, ctypes.byref(p)), "mma_host_alloc")
    return p.value or 0


def mma_host_free(ptr: int) -> None:
    _check(lib.mma_host_free(ptr), "mma_host_free")


class PinnedBuffer:
    """Owner of an mma_host_alloc allocation with a zero-copy numpy uint8 view."""

    def __init__(self, nbytes: int):
        self.nbytes = int(nbytes)
        self.ptr = mma_host_alloc(self.nbytes) if self.nbytes else 0
        self.array = (np.ctypeslib.as_array((ctypes.c_uint8 * self.nbytes).from_address(self.ptr))
                      if self.nbytes else np.zeros(0, np.uint8))

    def free(self) -> None:
        if self.ptr:
            self.array = None
            mma_host_free(self.ptr)
            self.ptr = 0

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.free()


# ------------------------------------------------------------------ transfers
def mma_memcpy_async(dst, src, nbytes: int, direction: int, stream=None) -> None:
    _check(lib.mma_memcpy_async(_ptr(dst), _ptr(src), nbytes, direction, _stream(stream)), "mma_memcpy_async")


def mma_memcpy(dst, src, nbytes: int, direction: int) -> None:
    """Blocking copy on the legacy default stream; returns once the data has arrived."""
    _check(lib.mma_memcpy(_ptr(dst), _ptr(src), nbytes, direction), "mma_memcpy")


def mma_memcpy_stream(dst, src, nbytes: int, direction: int, stream=None) -> int:
    """Blocking copy ordered on `stream`; returns the outcome (MMA_COPY_*). A failure raises MMAError,
    whose `outcome` attribute is set."""
    out = ctypes.c_int32(-1)
    st = lib.mma_memcpy_stream(_ptr(dst), _ptr(src), nbytes, direction, _stream(stream), ctypes.byref(out))
    try:
        _check(st, "mma_memcpy_stream")
    except MMAError as e:
        e.outcome = out.value
        raise
    return out.value


def mma_weights_load(copies: Sequence[Tuple[object, object, int]], direction: int, stream=None) -> None:
    """copies: (dst, src, nbytes) triples."""
    n = len(copies)
    arr = (mma_copy_desc_t * max(n, 1))()
    for i, (d, s, b) in enumerate(copies):
        arr[i].dst, arr[i].src, arr[i].bytes = _ptr(d), _ptr(s), int(b)
    _check(lib.mma_weights_load(arr, n, direction, _stream(stream)), "mma_weights_load")


def kv_layout(num_layers, block_tokens, kv_heads, head_dim, elem_bytes, gpu_num_blocks, host_num_slots,
              gpu_layout: int = 0) -> mma_kv_layout_t:
    return mma_kv_layout_t(num_layers, block_tokens, kv_heads, head_dim, elem_bytes, gpu_num_blocks,
                           host_num_slots, gpu_layout)


def layer_table(gpu_layers) -> ctypes.Array:
    """The per-layer GPU base addresses as the C array the KV calls take. A caller that moves
    KV between the same layer tensors many times can build it once and pass it as
    `gpu_layers`; a fresh one costs about 0.3 us per layer."""
    if isinstance(gpu_layers, ctypes.Array):
        return gpu_layers
    ptrs = [_ptr(t) for t in gpu_layers]
    return (ctypes.c_void_p * max(len(ptrs), 1))(*ptrs)


def mma_kv_fetch(layout: mma_kv_layout_t, host_pool, gpu_layers, host_slots, gpu_blocks, stream=None) -> None:
    hs, gb = _i32(host_slots), _i32(gpu_blocks)
    if hs.size != gb.size:
        raise ValueError("host_slots and gpu_blocks differ in length")
    lt = layer_table(gpu_layers)  # a local, so the array outlives the call
    _check(lib.mma_kv_fetch(ctypes.byref(layout), _ptr(host_pool), lt,
                            hs.ctypes.data, gb.ctypes.data, hs.size, _stream(stream)), "mma_kv_fetch")


def mma_kv_fetch_noalloc(layout: mma_kv_layout_t, host_pool, gpu_layers, host_slots, gpu_blocks,
                         stream=None) -> None:
    hs, gb = _i32(host_slots), _i32(gpu_blocks)
    if hs.size != gb.size:
        raise ValueError("host_slots and gpu_blocks differ in length")
    lt = layer_table(gpu_layers)  # a local, so the array outlives the call
    _check(lib.mma_kv_fetch_noalloc(ctypes.byref(layout), _ptr(host_pool), lt,
                                    hs.ctypes.data, gb.ctypes.data, hs.size, _stream(stream)),
           "mma_kv_fetch_noalloc")


def mma_kv_offload(layout: mma_kv_layout_t, host_pool, gpu_layers, gpu_blocks, host_slots, stream=None) -> None:
    gb, hs = _i32(gpu_blocks), _i32(host_slots)
    if hs.size != gb.size:
        raise ValueError("host_slots and gpu_blocks differ in length")
    lt = layer_table(gpu_layers)  # a local, so the array outlives the call
    _check(lib.mma_kv_offload(ctypes.byref(layout), _ptr(host_pool), lt,
                              gb.ctypes.data, hs.ctypes.data, hs.size, _stream(stream)), "mma_kv_offload")


def mma_digest_u32(dev_ptr, nbytes: int, dev_out, stream=None) -> None:
    _check(lib.mma_digest_u32(_ptr(dev_ptr), nbytes, _ptr(dev_out), _stream(stream)), "mma_digest_u32")


# ------------------------------------------------------------------ status
def mma_get_stats() -> dict:
    s = mma_stats_t()
    _check(lib.mma_get_stats(ctypes.byref(s)), "mma_get_stats")
    return s.as_dict()


def mma_reset_stats() -> None:
    _check(lib.mma_reset_stats(), "mma_reset_stats")


def mma_status_str(status: int) -> str:
    return lib.mma_status_str(status).decode()


def mma_last_error() -> str:
    return lib.mma_last_error().decode(errors="replace")


def mma_clear_error() -> None:
    _check(lib.mma_clear_error(), "mma_clear_error")


def mma_trace_enable(on: bool = True) -> None:
    _check(lib.mma_trace_enable(1 if on else 0), "mma_trace_enable")


def mma_trace_read(cap: int = 65536) -> List[dict]:
    buf = (mma_trace_rec_t * cap)()
    n = _U64()
    _check(lib.mma_trace_read(buf, cap, ctypes.byref(n)), "mma_trace_read")
    return [buf[i].as_dict() for i in range(n.value)]


def mma_test_set_fault(kind: int, value: int) -> None:
    _check(lib.mma_test_set_fault(kind, value), "mma_test_set_fault")


# ------------------------------------------------------------------ host-only
def _plan_call(fn, name, *args) -> List[Tuple[int, int, int, int]]:
    n = _U64()
    _check(fn(*args, None, 0, ctypes.byref(n)), name)
    out = (mma_plan_entry_t * max(n.value, 1))()
    _check(fn(*args, out, n.value, ctypes.byref(n)), name)
    return [(out[i].item, out[i].offset, out[i].bytes, out[i].flags) for i in range(n.value)]


def mma_plan_list(sizes: Iterable[int], chunk: int, fallback: int, small: int) -> List[Tuple[int, int, int, int]]:
    s = np.ascontiguousarray(np.asarray(list(sizes), dtype=np.uint64))
    return _plan_call(lib.mma_plan_list, "mma_plan_list", s.ctypes.data_as(ctypes.POINTER(_U64)), s.size,
                      chunk, fallback, small)


def mma_plan_kv(n_blocks: int, pieces_per_block: int, piece_bytes: int, chunk: int):
    return _plan_call(lib.mma_plan_kv, "mma_plan_kv", n_blocks, pieces_per_block, piece_bytes, chunk)


def mma_validate_kv_tables(src, src_count: int, dst, dst_count: int) -> bool:
    s, d = _i32(src), _i32(dst)
    if s.size != d.size:
        return False
    st = lib.mma_validate_kv_tables(s.ctypes.data_as(ctypes.POINTER(_I32)), src_count,
                                    d.ctypes.data_as(ctypes.POINTER(_I32)), dst_count, s.size)
    return st == MMA_OK


def mma_kv_layout_sizes(layout: mma_kv_layout_t) -> dict:
    """Bytes of one piece, one host slot, the host pool and one GPU layer tensor; MMAError if the
    layout is invalid or a size does not fit 64 bits."""
    out = [_U64() for _ in range(4)]
    _check(lib.mma_kv_layout_sizes(ctypes.byref(layout), *[ctypes.byref(v) for v in out]), "mma_kv_layout_sizes")
    return dict(zip(("piece", "slot", "pool", "layer"), (v.value for v in out)))
