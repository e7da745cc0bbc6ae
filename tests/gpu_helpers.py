"""Shared helpers of the GPU tests: library sessions with a given path set, pinned
buffers and device buffers filled from the seeded workload generators."""
from __future__ import annotations

import contextlib
import sys

import numpy as np
import torch

import paper_2512_16056_amd as mma

# Path sets exercised by the parity tests: CU path only (small transfers then run as
# self-contained launches), SDMA engines only, both -- with every transfer kept on the
# multipath engine (cu_whole_bytes[_d2h]=1), so that small cases still mix the paths.
PATHS = {
    "cu": dict(path_mask_h2d=mma.MMA_PATH_CU, path_mask_d2h=mma.MMA_PATH_CU),
    "sdma": dict(path_mask_h2d=0x3, path_mask_d2h=0x3),
    "both": dict(cu_whole_bytes=1, cu_whole_bytes_d2h=1),
}


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


@contextlib.contextmanager
def session(paths: str = "both", **overrides):
    cfg = mma.mma_config_default()
    cfg.watchdog_ms = 5000  # bound every wait of a test run
    for k, v in {**PATHS[paths], **overrides}.items():
        setattr(cfg, k, v)
    mma.mma_clear_error()
    mma.mma_init(0, cfg)
    try:
        yield mma.mma_get_config()
    finally:
        torch.cuda.synchronize()
        mma.mma_finalize()


def device_bytes(n: int, fill: int | None = None) -> torch.Tensor:
    t = torch.empty(max(n, 1), dtype=torch.uint8, device="cuda")
    if fill is not None:
        t.fill_(fill)
    return t


def to_host(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy()


def from_host(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.array(a, dtype=np.uint8, copy=True)).to("cuda")
