"""Child process of test_gpu_interpose.py, run with libmma_interpose.so in LD_PRELOAD: plain torch
copies (no call into this package) must be exact, and copies of pinned memory at or above the
threshold must have gone through libmma. Prints one JSON line."""
import json
import sys

import numpy as np
import torch


def main():
    torch.cuda.set_device(0)
    r = np.random.default_rng(5)
    out = {}
    for n in (8 << 20, (3 << 20) + 5, 4096):
        src = torch.from_numpy(r.integers(0, 256, n, dtype=np.uint8)).pin_memory()
        dev = torch.full((n,), 0xA5, dtype=torch.uint8, device="cuda")
        dev.copy_(src, non_blocking=True)                      # hipMemcpyAsync H2D
        back = torch.full((n,), 0x5A, dtype=torch.uint8).pin_memory()
        back.copy_(dev, non_blocking=True)                     # hipMemcpyAsync D2H
        torch.cuda.synchronize()
        out[f"pinned_{n}"] = bool(torch.equal(back, src))
        pageable = torch.from_numpy(r.integers(0, 256, n, dtype=np.uint8))
        dev2 = pageable.to("cuda")                             # pageable: left to the runtime
        out[f"pageable_{n}"] = bool(torch.equal(dev2.cpu(), pageable))
    import paper_2512_16056_amd as mma                         # the library the interposer loaded
    st = mma.mma_get_stats()
    out["transfers"] = st["transfers"]
    out["failed"] = st["failed_transfers"]
    out["path_bytes"] = sum(st["path_bytes"])
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
