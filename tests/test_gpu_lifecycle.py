"""Process lifecycle: a program that copies through the library and exits without mma_finalize
must exit cleanly (the engine threads are stopped when the library is unloaded, before the HIP
runtime's own teardown), with the data exact."""
import os
import subprocess
import sys
import textwrap

import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = textwrap.dedent("""
    import numpy as np, torch
    import paper_2512_16056_amd as mma
    torch.cuda.set_device(0)
    mma.mma_init(0)
    n = (8 << 20) + 3
    src = mma.PinnedBuffer(n)
    src.array[:] = np.arange(n, dtype=np.uint64).astype(np.uint8)
    dst = torch.empty(n, dtype=torch.uint8, device="cuda")
    mma.mma_memcpy_async(dst, src, n, mma.MMA_H2D)
    torch.cuda.synchronize()
    assert np.array_equal(dst.cpu().numpy(), src.array)
    print("copied", flush=True)
    # no mma_finalize: exit with the engine threads still running
""")


def test_exit_without_finalize_is_clean():
    env = dict(os.environ, PYTHONPATH=ROOT + os.pathsep + os.environ.get("PYTHONPATH", ""))
    print("child: copy then exit without mma_finalize", flush=True)
    r = subprocess.run([sys.executable, "-u", "-c", CHILD], env=env, capture_output=True, text=True, timeout=240)
    print(r.stdout[-1000:], r.stderr[-2000:])
    assert "copied" in r.stdout
    assert r.returncode == 0
