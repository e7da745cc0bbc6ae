"""Process lifecycle: mma_finalize with transfers still in flight waits for them; a program that
copies through the library and exits without mma_finalize
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


@pytest.mark.parametrize("control", [0, 1])
def test_finalize_waits_for_transfers_in_flight(control):
    """mma_finalize right after enqueuing, with nothing synchronised: a 256 MiB host->device copy
    queued behind a spin kernel on a stream of its own (the engine thread drives it under host
    control) and a 3 MiB whole launch. finalize waits until both have retired and returns MMA_OK;
    the bytes are exact, and the library initialises again."""
    import numpy as np

    import paper_2512_16056_amd as mma
    from gpu_helpers import log
    from oracle import copy as ocopy
    import workloads as W

    n, m = 256 << 20, (3 << 20) + 5
    src_np = np.ascontiguousarray(W.uniform_bytes(51, control, 0, n))
    log(f"finalize with transfers in flight, control={control}")
    mma.mma_init(0, control=control, watchdog_ms=5000)
    try:
        src = mma.PinnedBuffer(n)
        src.array[:] = src_np
        dst = torch.full((n,), W.WEIGHT_POISON, dtype=torch.uint8, device="cuda")
        dst2 = torch.full((m,), W.WEIGHT_POISON, dtype=torch.uint8, device="cuda")
        st = torch.cuda.Stream()
        torch.cuda.synchronize()
        with torch.cuda.stream(st):
            torch.cuda._sleep(2_000_000)
        mma.mma_memcpy_async(dst, src, n, mma.MMA_H2D, st)
        mma.mma_memcpy_async(dst2, src.ptr + 7, m, mma.MMA_H2D, st)
    finally:
        mma.mma_finalize()
    torch.cuda.synchronize()
    assert np.array_equal(dst.cpu().numpy(), ocopy.memcpy(np.full(n, W.WEIGHT_POISON, np.uint8), 0, src_np, 0, n))
    assert np.array_equal(dst2.cpu().numpy(), ocopy.memcpy(np.full(m, W.WEIGHT_POISON, np.uint8), 0, src_np, 7, m))
    src.free()
    mma.mma_init(0)
    mma.mma_finalize()


def test_init_rejects_invalid_configurations():
    """mma_init refuses each invalid configuration with MMA_ERR_INVALID_ARG and stays uninitialised
    (a chunk size near 2^64 among them, whose ring-entry count would wrap if formed as chunk + sub);
    a second mma_init is MMA_ERR_ALREADY_INITIALIZED; a device index out of range is refused."""
    import paper_2512_16056_amd as mma

    bad = [dict(cu_sub_bytes=100), dict(cu_sub_bytes=128), dict(chunk_bytes=17),
           dict(chunk_bytes=(1 << 64) - 16), dict(chunk_bytes=1 << 40), dict(queue_depth=17),
           dict(cu_workgroups=257), dict(cu_queue_depth=65), dict(engine_nap_us=1001),
           dict(static_cu_percent=101), dict(control=2)]
    for over in bad:
        with pytest.raises(mma.MMAError) as e:
            mma.mma_init(0, **over)
        assert e.value.name == "MMA_ERR_INVALID_ARG", over
        with pytest.raises(mma.MMAError) as e:
            mma.mma_get_config()
        assert e.value.name == "MMA_ERR_NOT_INITIALIZED", over
    with pytest.raises(mma.MMAError) as e:
        mma.mma_init(torch.cuda.device_count())
    assert e.value.name == "MMA_ERR_INVALID_ARG"
    mma.mma_init(0)
    try:
        with pytest.raises(mma.MMAError) as e:
            mma.mma_init(0)
        assert e.value.name == "MMA_ERR_ALREADY_INITIALIZED"
        assert mma.mma_get_config().chunk_bytes == 2 << 20
    finally:
        mma.mma_finalize()


def test_environment_zero_selects_defaults():
    """Configured from the environment (mma_init without a configuration), 0 and values that do not
    parse select the defaults as 0 does in a configuration; a copy then runs byte-exact."""
    import numpy as np

    import paper_2512_16056_amd as mma
    from oracle import copy as ocopy
    import workloads as W

    keys = {"MMA_CHUNK_BYTES": "0", "MMA_CU_WGS": "0", "MMA_QUEUE_DEPTH": "x", "MMA_CU_QUEUE_DEPTH": "0",
            "MMA_CU_SUB_BYTES": "0", "MMA_WATCHDOG_MS": "none", "MMA_CU_WHOLE_BYTES": "0"}
    saved = {k: os.environ.get(k) for k in keys}
    os.environ.update(keys)
    try:
        mma.mma_init(0)
    finally:
        for k, v in saved.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    try:
        c, d = mma.mma_get_config(), mma.mma_config_default()
        for f in ("chunk_bytes", "cu_workgroups", "queue_depth", "cu_queue_depth", "cu_sub_bytes", "watchdog_ms",
                  "cu_whole_bytes"):
            assert getattr(c, f) == getattr(d, f), f
        n = (40 << 20) + 5
        src_np = np.ascontiguousarray(W.uniform_bytes(71, 0, 0, n))
        src = mma.PinnedBuffer(n)
        src.array[:] = src_np
        dst = torch.full((n,), W.WEIGHT_POISON, dtype=torch.uint8, device="cuda")
        mma.mma_memcpy_async(dst, src, n, mma.MMA_H2D)
        torch.cuda.synchronize()
        assert np.array_equal(dst.cpu().numpy(), ocopy.memcpy(np.full(n, W.WEIGHT_POISON, np.uint8), 0, src_np, 0, n))
        src.free()
    finally:
        mma.mma_finalize()
