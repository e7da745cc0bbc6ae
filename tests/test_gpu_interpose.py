"""Transparent interposition (Section 3.2, Transfer Task Interceptor): an unmodified torch
program run with libmma_interpose.so in LD_PRELOAD.

Every interposed route -- torch's asynchronous and blocking copies, and direct calls of
hipMemcpyAsync (with an explicit kind, and with hipMemcpyDefault, where the interposer reads the
direction from the pointers), hipMemcpy and hipMemcpyWithStream (also on an idle stream of its
own, where the copy engines start before the kernel launch) -- moves bytes in each direction
on its own, compared with the oracle. Pinned copies at or above the threshold go through the
multipath library (one transfer each, copy engines included above the whole-launch
limit under host control); copies below it stay with the runtime. Under host-forced
faults, a failed blocking copy still delivers its bytes and says so on stderr, and a
failed asynchronous copy is reported by the next interposed call. These tests send every
eligible copy through the library (MMA_INTERPOSE_SYNC=1, MMA_INTERPOSE_IDLE=1); the last
one checks the defaults: blocking copies, and asynchronous ones on a stream with nothing
pending, stay with the runtime, whose copy is the faster there.
"""
import json
import os
import subprocess
import sys

import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2512_16056_amd", "libmma_interpose.so")
THRESHOLD = 32 * 1024


def run_child(control: str, *args, sync: bool = True, idle: bool = True):
    assert os.path.exists(LIB), "build with python paper_2512_16056_amd/build.py"
    env = dict(os.environ)
    env["MMA_CONTROL"] = control  # the interposer initialises the library from the environment
    env.pop("MMA_INTERPOSE_SYNC", None)
    if sync:  # blocking copies through the library too (off by default)
        env["MMA_INTERPOSE_SYNC"] = "1"
    env.pop("MMA_INTERPOSE_IDLE", None)
    if idle:  # asynchronous copies on an idle stream through the library too (off by default)
        env["MMA_INTERPOSE_IDLE"] = "1"
    # keep whatever is preloaded already; add the interposer after it
    env["LD_PRELOAD"] = (env.get("LD_PRELOAD", "") + " " + LIB).strip()
    env["MMA_WATCHDOG_MS"] = "2000"
    env["PYTHONPATH"] = ROOT + os.pathsep + env.get("PYTHONPATH", "")
    print(f"child: interpose_child.py {' '.join(args)} control={control}", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "tests", "interpose_child.py"), *args], env=env,
                       capture_output=True, text=True, timeout=240)
    print(r.stdout[-3000:], r.stderr[-3000:])
    assert r.returncode == 0
    return json.loads(r.stdout.strip().splitlines()[-1]), r.stderr


@pytest.mark.parametrize("control", ["0", "1"])
def test_interposed_routes(control):
    res, _ = run_child(control)
    assert len(res) == 7 * 3 * 2
    for key, r in res.items():
        route, direction, n = key.rsplit("/", 2)
        n = int(n)
        assert r["rc"] == 0 and r["exact"], key
        assert r["failed"] == 0, key
        if n >= THRESHOLD:
            assert r["transfers"] == 1 and r["sdma"] + r["cu"] == n, (key, r)
            if control == "0" and n > (24 << 20):
                # the multipath engine: the copy engines carried part of it
                assert r["sdma"] > 0 and r["cu"] > 0, (key, r)
        else:
            assert r["transfers"] == 0, (key, r)


def test_interposed_failures():
    res, err = run_child("0", "faults")
    # blocking copy: libmma's copy failed (watchdog), was retired, re-issued by the runtime
    assert res["sync_rc"] == 0 and res["sync_exact"], res
    assert res["sync"]["failed"] == 1, res
    assert "hipMemcpy: copy of" in err and "copied again by the runtime" in err
    # asynchronous copy: enqueued, failed later; the next interposed call reports it and copies nothing
    assert res["async_rc"] == 0 and res["async"]["failed"] == 1, res
    assert res["async_sync_status"] == -6, res  # MMA_ERR_TRANSFER_FAILED, still pending
    assert res["next_rc"] == 999 and res["next_untouched"], res
    assert "an earlier copy through libmma failed" in err
    # the state is cleared: copies go through libmma again
    assert res["after_rc"] == 0 and res["after_exact"] and res["after"]["transfers"] == 1, res


def test_interposer_defaults():
    """Without MMA_INTERPOSE_SYNC and MMA_INTERPOSE_IDLE: blocking copies stay with the runtime (on
    one GPU a blocking caller does not wait less through the library), and so do asynchronous ones
    on a stream with nothing pending (the runtime's copy engine starts sooner than a kernel); an
    asynchronous copy queued behind other work goes through the library. An earlier asynchronous
    failure is reported by the next call even when that call's copy would stay with the runtime."""
    res, err = run_child("0", "defaults", sync=False, idle=False)
    copies = {k: v for k, v in res.items() if k != "idle_report"}
    assert all(r["rc"] == 0 and r["exact"] for r in copies.values()), res
    assert res["hipMemcpyAsync/busy"]["transfers"] == 1, res
    assert res["hipMemcpyAsync/idle"]["transfers"] == 0, res
    assert res["hipMemcpy"]["transfers"] == 0 and res["hipMemcpyWithStream"]["transfers"] == 0, res
    rep = res["idle_report"]
    assert rep["failed_rc"] == 0 and rep["failed"]["failed"] == 1, res  # the busy-stream copy failed (watchdog)
    assert rep["next_rc"] == 999 and rep["next_untouched"], res  # reported by the idle-stream call
    assert "an earlier copy through libmma failed" in err
    assert rep["after_rc"] == 0 and rep["after_exact"] and rep["after"]["transfers"] == 0, res
