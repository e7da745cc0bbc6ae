"""Transparent interposition (Section 3.2): an unmodified torch program run with
libmma_interpose.so in LD_PRELOAD. Its pinned host<->device copies at or above the threshold go
through the multipath library and stay byte-exact; pageable copies and copies below the
threshold stay with the runtime."""
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


@pytest.mark.parametrize("control", ["0", "1"])
def test_torch_copies_through_interposer(control):
    assert os.path.exists(LIB), "build with python paper_2512_16056_amd/build.py"
    env = dict(os.environ)
    env["MMA_CONTROL"] = control  # the interposer initialises the library from the environment
    # keep whatever is preloaded already; add the interposer after it
    env["LD_PRELOAD"] = (env.get("LD_PRELOAD", "") + " " + LIB).strip()
    env["MMA_WATCHDOG_MS"] = "5000"
    env["PYTHONPATH"] = ROOT + os.pathsep + env.get("PYTHONPATH", "")
    print("child: interpose_child.py with the interposer preloaded", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "tests", "interpose_child.py")], env=env,
                       capture_output=True, text=True, timeout=240)
    print(r.stdout[-2000:], r.stderr[-2000:])
    assert r.returncode == 0
    res = json.loads(r.stdout.strip().splitlines()[-1])
    assert all(v for k, v in res.items() if k.startswith(("pinned_", "pageable_"))), res
    # two intercepted copies (H2D + D2H) for each of the two sizes above 32 KiB
    assert res["transfers"] >= 4 and res["failed"] == 0, res
    assert res["path_bytes"] >= 2 * ((8 << 20) + (3 << 20) + 5), res
