"""The C ABI used from plain C: tests/cpp/c_abi_example.c includes only include/mma.h and
the HIP C API, is compiled by gcc as C11 and linked against the in-tree libmma.so.

On the CPU this checks that the public header is valid C and that every call the program
makes links. On the GPU the program runs as its own process (no Python in it), under both
control modes, and checks its copies byte for byte against their sources."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "cpp", "c_abi_example.c")
PKG = os.path.join(ROOT, "paper_2512_16056_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def _compile(out):
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    if not os.path.exists(os.path.join(PKG, "libmma.so")):
        pytest.skip("libmma.so not built (python paper_2512_16056_amd/build.py)")
    cmd = [cc, "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           f"-I{os.path.join(ROCM, 'include')}", f"-I{os.path.join(ROOT, 'include')}", SRC, "-o", out,
           f"-L{PKG}", "-lmma", f"-L{os.path.join(ROCM, 'lib')}", "-lamdhip64",
           f"-Wl,-rpath,{PKG}", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]


def test_c_program_compiles_and_links(tmp_path):
    _compile(str(tmp_path / "c_abi"))


@pytest.mark.gpu
@pytest.mark.parametrize("control", ["0", "1"])
def test_c_program_runs(tmp_path, control):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    exe = str(tmp_path / "c_abi")
    _compile(exe)
    env = dict(os.environ)
    env["MMA_CONTROL"] = control
    env["MMA_WATCHDOG_MS"] = "5000"
    print(f"c_abi_example MMA_CONTROL={control}", flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=180, env=env)
    print(r.stdout[-3000:], r.stderr[-3000:])
    assert r.returncode == 0 and "ALL OK" in r.stdout
