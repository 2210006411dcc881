"""The C ABI from plain C: the example program compiles against include/topkv.h
as C11 and links against libtopkv.so (CPU), and runs bit-exact on the GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2607_28633_amd")
SOURCE = os.path.join(PKG, "examples", "roundtrip.c")


def _build(tmp_path):
    from paper_2607_28633_amd.build import LIBRARY, build_library
    if not os.path.exists(LIBRARY):
        build_library()
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    exe = str(tmp_path / "roundtrip")
    cmd = [cc, "-std=c11", "-Wall", "-Wextra", "-Werror=implicit-function-declaration", "-D__HIP_PLATFORM_AMD__",
           "-I/opt/rocm/include", f"-I{ROOT}/include", SOURCE, f"-L{PKG}", "-ltopkv", "-L/opt/rocm/lib",
           "-lamdhip64", "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def test_example_compiles_and_links_as_c(tmp_path):
    assert os.path.exists(_build(tmp_path))


@pytest.mark.gpu
def test_example_runs(tmp_path):
    exe = _build(tmp_path)
    env = dict(os.environ, LD_LIBRARY_PATH=f"{PKG}:/opt/rocm/lib:" + os.environ.get("LD_LIBRARY_PATH", ""))
    print(f"[c example] {exe}", flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0 and "roundtrip ok" in r.stdout, r.stdout + r.stderr
