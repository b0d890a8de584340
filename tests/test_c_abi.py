"""The C ABI from C: a C99 program compiled against include/visionpulse.h and
linked to the built library runs its host-side checks (no GPU needed)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2605_31457_amd")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_c_client_compiles_links_and_runs(tmp_path):
    lib = os.path.join(PKG, "libvisionpulse.so")
    if not os.path.exists(lib):
        pytest.skip("library not built")
    exe = tmp_path / "abi_smoke"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "c", "abi_smoke.c"), "-L", PKG, "-lvisionpulse",
           f"-Wl,-rpath,{PKG}", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout
    # the struct sizes seen from C are the ones the Python binding declares
    import ctypes
    from paper_2605_31457_amd import vp
    assert f"sizeof vp_shape {ctypes.sizeof(vp.vp_shape)}," in r.stdout
    assert f"vp_layout {ctypes.sizeof(vp.vp_layout)}," in r.stdout
    assert f"vp_params {ctypes.sizeof(vp.vp_params)})" in r.stdout
