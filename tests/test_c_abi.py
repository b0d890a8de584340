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


def _clang_asan_runtime():
    import glob
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return os.path.dirname(hits[-1]) if hits else None


@pytest.mark.skipif(not os.path.exists("/opt/rocm/llvm/bin/clang") or _clang_asan_runtime() is None,
                    reason="clang or its sanitizer runtime not available")
def test_host_code_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    """The library's host code (argument checks, plans, workspace carving) built
    with AddressSanitizer and UBSan (host side only) and driven by the C client."""
    import sys
    sys.path.insert(0, ROOT)
    from paper_2605_31457_amd import build as B
    lib = tmp_path / "libvisionpulse.so"
    srcs = [os.path.join(B.CSRC, x) for x in B.SOURCES]
    flags = [f for f in B.HIPCC_FLAGS if f != "-O3"]
    cmd = [B.hipcc(), *flags, "-O1", "-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-I", B.INCLUDE, "-I", B.CSRC, *srcs, "-o", str(lib)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    rt = _clang_asan_runtime()
    exe = tmp_path / "abi_smoke_asan"
    cmd = ["/opt/rocm/llvm/bin/clang", "-std=c99", "-g", "-fsanitize=address,undefined", "-shared-libsan",
           "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c", "abi_smoke.c"),
           "-L", str(tmp_path), "-lvisionpulse", f"-Wl,-rpath,{tmp_path}", f"-Wl,-rpath,{rt}", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout
