"""AddressSanitizer pass over the library's host code (CPU only): the C-ABI layer
(bc_api.cpp: argument checks, the buffer registry, bc_fold_bn, bc_repack_weights) is
rebuilt with ASan instrumentation on the host side only, linked with the already built
kernel objects into a separate library under the build directory, and driven by
tests/asan_driver.c, which exercises every validation path with exact-size heap arrays
and fake device addresses (all rejected before anything is enqueued). Any host memory
error makes the driver abort."""
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2108_09376_amd")
BUILD = os.path.join(PKG, "_build")

no_gpu = pytest.mark.skipif(__import__("torch").cuda.is_available(),
                            reason="the driver passes fake device addresses; run where no GPU is visible")


def _hipcc():
    for c in ("/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    pytest.skip("hipcc not found")


@no_gpu
def test_host_code_under_address_sanitizer(tmp_path):
    objs = [o for o in glob.glob(os.path.join(BUILD, "*.o")) if not o.endswith("bc_api.cpp.o")]
    if not objs:
        from paper_2108_09376_amd import build
        build.build()
        objs = [o for o in glob.glob(os.path.join(BUILD, "*.o")) if not o.endswith("bc_api.cpp.o")]
    hipcc = _hipcc()
    asan_obj = str(tmp_path / "bc_api_asan.o")
    lib = str(tmp_path / "libblockcopy_asan.so")
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-fPIC", "-std=c++17", "-fno-omit-frame-pointer",
             "-Xarch_host", "-fsanitize=address"]
    subprocess.check_call([hipcc, *flags, "-I", os.path.join(ROOT, "include"), "-c",
                           os.path.join(PKG, "csrc", "bc_api.cpp"), "-o", asan_obj],
                          stderr=subprocess.DEVNULL)
    subprocess.check_call([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-Xarch_host",
                           "-fsanitize=address", "-o", lib, asan_obj, *objs], stderr=subprocess.DEVNULL)
    clang = shutil.which("clang") or "/opt/rocm/llvm/bin/clang"
    exe = str(tmp_path / "asan_driver")
    subprocess.check_call([clang, "-fsanitize=address", "-g", "-O1", "-o", exe,
                           os.path.join(ROOT, "tests", "asan_driver.c"), lib, "-lm",
                           f"-Wl,-rpath,{tmp_path}"])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:abort_on_error=0")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    print(r.stdout, r.stderr[-4000:])
    assert r.returncode == 0 and "asan driver ok" in r.stdout
    assert "ERROR: AddressSanitizer" not in r.stderr and "ERROR: LeakSanitizer" not in r.stderr
