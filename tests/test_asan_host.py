"""The host code of the library under AddressSanitizer, without a GPU: the
translation unit that holds the ABI and the host orchestration is compiled with
-fsanitize=address for its host code only (the device code of the same file is
built as usual), linked with the library's kernel objects, and driven by a C99
program (tests/c_client/asan_host.c) through the paths that run without a
device: argument and snapshot validation, the threaded per-row sort of a 1.6M-arc
snapshot, the error path when no device can be selected, and ripple_destroy of
partly built contexts. Any heap or stack error, or use after free, aborts the
program with a report."""
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2505_12112_amd")
CLANG = "/opt/rocm/llvm/bin/clang"


@pytest.mark.slow
def test_host_code_under_address_sanitizer(tmp_path):
    from paper_2505_12112_amd import build as B
    try:
        hipcc = B.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    kernels = sorted(glob.glob(os.path.join(PKG, "_build", "k_*.hip.o")))
    if len(kernels) < 3 or not os.path.exists(CLANG):
        pytest.skip("the library is not built (run __graft_entry__.build())")
    host_obj = tmp_path / "ripple_api_asan.o"
    flags = [f for f in B.HIPCC_FLAGS]
    sanitize = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]
    subprocess.run([hipcc, *flags, *sanitize, "-c", os.path.join(PKG, "csrc", "ripple_api.hip"), "-o",
                    str(host_obj)], check=True, capture_output=True)
    lib = tmp_path / "libripple.so"
    subprocess.run([hipcc, f"--offload-arch={B.ARCH}", "-shared", "-fPIC", "-Xarch_host", "-fsanitize=address",
                    str(host_obj), *kernels, "-o", str(lib)], check=True, capture_output=True)
    exe = tmp_path / "asan_host"
    subprocess.run([CLANG, "-std=c99", "-g", "-fsanitize=address", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c_client", "asan_host.c"), "-L", str(tmp_path), "-lripple",
                    f"-Wl,-rpath,{tmp_path}", "-o", str(exe)], check=True, capture_output=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", HIP_VISIBLE_DEVICES="")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0 and "asan host ok" in r.stdout, r.stdout[-3000:] + r.stderr[-3000:]
    assert "AddressSanitizer" not in r.stderr, r.stderr[-3000:]
