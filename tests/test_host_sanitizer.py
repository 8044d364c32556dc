"""The library's host code (argument validation, workspace carving and sizing,
the window rule, the host-pool pointer check) under AddressSanitizer and
UndefinedBehaviorSanitizer.  A copy of libLouisKV is built with both
sanitizers on its host code only (`-Xarch_host` before each flag; the device
code is built as usual) and a plain C program (tests/c_abi/validate_host.c)
linked with the same sanitizers calls every entry point with arguments that
must be refused before any launch.  CPU only: on a machine with a GPU the
test is skipped, so that no call can reach a device."""
import glob
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2510_11292_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang"

pytestmark = pytest.mark.slow


def _gpu_visible() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.mark.skipif(not os.path.exists(HIPCC) or not os.path.exists(CLANG), reason="ROCm toolchain not found")
@pytest.mark.skipif(_gpu_visible(), reason="runs only where no GPU can be reached")
def test_host_code_under_address_and_ub_sanitizers():
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-Xclang", "-target-feature", "-Xclang",
             "-packed-fp32-ops", "-Wno-unused-command-line-argument", "-I", os.path.join(ROOT, "include"),
             "-I", CSRC]
    with tempfile.TemporaryDirectory() as tmp:
        objs, procs = [], []
        for src in sorted(glob.glob(os.path.join(CSRC, "*.hip"))):
            obj = os.path.join(tmp, os.path.basename(src) + ".o")
            procs.append(subprocess.Popen([HIPCC, *flags, *san, "-c", src, "-o", obj], stderr=subprocess.PIPE,
                                          text=True))
            objs.append(obj)
        for pr in procs:
            _, err = pr.communicate()
            assert pr.returncode == 0, err[-3000:]
        lib = os.path.join(tmp, "liblouiskv.so")
        r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *san, *objs, "-o", lib],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        exe = os.path.join(tmp, "validate_host")
        r = subprocess.run([CLANG, "-std=c11", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                            "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c_abi", "validate_host.c"),
                            "-L", tmp, "-llouiskv", "-L/opt/rocm/lib", "-lamdhip64", f"-Wl,-rpath,{tmp}",
                            "-Wl,-rpath,/opt/rocm/lib", "-o", exe], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
                   UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
        r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
        print(r.stdout[-2000:])
        assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-4000:]
        assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-2000:])
        assert "0 failed checks" in r.stdout
