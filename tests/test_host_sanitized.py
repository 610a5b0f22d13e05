"""The runtime's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only): build the library with both sanitizers on its host code
(build.build_host_sanitized), link tests/host_abi_driver.c against it with
the sanitizer runtime, and run it with every device hidden.  The driver goes
through the C ABI's validation and error paths -- bad shapes, null handles,
out-of-range batch shapes, a valid model whose allocation fails, an accept
call whose first HIP call fails -- and checks each status; any sanitizer
report aborts it."""
import os
import shutil
import subprocess

import pytest

from paper_2405_14105_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = shutil.which("clang", path="/opt/rocm/llvm/bin") or shutil.which("clang")


@pytest.mark.skipif(CLANG is None, reason="no clang to link the sanitizer runtime")
def test_host_abi_paths_under_asan_and_ubsan(tmp_path):
    lib = build.build_host_sanitized(str(tmp_path))
    exe = str(tmp_path / "host_abi_driver")
    r = subprocess.run([CLANG, "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                        "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "host_abi_driver.c"),
                        "-L", str(tmp_path), "-ldsi_san", f"-Wl,-rpath,{tmp_path}", "-o", exe],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ)
    env.update(ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", HIP_VISIBLE_DEVICES="-1",
               ROCR_VISIBLE_DEVICES="-1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert r.returncode == 0 and "host ABI paths ok" in r.stdout, out[-4000:]
    assert os.path.exists(lib)
