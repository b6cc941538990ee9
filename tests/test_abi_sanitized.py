"""The C ABI layer (vidax.cpp: argument validation, overlap checks, status
strings) built with AddressSanitizer and UndefinedBehaviorSanitizer on the
host side, running the CPU ABI tests (tests/test_lib_abi.py) in a child
process.  The kernel launchers are replaced by stand-ins that fail loudly
(tests/abi_stub_launchers.cpp): none of these checks may reach a launch.  No
GPU code is instrumented (the sanitizer flags apply to the host pass only)."""

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


def _asan_runtime():
    try:
        out = subprocess.run([HIPCC, "--print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                             text=True, timeout=60).stdout.strip()
    except (OSError, subprocess.SubprocessError):
        return None
    if out and os.path.isabs(out) and os.path.exists(out):
        return out
    import glob

    cands = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return cands[-1] if cands else None


def test_abi_checks_under_asan_and_ubsan(tmp_path):
    rt = _asan_runtime()
    if not os.path.exists(HIPCC) or rt is None:
        pytest.skip("hipcc or the sanitizer runtime is not available")
    lib = str(tmp_path / "libvidax_san.so")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-fPIC", "-shared", "-std=c++17",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2609_18077_amd", "csrc"),
           os.path.join(ROOT, "paper_2609_18077_amd", "csrc", "vidax.cpp"),
           os.path.join(ROOT, "tests", "abi_stub_launchers.cpp"), "-o", lib]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert res.returncode == 0, res.stderr[-4000:]
    runner = tmp_path / "run.py"
    runner.write_text(
        "import sys\n"
        f"sys.path.insert(0, {ROOT!r})\n"
        "import paper_2609_18077_amd as vx\n"
        f"vx.LIB_PATH = {lib!r}\n"
        "import pytest\n"
        f"sys.exit(pytest.main(['-q', '-p', 'no:cacheprovider', {os.path.join(ROOT, 'tests', 'test_lib_abi.py')!r}]))\n")
    env = dict(os.environ, LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    res = subprocess.run([sys.executable, str(runner)], capture_output=True, text=True, timeout=600, env=env,
                         cwd=str(tmp_path))
    assert res.returncode == 0, (res.stdout[-4000:], res.stderr[-4000:])
    assert " passed" in res.stdout
