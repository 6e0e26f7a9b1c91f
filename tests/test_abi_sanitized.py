"""The C-ABI validation layer (csrc/api.cpp) under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU.

api.cpp is built for the host with g++ (no device code: the kernel
launchers are replaced by host stand-ins, tests/sanitize/launch_stubs.cpp)
into a shared library that the ctypes binding loads in place of
libnvfp4.so; then tests/test_abi.py runs against it in a child process with
the sanitizer runtime preloaded.  Any sanitizer report fails the run.
"""

import os
import shutil
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def _libasan():
    r = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.exists(os.path.join(ROCM, "lib", "libamdhip64.so")),
                    reason="needs g++ and the HIP runtime library")
def test_abi_validation_under_asan_ubsan():
    asan = _libasan()
    if asan is None:
        pytest.skip("no libasan for g++")
    tmp = tempfile.mkdtemp(prefix="nvfp4_san_")
    try:
        so = os.path.join(tmp, "libnvfp4_san.so")
        san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
        cmd = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-shared", "-D__HIP_PLATFORM_AMD__",
               "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
               "-I", os.path.join(ROOT, "paper_2609_04098_amd", "csrc")] + san + [
            os.path.join(ROOT, "paper_2609_04098_amd", "csrc", "api.cpp"),
            os.path.join(ROOT, "tests", "sanitize", "launch_stubs.cpp"),
            "-L", os.path.join(ROCM, "lib"), "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-lamdhip64",
            "-o", so]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        code = ("import sys; sys.path.insert(0, %r); "
                "import paper_2609_04098_amd.nvfp4 as C; C.LIB_PATH = %r; "
                "import pytest; sys.exit(pytest.main(['-q', '-p', 'no:cacheprovider', %r]))"
                % (ROOT, so, os.path.join(ROOT, "tests", "test_abi.py")))
        # PYTHONMALLOC=malloc: Python's own buffers (the ctypes arrays passed
        # in, e.g. segment tables) come from malloc, so the sanitizer guards
        # them too.  Reports go to files (pytest captures the child's stderr).
        logs = os.path.join(tmp, "report")
        env = dict(os.environ, LD_PRELOAD=asan, PYTHONDONTWRITEBYTECODE="1", PYTHONMALLOC="malloc",
                   HIP_VISIBLE_DEVICES="",
                   ASAN_OPTIONS="detect_leaks=0:verify_asan_link_order=0:exitcode=97:log_path=" + logs,
                   UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1:exitcode=98:log_path=" + logs)
        r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                           timeout=600)
        reports = [os.path.join(tmp, f) for f in os.listdir(tmp) if f.startswith("report")]
        text = "".join(open(f).read() for f in reports)
        assert not reports, text[:4000]
        assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
        assert " passed" in r.stdout
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
