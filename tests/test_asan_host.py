"""The host side of the library under AddressSanitizer (CPU only).

liboc_asan.so is the same library with its host code instrumented: argument
and shape checks, planning and workspace layout, the Layered Cache schedule,
the stage timer, the error record.  The CPU tests that load the library run
against it in a child process with the sanitizer runtime preloaded: every
rejection path of the C-ABI, the plan and workspace queries, and the
schedule on tables of many shapes must pass with no sanitizer report.  A
positive control first shows that the preloaded runtime does report a
planted heap overflow in a throwaway host snippet built with the same flags,
so a clean run means something.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
from paper_2607_23844_amd import build as B  # noqa: E402

LIB_TESTS = ["tests/test_abi.py", "tests/test_oracle_layered.py", "tests/test_bench_host.py"]


@pytest.fixture(scope="module")
def asan_env(tmp_path_factory):
    lib = B.build(asan=True)
    env = dict(os.environ)
    env.update(LD_PRELOAD=B.asan_runtime(), OC_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:alloc_dealloc_mismatch=0:abort_on_error=0:exitcode=86")
    return env, tmp_path_factory.mktemp("asan")


def test_sanitizer_runtime_reports_a_planted_overflow(asan_env):
    env, tmp = asan_env
    src = tmp / "planted.cpp"
    src.write_text('#include <cstdlib>\n'
                   'extern "C" int planted(int n) {\n'
                   '    int *a = (int *)std::malloc(4 * n); int s = 0;\n'
                   '    for (int i = 0; i <= n; ++i) s += a[i];   // one past the end\n'
                   '    std::free(a); return s;\n'
                   '}\n')
    so = tmp / "planted.so"
    subprocess.run([B._hipcc(), "-O1", "-fPIC", "-shared", *B.ASAN_FLAGS, "-o", str(so), str(src)], check=True,
                   capture_output=True)
    r = subprocess.run([sys.executable, "-c", f"import ctypes; ctypes.CDLL({str(so)!r}).planted(4)"], env=env,
                       capture_output=True, text=True)
    assert r.returncode == 86 and "heap-buffer-overflow" in r.stderr, r.stderr[-2000:]


def test_library_host_paths_clean_under_asan(asan_env):
    env, _ = asan_env
    # the child loads the sanitized build (checked through the loader's path)
    probe = subprocess.run([sys.executable, "-c",
                            "import paper_2607_23844_amd._lib as L; L.lib(); print(L.LIB_PATH)"],
                           env=env, cwd=ROOT, capture_output=True, text=True)
    assert probe.returncode == 0 and probe.stdout.strip().endswith("liboc_asan.so"), probe.stderr[-2000:]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-m", "not gpu", "-p", "no:cacheprovider", *LIB_TESTS],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=600)
    assert "AddressSanitizer" not in r.stderr + r.stdout, (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert " passed" in r.stdout
