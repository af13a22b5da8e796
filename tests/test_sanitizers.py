"""The host half of the library (page pool, planner, pass validation, pacing)
under AddressSanitizer and UndefinedBehaviorSanitizer.

The sanitizer build (libpdec_host_san.so, `python -m paper_2609_36899_amd.build
--sanitize`) makes every finding fatal; the host tests run against it in a
child interpreter with the sanitizer runtimes preloaded.  CPU only."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _have_sanitizers():
    try:
        from paper_2609_36899_amd import build
        return all(os.path.isabs(p) and os.path.exists(p)
                   for p in build.sanitizer_preload().split(":"))
    except (OSError, subprocess.CalledProcessError):
        return False


@pytest.mark.skipif(not _have_sanitizers(), reason="g++ sanitizer runtimes not installed")
def test_host_library_tests_pass_under_asan_and_ubsan():
    from paper_2609_36899_amd import build
    lib = build.build_host(sanitize=True)
    env = dict(os.environ)
    env.update(PDEC_HOST_LIB=lib, LD_PRELOAD=build.sanitizer_preload(),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1",
               PYTHONPATH=ROOT)
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_host_pool.py")],
                       cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                       text=True, timeout=600)
    tail = r.stdout[-4000:]
    assert r.returncode == 0, tail
    assert "passed" in tail and "AddressSanitizer" not in tail and "runtime error" not in tail


@pytest.mark.skipif(not _have_sanitizers(), reason="g++ sanitizer runtimes not installed")
def test_sanitizer_build_catches_a_planted_overflow(tmp_path):
    """The preload and flags do detect a heap overflow (the check is live;
    UBSan's object-size check or ASan may report it first)."""
    from paper_2609_36899_amd import build
    src = tmp_path / "bad.cpp"
    src.write_text('extern "C" int bad(int i) { int* p = new int[4]; int v = p[i]; '
                   'delete[] p; return v; }\n')
    so = tmp_path / "libbad.so"
    subprocess.run(["g++", *build.SANITIZE_FLAGS, "-shared", "-fPIC", str(src), "-o", str(so)],
                   check=True)
    env = dict(os.environ, LD_PRELOAD=build.sanitizer_preload(),
               ASAN_OPTIONS="detect_leaks=0")
    code = f"import ctypes; ctypes.CDLL({str(so)!r}).bad(4)"
    r = subprocess.run([sys.executable, "-c", code], env=env, stdout=subprocess.PIPE,
                       stderr=subprocess.STDOUT, text=True, timeout=120)
    assert r.returncode != 0
    assert "heap-buffer-overflow" in r.stdout or "runtime error" in r.stdout, r.stdout[-2000:]
