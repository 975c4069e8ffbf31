"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

A build of the library whose host sources -- prefix metadata, work planner,
prefix-aware scheduler, KV-allocation search and the C ABI's validation --
g++ compiles with both sanitizers runs the CPU tests of that host logic in a
child process with the ASan runtime preloaded; any report ends the child with
an error. A positive control first shows that the same flags catch a heap
overflow in a throwaway snippet, so a silent sanitizer cannot pass the test.
"""

from __future__ import annotations

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HOST_TESTS = ["tests/test_host_meta.py", "tests/test_host_plan.py", "tests/test_schedule.py", "tests/test_kv_alloc.py"]


def _asan_runtime():
    r = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    if r.returncode != 0 or not os.path.isabs(path) or not os.path.exists(path):
        pytest.skip("g++ has no ASan runtime here")
    return path


def _env(asan, lib=None):
    env = dict(os.environ)
    env.update(LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    if lib:
        env["TTS_LIBRARY"] = lib
    return env


def test_sanitizer_flags_catch_a_planted_overflow(tmp_path):
    from paper_2509_00195_amd.build import SANITIZE

    asan = _asan_runtime()
    src = tmp_path / "overflow.cpp"
    src.write_text("#include <vector>\nint main(int c, char**) { std::vector<int> v(4); v.data()[4 + c] = 1; "
                   "return v[0]; }\n")
    exe = tmp_path / "overflow"
    subprocess.run(["g++", *SANITIZE, str(src), "-o", str(exe)], check=True, capture_output=True)
    r = subprocess.run([str(exe)], env=_env(asan), capture_output=True, text=True)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr


def test_host_logic_clean_under_asan_and_ubsan(tmp_path):
    from paper_2509_00195_amd.build import build_sanitized

    asan = _asan_runtime()
    lib = build_sanitized(str(tmp_path / "libtts_san.so"))
    env = _env(asan, lib)
    # the child loads the sanitized build, with the ASan runtime in the process
    probe = ("import paper_2509_00195_amd.tts as t; t.load(); "
             "maps = open('/proc/self/maps').read(); "
             f"assert t.LIB_PATH == {lib!r} and 'libasan' in maps and {lib!r} in maps")
    r = subprocess.run([sys.executable, "-c", probe], env=env, cwd=ROOT, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", *HOST_TESTS],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=1500)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert " passed" in r.stdout and "failed" not in r.stdout
