"""The oracle's C library under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

A scratch copy of the oracle, the workload generator and the oracle pin tests
is built with ``-fsanitize=address,undefined`` (gcc, host code only; every
sanitizer report aborts) and the pin tests run against that build in a
subprocess with the ASan runtime preloaded into Python.  An out-of-bounds
access, a use after free, a signed overflow, a misaligned load or a shift out
of range anywhere the pins reach fails this test.  The repository's own
oracle build is never touched.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

import pytest

from oracle import build as oracle_build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

PIN_FILES = ["test_oracle_routing.py", "test_oracle_layout.py", "test_oracle_moe.py",
             "test_oracle_adjustment.py"]

SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]


def _runtime(name: str) -> str | None:
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_pins_pass_under_asan_and_ubsan():
    asan = _runtime("libasan.so")
    if shutil.which("gcc") is None or asan is None:
        pytest.skip("gcc with the AddressSanitizer runtime is not installed")
    with tempfile.TemporaryDirectory(prefix="orc_san_") as tmp:
        shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(tmp, "oracle"),
                        ignore=shutil.ignore_patterns("*.so", "*.so.tmp*", "__pycache__"))
        shutil.copytree(os.path.join(ROOT, "workloads"), os.path.join(tmp, "workloads"),
                        ignore=shutil.ignore_patterns("__pycache__"))
        os.makedirs(os.path.join(tmp, "tests"))
        for f in ["conftest.py", "cases.py", *PIN_FILES]:
            shutil.copy(os.path.join(ROOT, "tests", f), os.path.join(tmp, "tests", f))
        shutil.copytree(os.path.join(ROOT, "tests", "golden"), os.path.join(tmp, "tests", "golden"))

        src = os.path.join(tmp, "oracle", "cap_oracle.c")
        lib = os.path.join(tmp, "oracle", "liboracle.so")
        # same flags as the regular oracle build, at -O1 so reports keep their frames
        cflags = [f for f in oracle_build.CFLAGS if f != "-O2"] + ["-O1", *SAN_FLAGS]
        r = subprocess.run(["gcc", *cflags, src, "-o", lib, "-lm"], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr
        # the loader rebuilds when the library is older than the source: keep it newer
        st = os.stat(src)
        os.utime(lib, (st.st_atime + 10, st.st_mtime + 10))

        env = dict(os.environ, PYTHONDONTWRITEBYTECODE="1", OMP_NUM_THREADS="2", LD_PRELOAD=asan,
                   ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:verify_asan_link_order=0",
                   UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
        # -s: pytest does not capture fd 2, so a report reaches the output before the abort
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-s", "-p", "no:cacheprovider", "-m", "not gpu",
                            *[os.path.join("tests", f) for f in PIN_FILES]],
                           cwd=tmp, env=env, capture_output=True, text=True, timeout=900)
        out = r.stdout[-4000:] + r.stderr[-4000:]
        assert r.returncode == 0, out
        assert "runtime error" not in out and "AddressSanitizer" not in out, out
        # the sanitized library, not a rebuilt plain one, was the one loaded
        assert os.path.getmtime(lib) == st.st_mtime + 10
