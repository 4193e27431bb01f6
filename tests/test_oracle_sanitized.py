"""The oracle's C code under AddressSanitizer and UBSan (CPU only).

The oracle keeps hand-grown request arrays (realloc, memmove) and mixes int64,
__int128 and binary128 arithmetic; a sanitized build runs the pins that drive
every part of it (brute-force placements with heartbeats, decode history and
moves, grouped placement, Algorithm 2) and must finish with no report."""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

from oracle import ref

HERE = os.path.dirname(os.path.abspath(__file__))


def test_oracle_pins_under_asan_and_ubsan(tmp_path):
    asan = subprocess.check_output(["gcc", "-print-file-name=libasan.so"], text=True).strip()
    if not os.path.isabs(asan) or not os.path.exists(asan):
        pytest.skip("gcc has no AddressSanitizer runtime here")
    lib = tmp_path / "liboracle_san.so"
    subprocess.check_call(["gcc", "-O1", "-g", "-std=gnu11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
                           "-fPIC", "-shared", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                           "-fno-omit-frame-pointer", "-o", str(lib), ref.SRC, "-lm"])
    env = dict(os.environ, LD_PRELOAD=asan, ORACLE_LIB=str(lib),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    sel = ("bruteforce or worked or footprint or lone or ties or router or grouped or rebalance or "
           "preemption or moves or move_ or invalid or sweep")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
                        os.path.join(HERE, "test_oracle.py"), "-k", sel],
                       env=env, cwd=os.path.dirname(HERE), capture_output=True, text=True, timeout=1200)
    tail = (r.stdout[-4000:] + "\n" + r.stderr[-4000:])
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in tail and "runtime error" not in tail, tail
    assert " passed" in r.stdout, tail
