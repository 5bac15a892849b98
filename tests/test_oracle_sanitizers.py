"""The oracle built with AddressSanitizer and UndefinedBehaviorSanitizer (CPU only): every pin
runs against that build in a child process, with any sanitizer report fatal, so that an
out-of-bounds access, a use of freed memory, a signed overflow or a misaligned access in the
oracle fails the suite instead of going unnoticed."""
import os
import subprocess
import sys

import pytest

import oracle

TESTS = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(TESTS)


def _runtime(name: str) -> str:
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True,
                          check=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else ""


def test_pins_pass_under_asan_and_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    if not asan:
        pytest.skip("gcc has no AddressSanitizer runtime here")
    so = str(tmp_path / "liboracle_asan.so")
    oracle.build(extra_flags=["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                              "-fno-omit-frame-pointer", "-g"], out=so)
    code = ("import sys, oracle, pins\n"
            f"L = oracle.lib({so!r})\n"
            "for pin in pins.ALL_PINS:\n"
            "    pin(L)\n"
            "    print('ok', pin.__name__, flush=True)\n")
    env = dict(os.environ, PYTHONPATH=os.pathsep.join([ROOT, TESTS]), LD_PRELOAD=asan,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="4")
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert out.count("ok pin_") == len(__import__("pins").ALL_PINS), out[-2000:]
