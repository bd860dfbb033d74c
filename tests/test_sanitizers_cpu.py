"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU):
the library's argument checks (paper_2608_18656_amd/csrc/fa_checks.h, the
code every entry point runs before touching the device) over a grid of
valid, extreme and overflowing arguments, and the fp64 oracles (attention,
rows, weights, Q8_0 product) on small and edge shapes.  Built with g++/gcc;
any sanitizer report or failed check fails the test."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-g", "-O1", "-fno-omit-frame-pointer", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]


def _build_and_run(cmd, exe):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0 and "sanitize" in r.stderr and "cannot find" in r.stderr:
        pytest.skip("sanitizer runtime not installed")
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr, r.stderr
    return r.stdout


def test_argument_checks_under_sanitizers(tmp_path):
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("no g++")
    exe = str(tmp_path / "checks")
    out = _build_and_run([cxx, "-std=c++17", "-Wall", "-Werror", *SAN, "-I", os.path.join(ROOT, "include"),
                          os.path.join(ROOT, "tests", "sanitize", "checks_driver.cpp"), "-o", exe], exe)
    assert "argument sets" in out


def test_oracles_under_sanitizers(tmp_path):
    cc = shutil.which("gcc")
    if cc is None:
        pytest.skip("no gcc")
    exe = str(tmp_path / "oracles")
    out = _build_and_run([cc, "-std=c11", "-Wall", "-Werror", "-ffp-contract=off", *SAN,
                          os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c"),
                          os.path.join(ROOT, "oracle", "fa_oracle.c"), os.path.join(ROOT, "oracle", "q8_oracle.c"),
                          "-o", exe, "-lm"], exe)
    assert "ok" in out
