"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The tree validation and window encoder of the library (csrc/encode.cpp) and the C oracle
are built with g++ / gcc and both sanitizers, then driven over random full trees at every
window depth 1..8, special values, row strides above the feature count, and corrupted
trees (tests/sanitize/*).  Any out-of-bounds access, use of freed memory or undefined
arithmetic aborts the driver; so does a window walk that reaches another leaf than the
direct walk of the tree.  The two drivers are separate programs: the oracle and the
library share no code.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
       "-fno-omit-frame-pointer"]


def _build(tmp_path, compiler, std, sources, name, includes=(), libs=()):
    if shutil.which(compiler) is None:
        pytest.skip("%s not available" % compiler)
    exe = str(tmp_path / name)
    cmd = ([compiler, std] + SAN + ["-I" + os.path.join(ROOT, d) for d in includes] +
           [os.path.join(ROOT, s) for s in sources] + list(libs) + ["-o", exe])
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return exe


def _run(exe, seed, n):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe, str(seed), str(n)], capture_output=True, text=True, env=env,
                       timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("ok"), r.stdout + r.stderr


def test_encoder_under_sanitizers(tmp_path):
    exe = _build(tmp_path, "g++", "-std=c++17",
                 ["tests/sanitize/encode_fuzz.cpp", "paper_1111_1373_amd/csrc/encode.cpp"],
                 "encode_fuzz", includes=("include", "paper_1111_1373_amd/csrc"))
    for seed in (1, 2, 3):
        _run(exe, seed, 400)


def test_oracle_under_sanitizers(tmp_path):
    exe = _build(tmp_path, "gcc", "-std=c99",
                 ["tests/sanitize/oracle_fuzz.c", "oracle/dtree_oracle.c"], "oracle_fuzz",
                 libs=("-lm",))
    for seed in (1, 2, 3):
        _run(exe, seed, 1000)
