"""The library's host code (arithmetic coder, container header parser,
deserialiser) under AddressSanitizer and UndefinedBehaviorSanitizer: a
randomised harness (tests/host_fuzz.cpp) is built with g++ against
csrc/coder.cpp and run on three seeds.  Any out-of-bounds access, signed
overflow or a decode mismatch on an intact stream fails the test.  The
oracle's C coder gets the same treatment (tests/oracle_fuzz.c); the two
harnesses share nothing."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_coder_and_parser_under_sanitizers(tmp_path):
    exe = str(tmp_path / "host_fuzz")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-pthread", os.path.join(HERE, "host_fuzz.cpp"),
           os.path.join(ROOT, "paper_2409_17836_amd", "csrc", "coder.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0", UBSAN_OPTIONS="print_stacktrace=1")
    for seed in (1, 2, 3):
        r = subprocess.run([exe, str(seed)], capture_output=True, text=True, env=env, timeout=300)
        assert r.returncode == 0, (seed, r.stdout[-500:], r.stderr[-3000:])
        assert "mismatches 0" in r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_coder_under_sanitizers(tmp_path):
    """The oracle's C coder under the same sanitizers (tests/oracle_fuzz.c):
    quantised tables keep their invariants, symbol strings and byte vectors
    round-trip."""
    exe = str(tmp_path / "oracle_fuzz")
    cmd = ["gcc", "-std=gnu11", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", os.path.join(HERE, "oracle_fuzz.c"),
           os.path.join(ROOT, "oracle", "coder.c"), "-lm", "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0")
    for seed in (1, 2):
        r = subprocess.run([exe, str(seed)], capture_output=True, text=True, env=env, timeout=300)
        assert r.returncode == 0, (seed, r.stdout[-500:], r.stderr[-3000:])
