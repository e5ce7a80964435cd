"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Builds tests/host/planner_check.cpp with the library's host sources (the planner,
the serialized-query parser and bulk ordering; none of them needs the GPU) by g++
with -fsanitize=address,undefined, twice:
- with the library's 64-bit page hashes;
- with SPANQ_TEST_HASH_BITS=6, which keeps six bits of every page hash, so that
  different pages collide all the time: the content check behind each index hit
  must turn every collision into a miss (section 2 looks blocks up by hash alone;
  this library also compares the stored tokens, page index and parent hash).
Each build runs random planning streams over small pools (evictions, refusals,
commit and release, both kernels' tilings, materialised repositioning) and checks
every hit against a shadow copy of what each page was written with, plus the
bounds of every page id and key range the kernels would read; then fuzzes the
parser and checks bulk orders are permutations.  Any sanitizer report fails the run.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2511_02749_amd", "csrc")
SOURCES = [os.path.join(ROOT, "tests", "host", "planner_check.cpp")] + [
    os.path.join(CSRC, f) for f in ("planner.cpp", "frontend.cpp", "bulk.cpp")]


def _build(tmp_path, hash_bits):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    exe = os.path.join(str(tmp_path), f"planner_check_{hash_bits or 64}")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"), "-I", CSRC]
    if hash_bits:
        cmd.append(f"-DSPANQ_TEST_HASH_BITS={hash_bits}")
    r = subprocess.run(cmd + SOURCES + ["-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return exe


@pytest.mark.parametrize("hash_bits", [0, 6], ids=["hash64", "hash6"])
def test_host_code_under_sanitizers(tmp_path, hash_bits):
    exe = _build(tmp_path, hash_bits)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    for seed in (1, 2, 3, 7):
        r = subprocess.run([exe, str(seed), "400"], capture_output=True, text=True, env=env, timeout=300)
        print(r.stdout, end="")
        assert r.returncode == 0, (r.stdout + r.stderr)[-6000:]
        assert "all checks passed" in r.stdout
