"""The library's host-side code under AddressSanitizer and
UndefinedBehaviorSanitizer, checked against the oracle on the CPU.

tests/sanitize/tier_fuzz.cpp links the product's host-only sources (the
tier's key map, recency list, pins and write admission, and the reuse-distance
capacity tool) with the oracle and drives both with the same seeded random
request streams: lookups with hits and edits, admission with and without a
published report, refused calls, allocation with eviction and exhaustion,
stores, pins held across requests, over-unpins, reports.  Every result and the
full metadata image must agree.  One long stream (80,000 requests) takes the
tier past the point where it starts dropping history no window can reach.
The oracle's hashing and copies also run on random ragged inputs (keys only
for full blocks; store then load reproduces pages and scales).  Planted
mistakes in a scratch copy of the tier (trimming one clock unit too much, a
hit not promoted) are caught by these seeds.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_33762_amd", "csrc")
ORACLE = os.path.join(ROOT, "oracle")
FLAGS = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
         "-fno-omit-frame-pointer"]
HIP_INCLUDE = "/opt/rocm/include"  # ea.h names hipStream_t from hip_runtime_api.h


@pytest.fixture(scope="module")
def fuzz_binary(tmp_path_factory):
    if not (shutil.which("gcc") and shutil.which("g++")):
        pytest.skip("gcc/g++ not available")
    if not os.path.exists(os.path.join(HIP_INCLUDE, "hip", "hip_runtime_api.h")):
        pytest.skip("HIP headers not available")
    d = tmp_path_factory.mktemp("sanitize")
    objs = []
    for src in ("eao.c", "eao_tier.c", "eao_stack.c"):
        o = str(d / (src + ".o"))
        subprocess.run(["gcc", "-std=c11"] + FLAGS + ["-c", os.path.join(ORACLE, src), "-o", o],
                       check=True)
        objs.append(o)
    exe = str(d / "tier_fuzz")
    subprocess.run(["g++", "-std=c++17"] + FLAGS +
                   ["-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                    "-I", HIP_INCLUDE, "-I", CSRC, "-I", ORACLE,
                    os.path.join(ROOT, "tests", "sanitize", "tier_fuzz.cpp"),
                    os.path.join(CSRC, "ea_tier_meta.cpp"), os.path.join(CSRC, "ea_stack.cpp")]
                   + objs + ["-o", exe], check=True)
    return exe


def run(exe, seed, requests):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe, str(seed), str(requests)], capture_output=True, text=True,
                       env=env, timeout=300)
    assert r.returncode == 0, f"seed {seed}: {r.stdout}\n{r.stderr}"
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr


@pytest.mark.parametrize("seed", range(1, 25))
def test_random_streams_match_the_oracle_under_sanitizers(fuzz_binary, seed):
    run(fuzz_binary, seed, 3000)


def test_long_stream_with_bounded_history_under_sanitizers(fuzz_binary):
    run(fuzz_binary, 99, 80_000)
