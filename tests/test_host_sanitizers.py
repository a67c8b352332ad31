"""The host-only library code under AddressSanitizer and UBSan (CPU only).

tests/host_sanitize/driver.cpp exercises the tile schedules, the topology map
and its cache file, the latency, partition-hash and home-map analyses, the
chunk lists and the attention page placement on synthetic inputs; it is built
with g++ (-fsanitize=address,undefined, no recovery) together with those
sources and stand-ins for the GPU-side symbols they reference, and must end
cleanly.  A planted overflow checks that the sanitizer is really active.
"""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_24270_amd", "csrc")
HOST_SOURCES = ["schedule.cpp", "topology.cpp", "topology_cache.cpp", "affinity.cpp", "interleave.cpp",
                "kv_place.cpp", "numa_host.cpp"]
FLAGS = ["-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
         "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I", os.path.join(ROOT, "include"), "-I", CSRC]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def build(out, sources):
    r = subprocess.run(["g++", *FLAGS, *sources, "-o", str(out)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]


def test_host_code_is_clean_under_sanitizers(tmp_path):
    exe = tmp_path / "driver"
    build(exe, [os.path.join(ROOT, "tests", "host_sanitize", "driver.cpp"),
                os.path.join(ROOT, "tests", "host_sanitize", "stubs.cpp")] +
          [os.path.join(CSRC, f) for f in HOST_SOURCES])
    r = subprocess.run([str(exe), str(tmp_path)], capture_output=True, text=True, env=ENV, timeout=300)
    assert r.returncode == 0 and "all checks passed" in r.stdout, (r.stdout[-3000:], r.stderr[-3000:])


def test_the_sanitizer_catches_a_planted_overflow(tmp_path):
    src = tmp_path / "planted.cpp"
    src.write_text("#include <vector>\nint main(int c, char**) { std::vector<int> v(4); return v.data()[3 + c]; }\n")
    exe = tmp_path / "planted"
    build(exe, [str(src)])
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=ENV, timeout=60)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr
