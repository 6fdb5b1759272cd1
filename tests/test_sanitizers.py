"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

- The input generators and the CPU oracle, built with gcc and both
  sanitizers, run every entry point on small matrices of every family
  (tests/sanitize/host_driver.c).
- The library's host code (planner, path routing, argument validation),
  built with the sanitizers on its host side only (-Xarch_host before each
  -fsanitize=, so no device code is instrumented), runs its host-only entry
  points (tests/sanitize/library_driver.cpp); no GPU is touched.
"""
import concurrent.futures as cf
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2607_22866_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host",
            "-fno-sanitize-recover=all"]


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, "%s\n%s\n%s" % (" ".join(cmd), r.stdout[-4000:], r.stderr[-4000:])
    return r


def test_generators_and_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "host_driver")
    _run(["gcc", "-O1", "-g", "-fopenmp", *SAN, "-o", exe, os.path.join(HERE, "host_driver.c"),
          os.path.join(ROOT, "workloads", "gen.c"), os.path.join(ROOT, "oracle", "spgemm_oracle.c"), "-lm"])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1", OMP_NUM_THREADS="4")
    r = _run([exe], env=env)
    assert r.stdout.count(" ok") == 7


@pytest.mark.skipif(not os.path.exists(HIPCC) or shutil.which("g++") is None, reason="needs hipcc and g++")
def test_library_host_code_under_sanitizers(tmp_path):
    from paper_2607_22866_amd import build

    def compile_one(src):
        obj = str(tmp_path / (os.path.splitext(src)[0] + ".o"))
        _run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-Xclang", "-target-feature",
              "-Xclang", "-packed-fp32-ops", *HOST_SAN, "-I", os.path.join(ROOT, "include"), "-c",
              os.path.join(CSRC, src), "-o", obj])
        return obj

    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 4)) as ex:
        objs = list(ex.map(compile_one, build.SOURCES))
    drv = str(tmp_path / "driver.o")
    _run(["g++", "-O1", "-g", "-std=c++17", *SAN, "-c", os.path.join(HERE, "library_driver.cpp"), "-o", drv])
    exe = str(tmp_path / "library_driver")
    _run([HIPCC, "--offload-arch=gfx950", *HOST_SAN, "-o", exe, drv, *objs])
    # the HIP runtime keeps allocations until exit; leaks are not this test's subject
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1")
    r = _run([exe], env=env)
    assert "library host checks ok" in r.stdout
