"""AddressSanitizer and UndefinedBehaviorSanitizer builds of the CPU oracle
and of the C-ABI library's host code, driven on the CPU.

tests/sanitize/oracle_driver.c runs every oracle function on small,
edge-case-heavy inputs (hub and isolated vertices, empty batches, undersized
capacities, out-of-range ids, every dtype pair); tests/sanitize/abi_driver.c
runs the host validation of every entry point with bad and good arguments
(nothing reaches the GPU).  Both must exit 0 with no sanitizer report.  The
library objects are built once per source state (cached by a hash of the
sources), with the sanitizers on the host pass only.
"""
import concurrent.futures as cf
import glob
import hashlib
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2303_00158_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
CACHE = os.path.join(ROOT, "paper_2303_00158_amd", "_build", "sanitize")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
SAN = "-fsanitize=address,undefined"
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def _run(exe, env):
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out
    assert "runtime error" not in out and "AddressSanitizer" not in out and "LeakSanitizer" not in out, out
    return out


def test_oracle_under_asan_and_ubsan(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not found")
    exe = str(tmp_path / "oracle_driver")
    cmd = ["gcc", "-std=c11", "-g", "-O1", "-fno-omit-frame-pointer", SAN, "-fno-sanitize-recover=undefined",
           "-ffp-contract=off", "-fopenmp", "-o", exe, os.path.join(HERE, "oracle_driver.c"),
           os.path.join(ROOT, "oracle", "oracle.c"), "-lm"]
    subprocess.run(cmd, check=True)
    assert "oracle driver: ok" in _run(exe, ENV)


def _sources_hash():
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(CSRC, "*")) + [os.path.join(INCLUDE, "gnn.h"),
                                                         os.path.join(HERE, "abi_driver.c")]):
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode() + fh.read())
    return h.hexdigest()[:16]


def test_abi_validation_under_asan_and_ubsan():
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not found")
    build = os.path.join(CACHE, _sources_hash())
    exe = os.path.join(build, "abi_driver")
    if not os.path.exists(exe):
        os.makedirs(build, exist_ok=True)
        flags = ["--offload-arch=gfx950", "-O1", "-g", "-fPIC", "-std=c++17", "-Xarch_host", SAN, "-Xarch_host",
                 "-fno-omit-frame-pointer", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", INCLUDE,
                 "-I", CSRC]

        def compile_one(src):
            obj = os.path.join(build, os.path.basename(src)[:-4] + ".o")
            subprocess.run([HIPCC, *flags, "-c", src, "-o", obj], check=True, capture_output=True)
            return obj

        srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
        with cf.ThreadPoolExecutor(min(8, os.cpu_count() or 1)) as ex:
            objs = list(ex.map(compile_one, srcs))
        drv = os.path.join(build, "driver.o")
        subprocess.run([HIPCC, "--offload-arch=gfx950", "-g", "-Xarch_host", SAN, "-I", INCLUDE, "-x", "c",
                        os.path.join(HERE, "abi_driver.c"), "-c", "-o", drv], check=True, capture_output=True)
        tmp = exe + ".tmp"
        subprocess.run([HIPCC, "--offload-arch=gfx950", "-Xarch_host", SAN, "-o", tmp, *objs, drv], check=True,
                       capture_output=True)
        os.replace(tmp, exe)
    env = dict(ENV, ASAN_OPTIONS="detect_leaks=0")  # the HIP runtime keeps its allocations until exit
    assert "abi driver: ok" in _run(exe, env)
