"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU).

The oracle (plain C) and the host half of the library (argument
validation, shard bounds, weights, tile tables and the load-balancing LP of
api.hip and balance.cpp; the device code is built as usual) are rebuilt with
ASan + UBSan, and the whole CPU test suite runs against those builds in a
child process.  Any sanitizer report is written to a log file and fails the
test, as does any failing test.  The GPU is never touched."""

import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _runtime(name):
    path = subprocess.check_output(["gcc", f"-print-file-name={name}"]).decode().strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def _build_oracle(out):
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                           "-fno-fast-math", "-Wall", "-Wextra", "-Werror", *SAN,
                           os.path.join(ROOT, "oracle", "dedloc_oracle.c"), "-o", out, "-lm"])


def _build_library(out, objdir):
    sys.path.insert(0, ROOT)
    from paper_2106_10207_amd import build as B
    host_san = [flag for f in SAN for flag in ("-Xarch_host", f)]  # host code only
    objs = []
    for src in B.SOURCES:
        obj = os.path.join(objdir, src.replace(".hip", ".o"))
        subprocess.check_call([B.hipcc(), *B.HIP_FLAGS, "-g", *host_san, "-c", os.path.join(B.CSRC, src),
                               "-o", obj], stderr=subprocess.DEVNULL)
        objs.append(obj)
    for src in B.HOST_SOURCES:
        obj = os.path.join(objdir, src.replace(".cpp", ".o"))
        subprocess.check_call(["g++", "-O1", "-g", "-std=c++17", "-fPIC", *SAN, "-I", os.path.join(ROOT, "include"),
                               "-c", os.path.join(B.CSRC, src), "-o", obj])
        objs.append(obj)
    subprocess.check_call([B.hipcc(), f"--offload-arch={B.ARCH}", "-shared", "-fPIC", *host_san, *objs,
                           "-o", out], stderr=subprocess.DEVNULL)


def test_cpu_suite_under_asan_and_ubsan(tmp_path):
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not (asan and ubsan and shutil.which("gcc")):
        pytest.skip("gcc's sanitizer runtimes are not installed")
    oracle_lib = str(tmp_path / "liboracle_san.so")
    lib = str(tmp_path / "libdedloc_san.so")
    _build_oracle(oracle_lib)
    _build_library(lib, str(tmp_path))
    logs = str(tmp_path / "report")
    env = dict(os.environ)
    env.update(LD_PRELOAD=f"{asan}:{ubsan}",
               ASAN_OPTIONS=f"detect_leaks=0:log_path={logs}",  # the interpreter's own allocations are not ours
               UBSAN_OPTIONS=f"print_stacktrace=1:log_path={logs}")
    # left out: this file, and the tests that build and run oracles of their
    # own (the mutants, the oracle's fast build), which the sanitized
    # libraries are not part of
    ignore = []
    for name in (os.path.basename(__file__), "test_oracle_mutants.py", "test_oracle_fast_build.py"):
        ignore += ["--ignore", os.path.join(ROOT, "tests", name)]
    code = (
        "import sys\n"
        "import oracle\n"
        "from paper_2106_10207_amd import dedloc as D\n"
        f"oracle._LIB = {oracle_lib!r}\n"
        f"D.LIB_PATH = {lib!r}\n"
        "import pytest\n"
        "sys.exit(pytest.main(['-x', '-q', '-p', 'no:cacheprovider', '-m', 'not gpu',\n"
        f"                      *{ignore!r}, 'tests']))\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=1200)
    reports = sorted(glob.glob(logs + "*"))
    text = "".join(open(f).read() for f in reports)
    assert not reports, text[:4000]
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert " passed" in r.stdout
