"""The C ABI from plain C (tests/c/round_c_abi.c): a C11 program that uses
include/dedloc.h and the HIP runtime's C API only, with hipMalloc'd buffers,
and checks the library against the oracle it also links.

* host (no GPU): the header compiles as C11 with -Wall -Wextra -Werror, the
  program links against libdedloc.so, and the host-only entry points
  (partition, weights, encoded sizes) and argument validation (zero
  weights, misaligned buffers, bad tensor tables, no peers) behave as
  declared;
* gpu: whole fp16 and int8 rounds (with and without the local peer's fp32
  gradient) and the encode, compared with the oracle to the usual bars."""

import os
import subprocess

import pytest

from tests.c import build_c


def _binary():
    srcs = [build_c.SRC, os.path.join(build_c.ROOT, "include", "dedloc.h")]
    libs = [os.path.join(build_c.ROOT, "paper_2106_10207_amd", "libdedloc.so"),
            os.path.join(build_c.ROOT, "oracle", "liboracle.so")]
    if not all(os.path.exists(p) for p in libs):
        pytest.skip("build the libraries first (__graft_entry__.build())")
    if not os.path.exists(build_c.BIN) or os.path.getmtime(build_c.BIN) < max(os.path.getmtime(p) for p in srcs):
        build_c.build()
    return build_c.BIN


def _run(*args):
    env = {k: v for k, v in os.environ.items() if k != "LD_PRELOAD"}  # a plain process
    return subprocess.run([_binary(), *args], capture_output=True, text=True, timeout=300, env=env)


def test_c_abi_host():
    r = _run("--host")
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c-abi host checks: ok" in r.stdout


@pytest.mark.gpu
def test_c_abi_rounds_on_device():
    r = _run()
    print(r.stdout, flush=True)
    assert r.returncode == 0, r.stdout + r.stderr
    # host checks, then four rounds (fp16 / int8, with and without the local
    # peer), each also through dedloc_round_noalloc
    assert r.stdout.count(": ok") == 9, r.stdout
