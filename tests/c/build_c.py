"""Build the plain-C consumer of the C ABI (tests/c/round_c_abi.c) against
the in-tree libdedloc.so and the oracle's liboracle.so (test infrastructure).

    python -m tests.c.build_c
"""

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "round_c_abi.c")
BIN = os.path.join(HERE, "round_c_abi")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build() -> str:
    """Compile and link the C program; returns its path."""
    pkg, orc = os.path.join(ROOT, "paper_2106_10207_amd"), os.path.join(ROOT, "oracle")
    tmp = BIN + ".tmp"
    subprocess.check_call([
        "gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
        "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), SRC, "-o", tmp,
        "-L", pkg, "-ldedloc", "-L", orc, "-loracle", "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm",
        # found next to the binary wherever the tree is copied
        "-Wl,-rpath,$ORIGIN/../../paper_2106_10207_amd:$ORIGIN/../../oracle:" + os.path.join(ROCM, "lib"),
    ])
    os.replace(tmp, BIN)
    return BIN


if __name__ == "__main__":
    print(build())
