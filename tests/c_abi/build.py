"""Compile caller.c, the plain C user of the library, next to this file.

gcc, C11, against include/diffopt.h and the HIP runtime API; linked to the
in-tree libdiffopt.so through a relative run path, so the built tree can move
(the library must be built first).
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
BIN = os.path.join(HERE, "caller")


def build() -> str:
    tmp = BIN + ".tmp%d" % os.getpid()
    subprocess.check_call([
        "gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
        "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
        os.path.join(HERE, "caller.c"), "-o", tmp,
        "-L", os.path.join(ROOT, "paper_2211_06934_amd"), "-ldiffopt",
        "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
        "-Wl,-rpath,$ORIGIN/../../paper_2211_06934_amd", "-Wl,-rpath," + os.path.join(ROCM, "lib")])
    os.replace(tmp, BIN)
    return BIN


if __name__ == "__main__":
    print(build())
