"""Build the C oracle into ``oracle/liboracle.so`` with gcc.

TEST INFRASTRUCTURE: the library is loaded only by the tests, the smoke check
and the CPU-baseline leg of the benchmark.
"""

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "svf_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


def build(force: bool = True, sanitize: bool = False) -> str:
    out = LIB if not sanitize else os.path.join(HERE, "liboracle_asan.so")
    if not force and os.path.exists(out) and os.path.getmtime(out) >= os.path.getmtime(SRC):
        return out
    cmd = ["gcc", "-O2", "-std=c99", "-Wall", "-Wextra", "-fPIC", "-shared", "-pthread",
           SRC, "-o", out + ".tmp"]
    if sanitize:
        cmd[1:1] = ["-g", "-fsanitize=address,undefined", "-fno-omit-frame-pointer"]
    subprocess.check_call(cmd)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(force=True, sanitize="--asan" in sys.argv))
