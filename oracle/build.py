"""Builds the CPU oracle (``libltdoracle.so``) with gcc.

Test infrastructure: the oracle library is loaded only by the test suite, the
smoke check and the benchmark's CPU-baseline leg.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libltdoracle.so")
# AddressSanitizer + UndefinedBehaviorSanitizer build of the same source, for
# the host sanitizer run of the oracle's tests (loaded in place of LIB when
# LTD_ORACLE_LIB names it; the process must preload the ASan runtime).
SAN_LIB = os.path.join(HERE, "libltdoracle_san.so")
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
             "-fno-omit-frame-pointer", "-g"]


def build(verbose: bool = False, sanitize: bool = False) -> str:
    src = os.path.join(HERE, "ltd_oracle.c")
    out = SAN_LIB if sanitize else LIB
    cmd = ["gcc", "-O1" if sanitize else "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
           "-Wall", "-Wextra", *(SAN_FLAGS if sanitize else []), "-o", out + ".tmp", src, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
