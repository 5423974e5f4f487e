"""Compile the CPU oracle (plain C, gcc) into oracle/liboracle.so.

Test infrastructure only: building the checker is not using it.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "taccl_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


def build_oracle(verbose=False):
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared", SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def build_oracle_sanitized(out_dir, verbose=False):
    """The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (clang,
    so that one runtime serves every sanitized library of the process)."""
    os.makedirs(out_dir, exist_ok=True)
    out = os.path.join(out_dir, "liboracle_san.so")
    cmd = ["/opt/rocm/llvm/bin/clang", "-O1", "-g", "-std=c11", "-Wall", "-Wextra", "-fPIC",
           "-shared", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
           "-fno-sanitize-recover=all", "-shared-libsan", SRC, "-o", out]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return out


if __name__ == "__main__":
    print(build_oracle(verbose=True))
