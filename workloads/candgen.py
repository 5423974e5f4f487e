"""Python side of the seeded candidate generator (see candgen.c).

Shared input code for the oracle and the GPU evaluator: it draws route
choices and priorities and holds none of the evaluation's arithmetic.
"""
import ctypes as ct
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "candgen.c")
LIB = os.path.join(HERE, "libcandgen.so")

_lib = None


def build_candgen(verbose=False):
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-O3", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared", SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def build_candgen_sanitized(out_dir, verbose=False):
    """The generator under AddressSanitizer and UndefinedBehaviorSanitizer."""
    os.makedirs(out_dir, exist_ok=True)
    out = os.path.join(out_dir, "libcandgen_san.so")
    cmd = ["/opt/rocm/llvm/bin/clang", "-O1", "-g", "-std=c11", "-Wall", "-Wextra", "-fPIC",
           "-shared", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
           "-fno-sanitize-recover=all", "-shared-libsan", SRC, "-o", out]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return out


def _load():
    global _lib
    if _lib is None:
        path = os.environ.get("TACCL_CANDGEN_LIB", LIB)
        if path == LIB and not os.path.exists(LIB):
            build_candgen()
        lib = ct.CDLL(path)
        lib.candgen_fill.restype = ct.c_int
        lib.candgen_fill.argtypes = [ct.c_uint64, ct.c_int64, ct.c_int64, ct.c_int, ct.c_void_p,
                                     ct.c_int, ct.c_void_p, ct.c_void_p]
        _lib = lib
    return _lib


def generate(seed, first, count, options, prio_stride):
    """Candidates first .. first+count-1.

    options[e] = number of route choices of route entry e (0 = unused entry).
    Returns (routes[count][len(options)] u8, prio[count][prio_stride] u32).
    """
    options = np.ascontiguousarray(options, dtype=np.int32)
    rs = len(options)
    routes = np.empty((count, rs), dtype=np.uint8)
    prio = np.empty((count, prio_stride), dtype=np.uint32)
    rc = _load().candgen_fill(int(seed), int(first), int(count), rs,
                              options.ctypes.data_as(ct.c_void_p), int(prio_stride),
                              routes.ctypes.data_as(ct.c_void_p),
                              prio.ctypes.data_as(ct.c_void_p))
    if rc != 0:
        raise ValueError("candgen_fill rejected its arguments")
    return routes, prio
