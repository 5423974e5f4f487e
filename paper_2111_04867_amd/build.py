"""Build the evaluator library (HIP for gfx950) into paper_2111_04867_amd/libtaccl.so."""
import glob
import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libtaccl.so")
ARCH = "gfx950"


def build_library(verbose=False, jobs=8):
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.cpp")) + glob.glob(os.path.join(CSRC, "*.hip")))
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    common = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-I" + os.path.join(ROOT, "include"),
              "-I" + CSRC]
    procs, objs = [], []
    for s in srcs:
        o = os.path.join(objdir, os.path.basename(s) + ".o")
        objs.append(o)
        # hipcc compiles every source as HIP; keep packed fp32 ops out of
        # device code (the host pass warns that it does not know the feature)
        cmd = ["hipcc", "--offload-arch=" + ARCH] + common
        cmd += ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
        cmd += ["-c", s, "-o", o]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append(subprocess.Popen(cmd, stderr=subprocess.PIPE, text=True))
        if len([p for p in procs if p.poll() is None]) >= jobs:
            procs[0].wait()
    # the seeded input generator (plain C, shared with the tests)
    gen_o = os.path.join(objdir, "candgen.c.o")
    objs.append(gen_o)
    procs.append(subprocess.Popen(["gcc", "-O3", "-std=c11", "-Wall", "-fPIC", "-fvisibility=hidden",
                                   "-c", os.path.join(ROOT, "workloads", "candgen.c"), "-o", gen_o],
                                  stderr=subprocess.PIPE, text=True))
    failed = False
    for p in procs:
        err = p.communicate()[1]
        # drop the host pass's note about the device-only feature flag
        lines = [ln for ln in err.splitlines() if "packed-fp32-ops" not in ln]
        if lines:
            print("\n".join(lines), flush=True)
        failed |= p.returncode != 0
    if failed:
        raise RuntimeError("hipcc failed")
    tmp = LIB + ".tmp"
    cmd = ["hipcc", "--offload-arch=" + ARCH, "-shared", "-fPIC"] + objs + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build_library(verbose=True))
