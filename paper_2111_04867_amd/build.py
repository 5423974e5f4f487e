"""Build the evaluator library (HIP for gfx950) into paper_2111_04867_amd/libtaccl.so."""
import glob
import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libtaccl.so")
ARCH = "gfx950"


def hip_flags():
    """Flags of every HIP compile, the library's objects and the device
    assembly alike. hipcc compiles every source as HIP; packed fp32 ops are
    kept out of device code (the host pass warns that it does not know the
    feature)."""
    return ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall",
            "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def device_asm(src, out):
    """Start compiling one source's device code to gfx950 assembly, as the
    library compiles it; returns the process (stderr piped)."""
    return subprocess.Popen(["hipcc"] + hip_flags() + ["--cuda-device-only", "-S", src, "-o", out],
                            stderr=subprocess.PIPE, text=True)


def build_library(verbose=False, jobs=8, only_changed=False, sanitize=False):
    """Compile every source (only_changed: skip sources whose object is newer
    than the source and every header, for quick rebuilds while editing).
    sanitize: host code under AddressSanitizer and UndefinedBehaviorSanitizer
    (device code unchanged), into _build/san/libtaccl_san.so; the process
    that loads it must preload clang's ASan runtime (tests/sanitize.py)."""
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.cpp")) + glob.glob(os.path.join(CSRC, "*.hip")))
    headers = glob.glob(os.path.join(CSRC, "*.h")) + glob.glob(os.path.join(ROOT, "include", "*.h"))
    newest_header = max(os.path.getmtime(h) for h in headers)
    objdir = os.path.join(PKG, "_build", "san") if sanitize else os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    # host-only sanitizers: each -fsanitize= goes to the host pass alone
    san = (["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]
           if sanitize else [])
    procs, objs = [], []
    for s in srcs:
        o = os.path.join(objdir, os.path.basename(s) + ".o")
        objs.append(o)
        if only_changed and os.path.exists(o) and \
                os.path.getmtime(o) > max(os.path.getmtime(s), newest_header):
            continue
        cmd = ["hipcc"] + hip_flags() + san + ["-c", s, "-o", o]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append(subprocess.Popen(cmd, stderr=subprocess.PIPE, text=True))
        if len([p for p in procs if p.poll() is None]) >= jobs:
            procs[0].wait()
    # the seeded input generator (plain C, shared with the tests)
    gen_o = os.path.join(objdir, "candgen.c.o")
    objs.append(gen_o)
    cc = (["/opt/rocm/llvm/bin/clang", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
           "-fno-sanitize-recover=all"] if sanitize else ["gcc"])
    procs.append(subprocess.Popen(cc + ["-O3", "-std=c11", "-Wall", "-fPIC", "-fvisibility=hidden",
                                        "-c", os.path.join(ROOT, "workloads", "candgen.c"),
                                        "-o", gen_o],
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
    out = os.path.join(objdir, "libtaccl_san.so") if sanitize else LIB
    tmp = out + ".tmp"
    link_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-shared-libsan"] if sanitize else []
    cmd = ["hipcc", "--offload-arch=" + ARCH, "-shared", "-fPIC"] + link_san + objs + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build_library(verbose=True))
