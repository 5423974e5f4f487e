"""Host sanitizer leg (CPU only): build the plan builder, the C ABI layer and
the seeded generator (the library's host code) and the C oracle under
AddressSanitizer + UndefinedBehaviorSanitizer, then run the whole CPU test
suite against those builds.

    python tests/sanitize.py [extra pytest args]

Device code is compiled as usual (only the host pass is instrumented); no
test of the CPU suite launches a kernel. The sanitizer runtime is clang's
and is preloaded into the test process, since the Python interpreter itself
is not instrumented. Leak checking is off (the interpreter keeps its own
allocations to the end); every other report aborts the run.
"""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def main():
    from oracle.build import build_oracle_sanitized
    from paper_2111_04867_amd.build import build_library
    from workloads.candgen import build_candgen_sanitized

    out = os.path.join(ROOT, "paper_2111_04867_amd", "_build", "san")
    lib = build_library(sanitize=True, only_changed=True)
    orc = build_oracle_sanitized(out)
    gen = build_candgen_sanitized(out)
    rt = subprocess.run(["/opt/rocm/llvm/bin/clang", "-print-file-name=libclang_rt.asan-x86_64.so"],
                        check=True, capture_output=True, text=True).stdout.strip()
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": rt,
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1:halt_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        "TACCL_LIB": lib, "TACCL_ORACLE_LIB": orc, "TACCL_CANDGEN_LIB": gen,
    })
    cmd = [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests"), "-x", "-q", "-m",
           "not gpu", "-p", "no:cacheprovider"] + sys.argv[1:]
    print("sanitized run:", " ".join(cmd), flush=True)
    return subprocess.run(cmd, env=env, cwd=ROOT).returncode


if __name__ == "__main__":
    sys.exit(main())
