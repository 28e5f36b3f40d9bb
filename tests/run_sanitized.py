"""Run the CPU test suite against sanitizer builds of the oracle and of the
library's host code (AddressSanitizer + UndefinedBehaviorSanitizer, clang's
shared runtime preloaded into the Python process).

    python tests/run_sanitized.py [extra pytest arguments]

Builds oracle/liboracle_san.so and paper_2504_11320_amd/libwait_sim_san.so,
then runs `pytest tests -m "not gpu"` with WAIT_ORACLE_LIB / WAIT_SIM_LIB
pointing at them.  Leak detection is off (the interpreter's own allocations
are not freed at exit); any report fails the run.  The ABI test of an
impossible host allocation is skipped (the sanitizer's allocator answers it).
"""
import glob
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def main() -> int:
    from oracle import oracle as O
    from paper_2504_11320_amd import build as Bd
    orc = os.path.join(ROOT, "oracle", "liboracle_san.so")
    lib = os.path.join(ROOT, "paper_2504_11320_amd", "libwait_sim_san.so")
    O.build_sanitized(orc)
    Bd.build(out=lib, sanitize=True)
    rt = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not rt:
        print("run_sanitized: clang ASan runtime not found", file=sys.stderr)
        return 2
    env = dict(os.environ)
    env.update(LD_PRELOAD=rt[-1], WAIT_ORACLE_LIB=orc, WAIT_SIM_LIB=lib, WAIT_SIM_SANITIZED="1",
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1:log_path=/tmp/wait_sim_asan",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1:log_path=/tmp/wait_sim_ubsan")
    cmd = [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests"), "-q", "-m", "not gpu",
           "-p", "no:cacheprovider"] + sys.argv[1:]
    for f in glob.glob("/tmp/wait_sim_asan*") + glob.glob("/tmp/wait_sim_ubsan*"):
        os.remove(f)
    rc = subprocess.run(cmd, env=env, cwd=ROOT).returncode
    reports = glob.glob("/tmp/wait_sim_asan*") + glob.glob("/tmp/wait_sim_ubsan*")
    for f in reports:  # a sanitizer report names the failing access
        print(f"---- {f}"); print(open(f).read()[:4000])
    return rc if rc != 0 else (1 if reports else 0)


if __name__ == "__main__":
    sys.exit(main())
