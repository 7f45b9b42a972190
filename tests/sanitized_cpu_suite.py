"""The CPU test suite under AddressSanitizer and UndefinedBehaviorSanitizer.

Builds the oracle (oracle.c), the input generator (synth.c) and the library's
host code (the device code is unchanged) with LLVM's ASan and UBSan into
separate ``*.san.so`` files (the AGNES_SANITIZE build option), then runs
``pytest -m "not gpu"`` against them in a child process with the sanitizer
runtime preloaded.  Any report ends the run with a failure: the builds stop at
the first UBSan finding and ASan aborts on the first error.  Leak checking is
off because the Python interpreter itself is not built for it.

    python tests/sanitized_cpu_suite.py [extra pytest arguments]

The exit status is pytest's.  Needs no GPU.
"""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
CHECKS = "address,undefined"


def runtime() -> str:
    clang = os.path.join(ROCM, "llvm", "bin", "clang")
    path = subprocess.check_output([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], text=True).strip()
    if not os.path.isfile(path):
        raise SystemExit("sanitizer runtime not found: " + path)
    return path


def main(argv) -> int:
    env = dict(os.environ, AGNES_SANITIZE=CHECKS)
    build = ("import oracle, synth\n"
             "from paper_2601_01473_amd import build\n"
             "print(oracle.build(), synth.build(), build.build(), sep='\\n')\n")
    print("# building with -fsanitize=" + CHECKS, flush=True)
    subprocess.check_call([sys.executable, "-c", build], cwd=ROOT, env=env)
    env["LD_PRELOAD"] = runtime()
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1:detect_odr_violation=0"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    cmd = [sys.executable, "-m", "pytest", "tests", "-x", "-q", "-m", "not gpu", *argv]
    print("# " + " ".join(cmd), flush=True)
    return subprocess.call(cmd, cwd=ROOT, env=env)


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
