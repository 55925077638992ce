"""Runs the CPU test suite against host code built under AddressSanitizer and
UndefinedBehaviorSanitizer (test infrastructure; no GPU needed):

    python tests/sanitize_host.py [extra pytest arguments]

Builds the library's host-only sources (planner, invoker, normalisation constants) and the
C oracle with -fsanitize=address,undefined (undefined behaviour aborts), then runs
`pytest -m "not gpu"` in a child process with GCC's ASan runtime preloaded (Python itself
is not instrumented; leak checking is off because the interpreter keeps its own
allocations until exit). Exits with pytest's status.
"""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def main() -> int:
    from paper_2404_09267_amd import build as B

    import oracle

    lib = B.build(sanitize=True)
    orc = oracle.build(force=True, path=os.path.join(B.BUILD, "sanitize", "liboracle.so"),
                       sanitize=True)
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], check=True,
                          capture_output=True, text=True).stdout.strip()
    env = dict(os.environ)
    env.update({"TG_LIBTG": lib, "TG_LIBORACLE": orc, "LD_PRELOAD": asan,
                "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
                "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1"})
    cmd = [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests"), "-q", "-m", "not gpu",
           "-p", "no:cacheprovider", *sys.argv[1:]]
    print("+", " ".join(cmd), flush=True)
    return subprocess.run(cmd, env=env, cwd=ROOT).returncode


if __name__ == "__main__":
    sys.exit(main())
