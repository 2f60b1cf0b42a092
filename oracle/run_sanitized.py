"""Run the CPU test suite against an AddressSanitizer + UndefinedBehaviorSanitizer
build of the oracle.

    python oracle/run_sanitized.py [test paths] [extra pytest arguments]

Builds ``libsom_oracle_san.so`` (gcc, -fsanitize=address,undefined,
-fno-sanitize-recover=all), checks that it really carries the instrumentation,
and runs ``pytest tests -m "not gpu"`` in a child process that preloads gcc's
libasan (the Python interpreter itself is not instrumented) and selects that
build with SOM_ORACLE_SANITIZE=1.  Any heap/stack overflow, use after free or
undefined behaviour inside the oracle aborts the child, so the exit status is
pytest's only when the oracle ran clean.  Leak checking is off: the interpreter
keeps its own allocations until exit by design.

Test infrastructure, like the rest of this directory.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def main(argv) -> int:
    env = dict(os.environ)
    env["SOM_ORACLE_SANITIZE"] = "1"
    # build in a child so this process never loads the instrumented library
    subprocess.run([sys.executable, "-c",
                    "import oracle; print('sanitized oracle:', oracle.build(force=True))"],
                   cwd=ROOT, env=env, check=True)
    lib = os.path.join(HERE, "libsom_oracle_san.so")
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True, check=True).stdout
    if "__asan_" not in syms or "__ubsan_" not in syms:
        print("sanitized oracle lacks ASan/UBSan instrumentation", file=sys.stderr)
        return 2
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True, check=True).stdout.strip()
    pre = env.get("LD_PRELOAD", "")
    env["LD_PRELOAD"] = asan + (":" + pre if pre else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1:strict_string_checks=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    # (the test that runs this script is left out of a whole-suite run)
    paths = [a for a in argv if a.startswith("tests")] or [
        "tests", "--ignore=tests/test_sanitized_oracle.py"]
    rest = [a for a in argv if not a.startswith("tests")]
    cmd = [sys.executable, "-m", "pytest", *paths, "-m", "not gpu", "-q",
           "-p", "no:cacheprovider", *rest]
    sys.stdout.flush()
    return subprocess.run(cmd, cwd=ROOT, env=env).returncode


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
