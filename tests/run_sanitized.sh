#!/bin/bash
# The CPU test suite against sanitizer builds: the oracle and the library's
# host code (argument validation, workspace carving, launch set-up) built
# with AddressSanitizer and UndefinedBehaviorSanitizer.  Device code is not
# instrumented.  Usage, from the repository root: bash tests/run_sanitized.sh
set -euo pipefail
cd "$(dirname "$0")/.."
python3 -c "from paper_2608_12780_amd import build; print(build.build(sanitize=True))"
python3 -c "import oracle; print(oracle.build(sanitize=True))"
ASAN_RT=$(gcc -print-file-name=libasan.so)
UBSAN_RT=$(gcc -print-file-name=libubsan.so)
# python itself is not instrumented: preload the runtimes; leak reports from
# the interpreter's own allocations are not this code's
export LD_PRELOAD="$ASAN_RT $UBSAN_RT"
export ASAN_OPTIONS=detect_leaks=0:abort_on_error=1:halt_on_error=1
export UBSAN_OPTIONS=print_stacktrace=1:halt_on_error=1
export SCOPE_LIBRARY=$PWD/paper_2608_12780_amd/libscope_san.so
export SCOPE_ORACLE_LIBRARY=$PWD/oracle/libscope_oracle_san.so
python3 -m pytest tests -q -m "not gpu" -p no:cacheprovider "$@"
