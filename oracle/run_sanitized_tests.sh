#!/bin/sh
# Runs the CPU test suite (pytest -m "not gpu") against the oracle built by
# gcc with AddressSanitizer and UndefinedBehaviorSanitizer, every report
# fatal. The interpreter itself is not instrumented, so the sanitizer
# runtimes are preloaded into it; leak reports are off (the interpreter's own
# allocations at exit are not the oracle's). Extra arguments go to pytest.
set -e
cd "$(dirname "$0")/.."
export NOPFS_ORACLE_SANITIZE=1
export ASAN_OPTIONS=detect_leaks=0:abort_on_error=1:allocator_may_return_null=1
export UBSAN_OPTIONS=print_stacktrace=1:halt_on_error=1
python -c "from oracle import ref; ref.build(force=True)"
LD_PRELOAD="$(gcc -print-file-name=libasan.so):$(gcc -print-file-name=libubsan.so)" \
  python -m pytest tests -m "not gpu" -q -p no:cacheprovider "$@"
