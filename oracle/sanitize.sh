#!/bin/bash
# Builds the oracle with AddressSanitizer and UndefinedBehaviorSanitizer
# (gcc, host code only) and runs the CPU test tier against that build: every
# oracle function the pins exercise, with out-of-bounds accesses, use after
# free and undefined behaviour made fatal. Leak checking is off: the Python
# interpreter that drives the tests keeps allocations alive at exit.
# Usage: bash oracle/sanitize.sh [extra pytest args]
set -euo pipefail
ROOT=$(cd "$(dirname "$0")/.." && pwd)
OUT=$(mktemp -d "${TMPDIR:-/tmp}/cagq_oracle_san.XXXXXX")
gcc -O1 -g -std=c99 -ffp-contract=off -fno-fast-math -fPIC -shared -fno-omit-frame-pointer \
    -fsanitize=address,undefined -fno-sanitize-recover=all \
    "$ROOT/oracle/cagq_oracle.c" -o "$OUT/libcagq_oracle.so" -lm
export CAGQ_ORACLE_LIB="$OUT/libcagq_oracle.so"
export LD_PRELOAD="$(gcc -print-file-name=libasan.so):$(gcc -print-file-name=libubsan.so)"
export ASAN_OPTIONS=detect_leaks=0:abort_on_error=1:halt_on_error=1
export UBSAN_OPTIONS=print_stacktrace=1:halt_on_error=1
cd "$ROOT"
python -m pytest tests -q -m "not gpu" -p no:cacheprovider "$@"
rm -rf "$OUT"
