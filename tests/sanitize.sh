#!/bin/bash
# CPU test suite with the oracle and the input generator's host code under AddressSanitizer and
# UndefinedBehaviorSanitizer: builds liboracle_san.so and libsynth_san.so beside the normal
# libraries, then runs the tests that need no GPU with the sanitizer runtime preloaded.
#   bash tests/sanitize.sh [extra pytest arguments]
set -e
cd "$(dirname "$0")/.."
python oracle/build.py --sanitize > /dev/null
python synth/build.py --sanitize > /dev/null
RT=$(/opt/rocm/lib/llvm/bin/clang++ -print-file-name=libclang_rt.asan-x86_64.so)
MPC_SANITIZE=1 LD_PRELOAD="$RT" ASAN_OPTIONS=detect_leaks=0:halt_on_error=1 UBSAN_OPTIONS=print_stacktrace=1 \
  python -m pytest tests -q -m "not gpu" "$@"
