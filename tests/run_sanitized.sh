#!/bin/bash
# The CPU test suite (-m "not gpu") with the oracle and the library's host
# code built with AddressSanitizer and UndefinedBehaviorSanitizer (clang; the
# device code is not instrumented).  Python itself is not instrumented: the
# sanitizer runtime is preloaded and leak detection is off (the interpreter
# keeps memory until exit).  Any report aborts the run; the reports are
# printed at the end and the exit status is pytest's.
set -uo pipefail
cd "$(dirname "$0")/.."
python -m paper_1607_00145_amd.build --sanitize --incremental > /dev/null || exit 1
python -c "import oracle; oracle.build(force=True, sanitize=True)" || exit 1
RT=$(/opt/rocm/llvm/bin/clang -print-file-name=libclang_rt.asan-x86_64.so)
REPORTS=$(mktemp -d)
export LD_PRELOAD="$RT"
export ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1:log_path=$REPORTS/asan"
export UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1:log_path=$REPORTS/ubsan"
export GETT_LIBRARY="$PWD/paper_1607_00145_amd/lib/libgett_asan.so"
export ORACLE_LIBRARY="$PWD/oracle/liboracle_asan.so"
python -m pytest tests -m "not gpu" -q -p no:cacheprovider "$@"
rc=$?
unset LD_PRELOAD
for f in "$REPORTS"/*; do
    [ -e "$f" ] || continue
    echo "=== sanitizer report $f"
    grep -v "in _Py\|python3.10+\|libffi\|_ctypes" "$f" | head -40
    [ "$rc" -eq 0 ] && rc=1
done
rm -rf "$REPORTS"
exit $rc
