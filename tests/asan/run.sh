#!/bin/bash
# Host sanitizer builds (CPU only): the fp64 oracle and the C ABI layer, each built
# with -fsanitize=address,undefined by gcc / g++ and run by a small driver.  The
# library's HIP objects are linked unchanged (their host parts are not instrumented);
# nothing here runs on a GPU.  Usage: tests/asan/run.sh [build dir]
set -euo pipefail
ROOT="$(cd "$(dirname "$0")/../.." && pwd)"
OUT="${1:-$ROOT/tests/asan/_build}"
mkdir -p "$OUT"
SAN="-fsanitize=address,undefined -fno-sanitize-recover=all -fno-omit-frame-pointer -g -O1"
export ASAN_OPTIONS="detect_leaks=1:abort_on_error=1"
export UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1"

gcc -std=c11 $SAN -pthread -ffp-contract=off "$ROOT/oracle/kla_oracle.c" "$ROOT/tests/asan/oracle_driver.c" \
    -lm -o "$OUT/oracle_driver"
"$OUT/oracle_driver"

# the library's other objects, as the last build left them (paper_2602_10743_amd/build.py)
BLD="$ROOT/paper_2602_10743_amd/_build"
OBJS=""
for src in $(python3 -c "import sys; sys.path.insert(0, '$ROOT/paper_2602_10743_amd'); import build; print(' '.join(build.SOURCES))"); do
    o="$BLD/${src%.*}.o"
    [ -f "$o" ] || { echo "missing $o: build the library first" >&2; exit 1; }
    [ "$src" = kla_api.cpp ] || OBJS="$OBJS $o"
done
g++ -std=c++17 $SAN -D__HIP_PLATFORM_AMD__ -I/opt/rocm/include -I"$ROOT/include" \
    -I"$ROOT/paper_2602_10743_amd/csrc" -c "$ROOT/paper_2602_10743_amd/csrc/kla_api.cpp" -o "$OUT/kla_api.o"
# the HIP runtime keeps allocations of its own until exit: leak reports are for the ABI layer only
ASAN_OPTIONS="detect_leaks=0:abort_on_error=1"
g++ -std=c++17 $SAN -I"$ROOT/include" -D__HIP_PLATFORM_AMD__ -I/opt/rocm/include \
    "$ROOT/tests/asan/abi_driver.cpp" "$OUT/kla_api.o" $OBJS -L/opt/rocm/lib -lamdhip64 \
    -Wl,-rpath,/opt/rocm/lib -o "$OUT/abi_driver"
ASAN_OPTIONS="$ASAN_OPTIONS" "$OUT/abi_driver"
