#!/bin/bash
# AddressSanitizer + UndefinedBehaviorSanitizer run of the host code, on the
# CPU (no GPU needed or used): the oracle, the placement generator and the
# library's host side (loader, boundary checks, scheduler) are rebuilt with
# both sanitizers, one runtime for all three (clang's), and the CPU test
# suite runs against those builds.  Device code is built as usual: the
# sanitizer flags apply to the host side only.
#
#   bash tests/sanitizers/run.sh [build dir]     (default /tmp/ss_sanitize)
set -euo pipefail
ROOT="$(cd "$(dirname "$0")/../.." && pwd)"
OUT="${1:-/tmp/ss_sanitize}"
LLVM=/opt/rocm/llvm/bin
mkdir -p "$OUT"
SAN_C="-fsanitize=address,undefined -fno-sanitize-recover=undefined -fno-omit-frame-pointer -g -O1"
echo "[sanitize] oracle and placement generator (clang)"
$LLVM/clang $SAN_C -std=c11 -fPIC -shared "$ROOT/oracle/ss_oracle.c" -o "$OUT/liboracle.so"
$LLVM/clang $SAN_C -std=c11 -fPIC -shared -pthread "$ROOT/paper_2608_15762_amd/synth/placements.c" -o "$OUT/libsynth.so"
echo "[sanitize] library, host side (hipcc)"
CSRC="$ROOT/paper_2608_15762_amd/csrc"
HOSTSAN="-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined -Xarch_host -fno-sanitize-recover=undefined -Xarch_host -fno-omit-frame-pointer"
OBJS=()
for src in abi.cpp gmg_load.cpp sched.cpp simulate.hip sim_fast.hip select.hip estimator.hip noalloc.hip; do
  lang=(); case "$src" in *.hip) lang=(-x hip);; esac
  /opt/rocm/bin/hipcc -O1 -g -std=c++17 -fPIC --offload-arch=gfx950 -Xclang -target-feature -Xclang -packed-fp32-ops \
    $HOSTSAN -I "$ROOT/include" -I "$CSRC" "${lang[@]}" -c "$CSRC/$src" -o "$OUT/$src.o"
  OBJS+=("$OUT/$src.o")
done
/opt/rocm/bin/hipcc -shared -fPIC --offload-arch=gfx950 $HOSTSAN -shared-libsan "${OBJS[@]}" -o "$OUT/libss.so"
RT="$($LLVM/clang -print-file-name=libclang_rt.asan-x86_64.so)"
[ -f "$RT" ] || RT="$(ls /opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so | head -1)"
echo "[sanitize] CPU suite against the sanitized builds (runtime $RT)"
cd "$ROOT"
# leaks are not checked: the Python interpreter itself holds memory until exit
LD_PRELOAD="$RT" ASAN_OPTIONS=detect_leaks=0:abort_on_error=1 UBSAN_OPTIONS=print_stacktrace=1:halt_on_error=1 \
  SS_ORACLE_LIB="$OUT/liboracle.so" SS_SYNTH_LIB="$OUT/libsynth.so" SS_LIBRARY="$OUT/libss.so" \
  python3 -m pytest tests/ -x -q -m "not gpu" -p no:cacheprovider
