#!/bin/bash
# CPU-only sanitizer run (no GPU needed), from the repository root: bash tests/sanitize_cpu.sh
#  1. the fp64 oracle built with gcc's AddressSanitizer and UndefinedBehaviorSanitizer, checked
#     against its pins (tests/test_oracle.py);
#  2. the library with its host code (argument validation, workspace planning, the checks of
#     the allocation-free entry point) built with clang's AddressSanitizer and
#     UndefinedBehaviorSanitizer for the host pass only (device code as usual), exercised by
#     tests/test_abi.py, whose calls all return before any work is enqueued.
# Each part runs in a process of its own with its compiler's sanitizer runtime preloaded.
set -euo pipefail
ROOT=$(cd "$(dirname "$0")/.." && pwd)
OUT=${SAN_OUT:-/tmp/lapattn_san}
mkdir -p "$OUT"
cd "$ROOT"

echo "== oracle (gcc -fsanitize=address,undefined)"
gcc -O1 -g -fno-omit-frame-pointer -fsanitize=address,undefined -fno-sanitize-recover=undefined \
    -ffp-contract=off -fno-fast-math -fopenmp -fPIC -shared -std=c11 -Wall -Wextra \
    -o "$OUT/liblapattn_oracle.so" oracle/lapattn_oracle.c -lm
LAPATTN_ORACLE_LIB="$OUT/liblapattn_oracle.so" \
LD_PRELOAD="$(gcc -print-file-name=libasan.so):$(gcc -print-file-name=libubsan.so)" \
ASAN_OPTIONS=detect_leaks=0 UBSAN_OPTIONS=halt_on_error=1:print_stacktrace=1 \
    python -m pytest tests/test_oracle.py -q -m "not gpu" -p no:cacheprovider

echo "== library host code (hipcc, host pass -fsanitize=address,undefined)"
HIPCC=${HIPCC:-/opt/rocm/bin/hipcc}
DEV="-Xclang -target-feature -Xclang -packed-fp32-ops"
objs=()
for src in fwd.hip fast.hip nsbig.hip bwd.hip dwc.hip; do
    "$HIPCC" --offload-arch=gfx950 -O3 -std=c++17 -fPIC -I include -c "paper_2604_20368_amd/csrc/$src" \
        -o "$OUT/${src%.*}.o" $DEV 2>/dev/null
    objs+=("$OUT/${src%.*}.o")
done
for src in noalloc.hip host.cpp; do
    "$HIPCC" --offload-arch=gfx950 -O1 -g -std=c++17 -fPIC -I include -fno-omit-frame-pointer \
        -Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined \
        -c "paper_2604_20368_amd/csrc/$src" -o "$OUT/${src%.*}.o" $DEV 2>/dev/null
    objs+=("$OUT/${src%.*}.o")
done
"$HIPCC" --offload-arch=gfx950 -shared -fPIC -Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined \
    -shared-libsan -o "$OUT/liblapattn.so" "${objs[@]}"
RT=$(ls /opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so | head -1)
LAPATTN_LIB="$OUT/liblapattn.so" LD_PRELOAD="$RT" ASAN_OPTIONS=detect_leaks=0 \
UBSAN_OPTIONS=halt_on_error=1:print_stacktrace=1 \
    python -m pytest tests/test_abi.py -q -m "not gpu" -p no:cacheprovider
echo "== sanitizer run clean"
