#!/bin/bash
# The CPU test suite (pytest -m "not gpu") under AddressSanitizer and
# UndefinedBehaviorSanitizer, on the CPU only: the oracle (strata_oracle.c) and
# the host code of every HIP source (argument validation, kernel selection and
# the launchers of libstrata) are rebuilt with the sanitizers into a scratch
# directory and loaded instead of the regular builds; device code is built as
# usual.  Usage: bash tests/run_host_sanitizers.sh [scratch dir]
set -euo pipefail
ROOT=$(cd "$(dirname "$0")/.." && pwd)
OUT=${1:-$(mktemp -d /tmp/strata_san.XXXXXX)}
mkdir -p "$OUT"
LLVM=/opt/rocm/llvm
RT=$(ls "$LLVM"/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so | head -1)
SAN="-fsanitize=address,undefined -fno-sanitize-recover=undefined -fno-omit-frame-pointer"

# the oracle, with clang (one sanitizer runtime in the process)
"$LLVM"/bin/clang -O1 -g -std=c11 -fopenmp -ffp-contract=off -fno-fast-math $SAN -fPIC -shared \
  "$ROOT"/oracle/strata_oracle.c -o "$OUT"/liboracle_san.so -lm

# libstrata: the host pass of every source with the sanitizers, the device pass unchanged
objs=()
for src in "$ROOT"/paper_2606_31248_amd/csrc/*.hip; do
  o="$OUT"/$(basename "${src%.hip}").o
  /opt/rocm/bin/hipcc --offload-arch=gfx950 -O1 -g -std=c++17 -fPIC \
    -Xclang -target-feature -Xclang -packed-fp32-ops \
    -Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined -Xarch_host -fno-omit-frame-pointer \
    -I "$ROOT"/include -I "$ROOT"/paper_2606_31248_amd/csrc -c "$src" -o "$o" 2> "$o.log" &
  objs+=("$o")
done
wait
/opt/rocm/bin/hipcc --offload-arch=gfx950 -shared -fPIC -o "$OUT"/libstrata_san.so "${objs[@]}"

cd "$ROOT"
LD_PRELOAD="$RT" ASAN_OPTIONS=detect_leaks=0:protect_shadow_gap=0 UBSAN_OPTIONS=print_stacktrace=1 \
  STRATA_ORACLE_LIB="$OUT"/liboracle_san.so STRATA_LIB="$OUT"/libstrata_san.so \
  python -m pytest tests -m "not gpu" -x -q -p no:cacheprovider
