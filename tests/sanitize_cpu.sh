#!/bin/bash
# CPU sanitizer leg: the oracle and the host code of libspexis (argument validation, workspace
# carving, launch set-up) built with AddressSanitizer and UndefinedBehaviorSanitizer, then the
# CPU test suite (-m "not gpu") run against those builds in a copy of the tree under
# _build/sanitize.  Device code is built as usual; only host code is instrumented.  Needs no GPU.
#
#   bash tests/sanitize_cpu.sh [extra pytest args]
set -euo pipefail
ROOT="$(cd "$(dirname "${BASH_SOURCE[0]}")/.." && pwd)"
OUT="$ROOT/_build/sanitize"
LLVM=/opt/rocm/llvm
RT="$(ls "$LLVM"/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so | head -1)"
rm -rf "$OUT"
mkdir -p "$OUT"
for d in include oracle paper_2609_34370_amd tests; do
  cp -r "$ROOT/$d" "$OUT/$d"
done
cp "$ROOT/pytest.ini" "$ROOT/bench.py" "$OUT/"
find "$OUT" -name "*.so" -delete
find "$OUT" -name "__pycache__" -prune -exec rm -rf {} +
CSRC="$OUT/paper_2609_34370_amd/csrc"
SAN="-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined -Xarch_host -fno-sanitize-recover=undefined -Xarch_host -fno-omit-frame-pointer"
OBJS=()
for src in append attention accept lm_head select lookahead linear pack api; do
  /opt/rocm/bin/hipcc -O1 -g -std=c++17 --offload-arch=gfx950 -fPIC \
    -Xclang -target-feature -Xclang -packed-fp32-ops $SAN \
    -I "$OUT/include" -I "$CSRC" -c "$CSRC/$src.hip" -o "$OUT/$src.o" 2>/dev/null
  OBJS+=("$OUT/$src.o")
done
/opt/rocm/bin/hipcc --offload-arch=gfx950 -shared -fPIC -Xarch_host -fsanitize=address \
  -Xarch_host -fsanitize=undefined "${OBJS[@]}" -o "$OUT/paper_2609_34370_amd/libspexis.so"
"$LLVM/bin/clang" -O1 -g -std=gnu11 -fopenmp -ffp-contract=off -fno-fast-math -fsanitize=address,undefined \
  -fno-sanitize-recover=undefined -fno-omit-frame-pointer -shared -fPIC "$OUT/oracle/spexis_oracle.c" \
  -o "$OUT/oracle/libspexis_oracle.so" -lm -Wl,-rpath,"$LLVM/lib"
cd "$OUT"
LD_PRELOAD="$RT" ASAN_OPTIONS=detect_leaks=0:abort_on_error=1:detect_odr_violation=0 \
  UBSAN_OPTIONS=halt_on_error=1:print_stacktrace=1 \
  python -m pytest -m "not gpu" -x -q -p no:cacheprovider "$@"
