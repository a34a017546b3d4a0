#!/bin/bash
# Builds tests/sanitize/abi_validation.cpp against the library's sources with AddressSanitizer
# and UndefinedBehaviorSanitizer on the host code (-Xarch_host: the device code is built plainly;
# the validation-only context it exercises launches no kernels).
#   tests/sanitize/build.sh <output binary>
set -euo pipefail
HERE="$(cd "$(dirname "$0")" && pwd)"
ROOT="$(cd "$HERE/../.." && pwd)"
SRC="$ROOT/paper_2606_09377_amd/csrc"
OUT="$1"
HIPCC="${HIPCC:-/opt/rocm/bin/hipcc}"
SAN=(-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined -Xarch_host -fno-sanitize-recover=all
     -Xarch_host -fno-omit-frame-pointer)
OBJS=()
TMP="$(mktemp -d)"
trap 'rm -rf "$TMP"' EXIT
for f in gemm.hip elementwise.hip conv.hip alpha.hip noalloc.hip; do
  "$HIPCC" -O1 -g -std=c++17 -fPIC --offload-arch=gfx950 "${SAN[@]}" -I "$ROOT/include" \
    -x hip -c "$SRC/$f" -o "$TMP/${f%.hip}.o" &
  OBJS+=("$TMP/${f%.hip}.o")
done
for f in api.cpp graph.cpp; do
  "$HIPCC" -O1 -g -std=c++17 -fPIC "${SAN[@]}" -I "$ROOT/include" -c "$SRC/$f" -o "$TMP/${f%.cpp}.o" &
  OBJS+=("$TMP/${f%.cpp}.o")
done
"$HIPCC" -O1 -g -std=c++17 "${SAN[@]}" -I "$ROOT/include" -c "$HERE/abi_validation.cpp" -o "$TMP/driver.o" &
wait
"$HIPCC" "${SAN[@]}" --offload-arch=gfx950 "${OBJS[@]}" "$TMP/driver.o" -o "$OUT"
