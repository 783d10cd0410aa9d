#!/bin/bash
# Build of every library source plus the ABI driver with the host code under
# AddressSanitizer and UndefinedBehaviorSanitizer (each -fsanitize= applies to
# the host pass only; the device code is compiled as usual and never run by
# the driver).  Usage: build.sh <output executable>
set -euo pipefail
HERE="$(cd "$(dirname "$0")" && pwd)"
ROOT="$(cd "$HERE/../.." && pwd)"
OUT="$1"
OBJ="$(mktemp -d)"
trap 'rm -rf "$OBJ"' EXIT
HIPCC="${HIPCC:-/opt/rocm/bin/hipcc}"
SAN=(-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined -Xarch_host -fno-sanitize-recover=undefined)
for src in "$ROOT"/paper_2607_12875_amd/csrc/*.hip; do
  "$HIPCC" --offload-arch=gfx950 -x hip -O1 -g -std=c++17 "${SAN[@]}" \
    -Xclang -target-feature -Xclang -packed-fp32-ops -I "$ROOT/include" \
    -I "$ROOT/paper_2607_12875_amd/csrc" -c "$src" -o "$OBJ/$(basename "$src").o" &
done
"$HIPCC" --offload-arch=gfx950 -x hip -O1 -g -std=c++17 "${SAN[@]}" -I "$ROOT/include" -c "$HERE/abi_driver.cpp" -o "$OBJ/driver.o" &
wait
"$HIPCC" --offload-arch=gfx950 "${SAN[@]}" -o "$OUT" "$OBJ"/*.o
