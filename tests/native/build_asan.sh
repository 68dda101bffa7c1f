#!/bin/bash
# Builds tests/native/abi_asan_driver: the library's sources and the driver
# with AddressSanitizer and UndefinedBehaviorSanitizer on the host code only (each -fsanitize follows
# -Xarch_host; the GPU code is not instrumented).  Run the result on a GPU with
# ASAN_OPTIONS=detect_leaks=0:quarantine_size_mb=4096: the HIP runtime keeps
# allocations until exit, and a quarantine larger than all the device memory
# the driver frees (about 2 GB) keeps ASan from recycling freed device chunks
# while the runtime unloads at exit, which fails one of ASan's own checks.
set -e
HERE=$(cd "$(dirname "$0")" && pwd)
ROOT=$(cd "$HERE/../.." && pwd)
SRC=$ROOT/paper_2007_06134_amd/csrc
OUT=${1:-$HERE/_build}
mkdir -p "$OUT"
INC="-I$ROOT/include -I$SRC"
FL="-O1 -g -std=c++17 -fno-omit-frame-pointer -Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined"
HIPCC=${HIPCC:-/opt/rocm/bin/hipcc}
$HIPCC $FL $INC --offload-arch=gfx950 -ffp-contract=off -Xclang -target-feature -Xclang -packed-fp32-ops -x hip -c "$SRC/kernels.hip" -o "$OUT/kernels.o"
$HIPCC $FL $INC --offload-arch=gfx950 -ffp-contract=off -Xclang -target-feature -Xclang -packed-fp32-ops -x hip -c "$SRC/noalloc.hip" -o "$OUT/noalloc.o"
$HIPCC $FL $INC -D__HIP_PLATFORM_AMD__ -ffp-contract=off -c "$SRC/runtime.cpp" -o "$OUT/runtime.o"
$HIPCC $FL $INC -D__HIP_PLATFORM_AMD__ -ffp-contract=off -c "$SRC/controller.cpp" -o "$OUT/controller.o"
$HIPCC $FL $INC -D__HIP_PLATFORM_AMD__ -c "$HERE/abi_asan_driver.cpp" -o "$OUT/driver.o"
$HIPCC -Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined --offload-arch=gfx950 "$OUT"/kernels.o "$OUT"/noalloc.o "$OUT"/runtime.o "$OUT"/controller.o "$OUT"/driver.o -L/opt/rocm/lib -lrocprofiler-sdk-roctx -Wl,-rpath,/opt/rocm/lib -o "$OUT/abi_asan_driver"
echo "$OUT/abi_asan_driver"
