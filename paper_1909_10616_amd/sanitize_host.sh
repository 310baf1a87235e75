#!/bin/bash
# Host-side memory and undefined-behaviour check, CPU only: rebuilds the host
# units of libgemmtune.so (space, search, runtime, lookup) with AddressSanitizer
# and UBSan on the host pass only, links them with the kernel objects of the
# last build, builds the oracle with the same sanitizers (clang, one runtime),
# and runs the CPU test suite against both with the runtime preloaded.
#   paper_1909_10616_amd/sanitize_host.sh [pytest arguments]
set -euo pipefail
R=$(cd "$(dirname "$0")/.." && pwd)
O=$R/_build/asan
mkdir -p "$O"
H=/opt/rocm/bin/hipcc
CXXF="-O1 -g -std=c++17 -fPIC --offload-arch=gfx950 -Xclang -target-feature -Xclang -packed-fp32-ops
      -munsafe-fp-atomics -I $R/include -I $R/paper_1909_10616_amd/csrc"
SAN="-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined -Xarch_host -fno-omit-frame-pointer
     -Xarch_host -fno-sanitize-recover=undefined"
ls "$R"/_build/gemm_*_c*.o > /dev/null   # kernel objects of a normal build
for u in space search runtime gemm_lookup; do
  $H $CXXF $SAN -x hip -c "$R/paper_1909_10616_amd/csrc/$u.cpp" -o "$O/$u.o" &
done
wait
$H --offload-arch=gfx950 -shared -fPIC -Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined \
   -shared-libsan "$O"/space.o "$O"/search.o "$O"/runtime.o "$O"/gemm_lookup.o \
   "$R"/_build/aux_kernels.o "$R"/_build/noalloc.o "$R"/_build/gemm_*_c*.o -o "$O/libgemmtune.so"
/opt/rocm/llvm/bin/clang -O1 -g -std=c11 -fPIC -shared -fsanitize=address,undefined \
   -fno-sanitize-recover=undefined -fno-omit-frame-pointer -shared-libsan \
   "$R/oracle/oracle.c" -o "$O/liboracle.so" -lpthread -lm
RT=$(ls /opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so | head -1)
cd "$R"
GT_SANITIZED_DIR="$O" LD_PRELOAD="$RT" PYTHONPATH="$R/tests${PYTHONPATH:+:$PYTHONPATH}" \
ASAN_OPTIONS=detect_leaks=0:halt_on_error=1:abort_on_error=1 \
UBSAN_OPTIONS=halt_on_error=1:print_stacktrace=1 \
python -m pytest -p asan_libs tests/ -m "not gpu" -q -p no:cacheprovider "$@"
