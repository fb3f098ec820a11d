#!/bin/bash
# CPU sanitizer run (AddressSanitizer + UndefinedBehaviorSanitizer) of the two C/C++ parts that run
# on the host: the oracle (oracle/oracle.c) and the library's host code (page pool, plan building,
# argument validation in paper_2608_13667_amd/csrc/api.hip).  Both are built instrumented into a
# scratch copy of the tree, and the CPU tests that exercise them run there: the oracle pins under
# gcc's runtime, the pool / ABI / schedule tests under clang's (one runtime per process).  Device
# code is built as usual: only the host side is instrumented.  No GPU is used.
#   usage: tests/sanitize.sh            (exit status 0 = clean)
set -euo pipefail
ROOT=$(cd "$(dirname "$0")/.." && pwd)
T=$(mktemp -d /tmp/fka_sanitize.XXXXXX)
trap 'rm -rf "$T"' EXIT
cp -r "$ROOT/oracle" "$ROOT/paper_2608_13667_amd" "$ROOT/tests" "$ROOT/include" "$T/"
rm -rf "$T"/oracle/*.so "$T"/paper_2608_13667_amd/*.so "$T"/oracle/__pycache__ "$T"/tests/__pycache__
export ASAN_OPTIONS=detect_leaks=0:abort_on_error=1:halt_on_error=1
export UBSAN_OPTIONS=print_stacktrace=1:halt_on_error=1

echo "[sanitize] oracle: gcc -fsanitize=address,undefined"
gcc -O1 -g -fno-omit-frame-pointer -fopenmp -fPIC -shared -std=c11 -fsanitize=address,undefined \
    -fno-sanitize-recover=all "$T/oracle/oracle.c" -o "$T/oracle/liboracle.so" -lm
touch "$T/oracle/liboracle.so"
nm -D "$T/oracle/liboracle.so" | grep -q __asan_report_load || { echo "oracle not instrumented"; exit 1; }
(cd "$T" && LD_PRELOAD="$(gcc -print-file-name=libasan.so) $(gcc -print-file-name=libubsan.so)" \
    python3 -m pytest tests/test_oracle_pins.py -x -q -p no:cacheprovider)

echo "[sanitize] library host code: hipcc -Xarch_host -fsanitize=address,undefined"
HIPCC=/opt/rocm/bin/hipcc
FLAGS=(--offload-arch=gfx950 -O1 -g -std=c++17 -fPIC -ffp-contract=off -Xclang -target-feature -Xclang
       -packed-fp32-ops -I "$T/include" -Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined
       -Xarch_host -fno-sanitize-recover=all -Xarch_host -fno-omit-frame-pointer)
mkdir -p "$T/obj"
for f in api kernels partials prefill; do
    "$HIPCC" "${FLAGS[@]}" -c "$T/paper_2608_13667_amd/csrc/$f.hip" -o "$T/obj/$f.o" 2> "$T/obj/$f.log" &
done
wait
CLANG_RT=$(ls /opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so | head -1)
/opt/rocm/llvm/bin/clang++ -shared -fPIC -fsanitize=address,undefined -shared-libsan "$T"/obj/*.o \
    -L/opt/rocm/lib -lamdhip64 -Wl,-rpath,/opt/rocm/lib -o "$T/paper_2608_13667_amd/libforkattn.so"
nm -D "$T/paper_2608_13667_amd/libforkattn.so" | grep -q __asan_report_load || { echo "library not instrumented"; exit 1; }
(cd "$T" && LD_PRELOAD="$CLANG_RT" \
    python3 -m pytest tests/test_pool.py tests/test_abi.py tests/test_schedule.py -x -q -m "not gpu" -p no:cacheprovider)
echo "[sanitize] schedule arithmetic (internal.h): tests/native/sched_check.cpp"
/opt/rocm/llvm/bin/clang++ -std=c++17 -O1 -g -fsanitize=address,undefined -fno-sanitize-recover=all \
    -I "$T/paper_2608_13667_amd/csrc" -I /opt/rocm/include -D__HIP_PLATFORM_AMD__ "$T/tests/native/sched_check.cpp" \
    -L/opt/rocm/lib -lamdhip64 -Wl,-rpath,/opt/rocm/lib -o "$T/obj/sched_check"
"$T/obj/sched_check" 3000
echo "[sanitize] clean"
