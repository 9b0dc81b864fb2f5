#!/bin/bash
# The CPU tests against sanitized host builds: the oracle and the library's
# host code (plan parsing, classification, workspace layout, argument checks)
# compiled with AddressSanitizer + UBSan by clang (no device code), loaded
# by the tests through TRE_HOST_SANITIZED=1 with clang's sanitizer runtime
# preloaded into python.  CPU only; extra arguments go to pytest.
set -euo pipefail
cd "$(dirname "$0")/.."
export TRE_HOST_SANITIZED=1
python -m paper_2603_08957_amd.build --host-sanitized
python -c "import oracle; oracle.build(force=True)"
RT=$(/opt/rocm/llvm/bin/clang -print-file-name=libclang_rt.asan-x86_64.so)
export ASAN_OPTIONS=detect_leaks=0:halt_on_error=1:abort_on_error=1
export UBSAN_OPTIONS=halt_on_error=1:print_stacktrace=1
# --capture=sys: sanitizer reports (written to fd 2) reach the terminal
LD_PRELOAD="$RT" python -m pytest tests -m "not gpu" -q -p no:cacheprovider --capture=sys "$@"
