#!/bin/bash
# The tests that need no GPU, under AddressSanitizer and
# UndefinedBehaviorSanitizer: builds the host code of the HIP library, the
# marshalling module and the oracle with both sanitizers, runs pytest with
# clang's sanitizer runtime preloaded into python, then rebuilds all three
# without the sanitizers.  Extra arguments go to pytest.
set -u
cd "$(dirname "$0")/.."
python -m paper_2106_04718_amd.build --sanitize > /dev/null && python oracle/build.py --sanitize > /dev/null || exit 1
RT=$(python -c "from paper_2106_04718_amd import build; print(build.sanitizer_runtime())") || exit 1
LD_PRELOAD="$RT" \
ASAN_OPTIONS=detect_leaks=0:alloc_dealloc_mismatch=0:verify_asan_link_order=0 \
UBSAN_OPTIONS=print_stacktrace=1:halt_on_error=1 \
python -m pytest tests -m "not gpu" -x -q -p no:cacheprovider "$@"
rc=$?
python -m paper_2106_04718_amd.build > /dev/null && python oracle/build.py > /dev/null || exit 1
exit $rc
