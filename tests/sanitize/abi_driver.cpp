// Sanitizer driver for the host side of the C ABI (test infrastructure):
// built with the library sources by tests/test_sanitizers.py with the host
// pass under -fsanitize=address,undefined (device code is unaffected) and
// run as a child process on a machine without a GPU.  It exercises the
// host-only paths: status strings, workspace and capacity queries over their
// whole argument ranges, and every entry point with arguments that the
// host checks must reject before anything is launched.  Exit status 0 when
// every check passes.
#include <stdint.h>
#include <stdio.h>

#include "memoplan.h"

static int failures = 0;
#define CHECK(c)                                                             \
    do {                                                                     \
        if (!(c)) {                                                          \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c);  \
            ++failures;                                                      \
        }                                                                    \
    } while (0)

int main() {
    for (int32_t s = -6; s <= 2; ++s) CHECK(mp_status_string(s) != nullptr);
    CHECK(mp_status_reset(nullptr, nullptr) == MP_EINVAL);

    const int64_t sizes[] = {-5, -1, 0, 1, 255, 2000, 4096, 4097, 100000, 1 << 20,
                             (int64_t)1 << 30, (int64_t)1 << 40, INT64_MAX};
    for (int32_t op = -1; op <= 9; ++op)
        for (int64_t a : sizes)
            for (int64_t b : sizes) {
                (void)mp_workspace_size(op, a, b, 16);
                (void)mp_workspace_size(op, a, 16, b);
                if (op != MP_OP_PLAN_TRACE) (void)mp_workspace_bytes(op, a, b, 7);
            }
    CHECK(mp_workspace_bytes(MP_OP_PLAN_BATCH, -1, 0, 1) == 0);
    CHECK(mp_workspace_bytes(99, 10, 10, 1) == 0);
    for (int64_t len : sizes) {
        const int64_t cap = mp_batch_pair_capacity(len);
        CHECK((len >= 0 && len <= MP_BATCH_MAX_TRACE_LEN) ? cap > 0 : cap == -1);
    }

    // every entry point rejects bad host arguments without launching
    int64_t dummy64[4] = {0, 0, 0, 0};
    int32_t dummy32[4] = {0, 0, 0, 0};
    uint8_t dummy8[4] = {0, 0, 0, 0};
    int64_t* p64 = dummy64;
    int32_t* p32 = dummy32;
    CHECK(mp_plan_batch(p64, 1, p32, p64, p32, p32, 1, 1, 7, p64, p64, p64, p64, 1 << 20, p32,
                        nullptr) == MP_EINVAL);  // unknown policy
    CHECK(mp_plan_batch(p64, -1, p32, p64, p32, p32, 1, 1, 0, p64, p64, p64, p64, 1 << 20, p32,
                        nullptr) == MP_EINVAL);  // negative count
    CHECK(mp_plan_batch(p64, 1, p32, p64, p32, p32, 1, 1, 0, p64, p64, p64, p64, 1, p32,
                        nullptr) == MP_EINVAL);  // workspace too small
    CHECK(mp_plan_batch(p64, 1, p32, p64, p32, p32, 1, 5000, 0, p64, p64, p64, p64, 1 << 20, p32,
                        nullptr) == MP_EINVAL);  // trace bound beyond the batched planner
    CHECK(mp_plan_batch(p64, 1, p32, p64, p32, p32, 1, 1, 0, p64, p64, p64, p64, 1 << 20, nullptr,
                        nullptr) == MP_EINVAL);  // no status word
    CHECK(mp_plan_trace(p64, p32, p32, -1, 1, 0, p64, p64, p64, 1 << 20, p32, nullptr) ==
          MP_EINVAL);
    CHECK(mp_plan_trace(p64, p32, p32, 1, 1, 9, p64, p64, p64, 1 << 20, p32, nullptr) ==
          MP_EINVAL);
    CHECK(mp_plan_trace(p64, p32, p32, 1, 1, 0, p64, p64, p64, 1 << 20, nullptr, nullptr) ==
          MP_EINVAL);
    CHECK(mp_live_bytes_profile(p64, p32, p32, -1, 1, p64, p64, p64, 64, p32, nullptr) ==
          MP_EINVAL);
    CHECK(mp_live_bytes_profile(p64, p32, p32, 1, -1, p64, p64, p64, 64, p32, nullptr) ==
          MP_EINVAL);
    CHECK(mp_live_bytes_profile(p64, p32, p32, 1, 1, p64, p64, p64, 0, p32, nullptr) ==
          MP_EINVAL);
    CHECK(mp_live_bytes_profile_noalloc(p64, p32, p32, 1, MP_LIVE_NOALLOC_MAX_OPS + 1, p64, p64,
                                        p32, nullptr) == MP_EINVAL);
    CHECK(mp_validate_plan(p64, p32, p32, p64, -1, p64, 1, p64, 0, p64, 1 << 20, p32, nullptr) ==
          MP_EINVAL);
    CHECK(mp_validate_plan(p64, p32, p32, p64, 1, p64, -1, p64, 0, p64, 1 << 20, p32, nullptr) ==
          MP_EINVAL);
    CHECK(mp_validate_plan(p64, p32, p32, p64, 1, p64, 1, p64, 0, p64, 0, p32, nullptr) ==
          MP_EINVAL);
    CHECK(mp_validate_batch(p64, -1, p64, p32, p32, p64, 1, 0, p64, 1, p64, 0, p64, 1 << 20, p32,
                            nullptr) == MP_EINVAL);
    CHECK(mp_probe_plan(p64, p32, p32, p64, -1, 1, dummy8, 64, dummy8, p64, p64, 1 << 20, p32,
                        nullptr) == MP_EINVAL);
    CHECK(mp_bump_plan(nullptr, 1, p64, p32, p32, -1, 1, p64, p64, p64, 1 << 20, p32, nullptr) ==
          MP_EINVAL);
    CHECK(mp_optimal_batch(p64, -1, p32, p64, p32, p32, 1, p64, p64, p32, nullptr) == MP_EINVAL);
    CHECK(mp_plan_breadth_batch(p64, 1, p32, p64, p32, p32, 1, 7, p64, p64, p32, nullptr) ==
          MP_EINVAL);
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("ABI sanitizer driver: all checks passed\n");
    return 0;
}
