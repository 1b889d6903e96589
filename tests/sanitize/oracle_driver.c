/*
 * Sanitizer driver for the CPU oracle (test infrastructure): built together
 * with oracle/memoplan_oracle.c under -fsanitize=address,undefined by
 * tests/test_sanitizers.py and run as a child process.  It calls every
 * oracle entry point on the hand-worked examples and on seeded random traces
 * and checks results that hold by definition (validity, live bytes by
 * direct sums, brute-force conflicts of a corrupted plan), so that an
 * out-of-bounds access or undefined behaviour in any path is reported.
 * Exit status 0 when every check passes.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "memoplan_oracle.h"

static int failures = 0;
#define CHECK(c)                                                         \
    do {                                                                 \
        if (!(c)) {                                                      \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            ++failures;                                                  \
        }                                                                \
    } while (0)

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint32_t rnd(uint32_t m) { /* xorshift64*, uniform enough for test inputs */
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return (uint32_t)((rng_state * 0x2545F4914F6CDD1Dull) >> 33) % m;
}

/* Hand-worked example E5 (five tensors, greedy above the optimum). */
static void hand_example(void) {
    const int64_t size[5] = {256, 64, 256, 192, 128};
    const int32_t first[5] = {3, 1, 0, 0, 2};
    const int32_t last[5] = {3, 2, 1, 2, 3};
    const int64_t want[5] = {0, 576, 0, 256, 448};
    int64_t off[5], peak = -1;
    CHECK(mpo_plan_trace(size, first, last, 5, 4, MPO_LOWEST_FIT, off, &peak) == 0);
    CHECK(peak == 640);
    for (int i = 0; i < 5; ++i) CHECK(off[i] == want[i]);
    int64_t opt_off[5], opt = -1;
    CHECK(mpo_optimal_plan(size, first, last, 5, 4, opt_off, &opt) == 0);
    CHECK(opt == 512);
    int64_t live[4], mx = -1;
    CHECK(mpo_live_bytes_profile(size, first, last, 5, 4, live, &mx) == 0);
    CHECK(mx == 512);
}

static void random_trace(int n, int32_t num_ops, int64_t* size, int32_t* first, int32_t* last) {
    for (int i = 0; i < n; ++i) {
        first[i] = (int32_t)rnd((uint32_t)num_ops);
        int32_t l = first[i] + (int32_t)rnd(6);
        last[i] = l < num_ops ? l : num_ops - 1;
        size[i] = 64 * (int64_t)(1 + rnd(64));
    }
}

static int meets(const int32_t* f, const int32_t* l, int i, int j) {
    return f[i] <= l[j] && f[j] <= l[i];
}

static void random_checks(int n, int32_t num_ops) {
    int64_t* size = malloc(sizeof(int64_t) * (size_t)n);
    int32_t* first = malloc(sizeof(int32_t) * (size_t)n);
    int32_t* last = malloc(sizeof(int32_t) * (size_t)n);
    int64_t* off = malloc(sizeof(int64_t) * (size_t)n);
    int64_t* live = malloc(sizeof(int64_t) * (size_t)num_ops);
    int32_t* order = malloc(sizeof(int32_t) * (size_t)n);
    uint8_t* clob = malloc((size_t)n);
    const int64_t cap = (int64_t)n * (n - 1) / 2 + 1;
    int64_t* pairs = malloc(sizeof(int64_t) * 2 * (size_t)cap);
    random_trace(n, num_ops, size, first, last);
    CHECK(mpo_check_trace(size, first, last, n, num_ops) == 0);
    CHECK(mpo_rank_order(size, first, n, order) == 0);
    for (int k = 1; k < n; ++k) {
        const int a = order[k - 1], b = order[k];
        CHECK(size[a] > size[b] || (size[a] == size[b] && (first[a] < first[b] ||
                                                           (first[a] == first[b] && a < b))));
    }
    for (int policy = 0; policy < 2; ++policy) {
        int64_t peak = -1, nconf = -1;
        CHECK(mpo_plan_trace(size, first, last, n, num_ops, policy, off, &peak) == 0);
        CHECK(mpo_validate_plan(size, first, last, off, n, pairs, cap, &nconf) == 0);
        CHECK(nconf == 0);
        int64_t peak_w = -1;
        int64_t* off_w = malloc(sizeof(int64_t) * (size_t)n);
        CHECK(mpo_plan_trace_w(size, first, last, n, num_ops, policy, 3, off_w, &peak_w) == 0);
        CHECK(peak_w == peak);
        CHECK(memcmp(off_w, off, sizeof(int64_t) * (size_t)n) == 0);
        free(off_w);
        int64_t nclob = -1;
        CHECK(mpo_probe_plan(size, first, last, off, n, num_ops, clob, &nclob) == 0);
        CHECK(nclob == 0);
        CHECK(mpo_plan_breadth(size, first, last, n, num_ops, policy, off, &peak) == 0);
        CHECK(mpo_validate_plan(size, first, last, off, n, pairs, cap, &nconf) == 0);
        CHECK(nconf == 0);
    }
    int64_t mx = -1;
    CHECK(mpo_live_bytes_profile(size, first, last, n, num_ops, live, &mx) == 0);
    for (int32_t t = 0; t < num_ops; ++t) {
        int64_t s = 0;
        for (int i = 0; i < n; ++i) s += (first[i] <= t && t <= last[i]) ? size[i] : 0;
        CHECK(live[t] == s);
    }
    int64_t bpeak = -1;
    CHECK(mpo_bump_plan(size, first, last, n, num_ops, off, &bpeak) == 0);
    CHECK(mpo_breadth_order(size, first, last, n, num_ops, order) == 0);
    /* a corrupted plan: everything at offset 0 conflicts exactly where lifetimes meet */
    memset(off, 0, sizeof(int64_t) * (size_t)n);
    int64_t nconf = -1, want = 0;
    for (int i = 0; i < n; ++i)
        for (int j = i + 1; j < n; ++j) want += meets(first, last, i, j);
    CHECK(mpo_validate_plan(size, first, last, off, n, pairs, cap, &nconf) == 0);
    CHECK(nconf == want);
    /* a pairs buffer one short reports capacity and still counts exactly */
    if (want > 0) {
        CHECK(mpo_validate_plan(size, first, last, off, n, pairs, want - 1, &nconf) == -2);
        CHECK(nconf == want);
    }
    if (n <= 8) {
        int64_t opt = -1;
        CHECK(mpo_optimal_plan(size, first, last, n, num_ops, off, &opt) == 0);
        CHECK(opt <= bpeak);
    }
    free(size); free(first); free(last); free(off); free(live); free(order); free(clob);
    free(pairs);
}

static void invalid_inputs(void) {
    int64_t size[2] = {64, -64};
    int32_t first[2] = {0, 0}, last[2] = {1, 1};
    int64_t off[2], peak;
    CHECK(mpo_check_trace(size, first, last, 2, 2) != 0);
    CHECK(mpo_plan_trace(size, first, last, 2, 2, MPO_LOWEST_FIT, off, &peak) != 0);
    size[1] = 64;
    last[1] = 5; /* beyond num_ops */
    CHECK(mpo_check_trace(size, first, last, 2, 2) != 0);
    peak = -1;
    CHECK(mpo_plan_trace(size, first, last, 0, 0, MPO_LOWEST_FIT, off, &peak) == 0);
    CHECK(peak == 0);
}

int main(void) {
    hand_example();
    invalid_inputs();
    for (int it = 0; it < 40; ++it) random_checks(1 + (int)rnd(60), 1 + (int32_t)rnd(40));
    random_checks(7, 5);
    random_checks(400, 200);
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("oracle sanitizer driver: all checks passed\n");
    return 0;
}
