// The host trajectory record (stride_records_*) under a sanitizer build: AddressSanitizer +
// UndefinedBehaviorSanitizer, or ThreadSanitizer.  Four threads put, get, plan and size the
// same store at once (overwriting each other's tasks), with and without masks, empty records,
// capacities below the record length and NULL optional outputs; then single-threaded checks of
// the restart pick against hand-worked values.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <thread>
#include <vector>

#include "../../include/stride.h"

#define EXPECT(c)                                                                        \
    do {                                                                                 \
        if (!(c)) {                                                                      \
            std::fprintf(stderr, "expectation failed at line %d: %s\n", __LINE__, #c); \
            std::exit(2);                                                                \
        }                                                                                \
    } while (0)

static void worker(stride_records *rec, int id) {
    std::vector<double> v;
    std::vector<uint8_t> m;
    for (int i = 0; i < 2000; ++i) {
        const int64_t task = (i * 7 + id) % 64;
        const int n = (i + id) % 13;  // 0 .. 12 units, including empty records
        v.assign((size_t)n, 0.0);
        m.assign((size_t)n, 1);
        for (int u = 0; u < n; ++u) {
            v[(size_t)u] = -0.1 * ((u * 5 + i) % 11);
            m[(size_t)u] = (uint8_t)((u + i) % 7 != 0);
        }
        EXPECT(stride_records_put(rec, task, n, n ? v.data() : nullptr,
                                  (i & 1) ? m.data() : nullptr) == STRIDE_OK);
        double out[4];
        uint8_t om[4];
        const int32_t got = stride_records_get(rec, task, 4, out, om);
        EXPECT(got >= 0 && got <= 12);
        EXPECT(stride_records_get(rec, task + 1000, 4, out, om) == -1);
        const int64_t tasks[3] = {task, (task + 1) % 64, 5000};
        const double alpha[3] = {-0.55, -INFINITY, 0.0};
        int32_t ks[3], k0[3], km[3];
        EXPECT(stride_records_plan(rec, 3, tasks, alpha, ks, k0, (i & 2) ? km : nullptr) == STRIDE_OK);
        EXPECT(ks[2] == -1 && k0[2] == 0);
        EXPECT(stride_records_size(rec) >= 1);
    }
}

int main() {
    stride_records *rec = stride_records_create();
    EXPECT(rec != nullptr);
    std::vector<std::thread> th;
    for (int t = 0; t < 4; ++t) th.emplace_back(worker, rec, t);
    for (auto &t : th) t.join();
    EXPECT(stride_records_size(rec) == 64);

    // the pick on known records: values -1, -3, -2, -4 with unit 2 wrong
    const double v[4] = {-1.0, -3.0, -2.0, -4.0};
    const uint8_t m[4] = {1, 1, 0, 1};
    EXPECT(stride_records_put(rec, 7, 4, v, m) == STRIDE_OK);
    const int64_t t7[1] = {7};
    int32_t ks, k0, km;
    const double a1[1] = {-10.0};
    EXPECT(stride_records_plan(rec, 1, t7, a1, &ks, &k0, &km) == STRIDE_OK);
    EXPECT(km == 2 && ks == 1 && k0 == 1);
    const double a2[1] = {-2.5};  // unit 1 (-3) is not above alpha: the run stops at 1
    EXPECT(stride_records_plan(rec, 1, t7, a2, &ks, &k0, &km) == STRIDE_OK);
    EXPECT(km == 1 && ks == 0 && k0 == 0);
    const double a3[1] = {NAN};   // nothing is above NaN
    EXPECT(stride_records_plan(rec, 1, t7, a3, &ks, &k0, &km) == STRIDE_OK);
    EXPECT(km == 0 && ks == -1 && k0 == 0);
    double back[2];
    uint8_t bm[2];
    EXPECT(stride_records_get(rec, 7, 2, back, bm) == 4 && back[1] == -3.0 && bm[0] == 1);
    EXPECT(stride_records_get(rec, 7, 0, nullptr, nullptr) == 4);

    // argument errors
    EXPECT(stride_records_put(nullptr, 1, 1, v, nullptr) == STRIDE_ERR_INVALID_ARG);
    EXPECT(stride_records_put(rec, 1, -1, v, nullptr) == STRIDE_ERR_INVALID_ARG);
    EXPECT(stride_records_put(rec, 1, 2, nullptr, nullptr) == STRIDE_ERR_INVALID_ARG);
    EXPECT(stride_records_plan(rec, 1, nullptr, a1, &ks, &k0, &km) == STRIDE_ERR_INVALID_ARG);
    EXPECT(stride_records_plan(rec, -1, t7, a1, &ks, &k0, &km) == STRIDE_ERR_INVALID_ARG);
    EXPECT(stride_records_get(nullptr, 7, 2, back, bm) == -1);
    EXPECT(stride_records_size(nullptr) == -1);
    stride_records_destroy(rec);
    stride_records_destroy(nullptr);
    std::printf("records driver ok\n");
    return 0;
}
