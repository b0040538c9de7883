// record.cpp -- the per-task trajectory record H(x) of the prefix buffer (host side).
//
// Algorithm 1 keeps, for every task x, the per-unit teacher signal of its last
// rollout ({lbar_k}, the record written after each rollout) and, at the next
// visit, reads it back to choose where to restart: K_max (the length of the
// leading run of correct units), k* (the weakest unit of that run, Eq. 6) and
// K0 (Sec. 4.2 steps 1-3); a task without a record starts from K0 = 0.
// The store is host memory owned through an opaque handle; all calls are
// thread-safe (one mutex).  Values are doubles (turn means from stride_score, or
// token log-probabilities in the single-turn setting), with an optional per-unit
// correctness mask.
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <unordered_map>
#include <vector>

#include "../../include/stride.h"

struct stride_records {
    std::mutex mu;
    std::unordered_map<int64_t, std::pair<std::vector<double>, std::vector<uint8_t>>> map;
};

namespace {

// Leading run of correct units and the lowest-index weakest one (Sec. 4.2, Eq. 6).
void pick(const std::vector<double> &v, const std::vector<uint8_t> &mask, double alpha,
          int32_t *k_star, int32_t *k0, int32_t *k_max) {
    const int32_t n = (int32_t)v.size();
    int32_t km = 0;
    while (km < n && (mask.empty() || mask[km] != 0) && v[km] > alpha) ++km;
    int32_t best = -1;
    for (int32_t u = 0; u < km; ++u)
        if (best < 0 || v[u] < v[best]) best = u;
    *k_star = best;
    *k0 = best > 0 ? best : 0;
    *k_max = km;
}

}  // namespace

extern "C" {

stride_records *stride_records_create(void) { return new (std::nothrow) stride_records(); }

void stride_records_destroy(stride_records *rec) { delete rec; }

stride_status stride_records_put(stride_records *rec, int64_t task, int32_t n_units,
                                 const double *values, const uint8_t *mask) {
    if (!rec) return STRIDE_ERR_INVALID_ARG;
    if (n_units < 0 || (n_units > 0 && !values)) return STRIDE_ERR_INVALID_ARG;
    std::vector<double> v(values, values + n_units);
    std::vector<uint8_t> m;
    if (mask) m.assign(mask, mask + n_units);
    std::lock_guard<std::mutex> lock(rec->mu);
    rec->map[task] = std::make_pair(std::move(v), std::move(m));
    return STRIDE_OK;
}

int32_t stride_records_get(stride_records *rec, int64_t task, int32_t capacity, double *values,
                           uint8_t *mask) {
    if (!rec) return -1;
    std::lock_guard<std::mutex> lock(rec->mu);
    auto it = rec->map.find(task);
    if (it == rec->map.end()) return -1;
    const auto &v = it->second.first;
    const auto &m = it->second.second;
    const int32_t n = (int32_t)v.size();
    const int32_t c = capacity < n ? capacity : n;
    if (values && c > 0) std::memcpy(values, v.data(), sizeof(double) * (size_t)c);
    if (mask && c > 0) {
        if (m.empty())
            std::memset(mask, 1, (size_t)c);
        else
            std::memcpy(mask, m.data(), (size_t)c);
    }
    return n;
}

int64_t stride_records_size(stride_records *rec) {
    if (!rec) return -1;
    std::lock_guard<std::mutex> lock(rec->mu);
    return (int64_t)rec->map.size();
}

stride_status stride_records_plan(stride_records *rec, int32_t n_tasks, const int64_t *tasks,
                                  const double *alpha, int32_t *k_star, int32_t *k0,
                                  int32_t *k_max) {
    if (!rec || n_tasks < 0) return STRIDE_ERR_INVALID_ARG;
    if (n_tasks > 0 && (!tasks || !alpha || !k_star || !k0)) return STRIDE_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lock(rec->mu);
    for (int32_t i = 0; i < n_tasks; ++i) {
        auto it = rec->map.find(tasks[i]);
        int32_t ks = -1, z = 0, km = 0;
        if (it != rec->map.end()) pick(it->second.first, it->second.second, alpha[i], &ks, &z, &km);
        k_star[i] = ks;
        k0[i] = z;
        if (k_max) k_max[i] = km;
    }
    return STRIDE_OK;
}

}  // extern "C"
