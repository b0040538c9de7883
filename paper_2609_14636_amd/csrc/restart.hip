// restart.hip -- prefix-buffer restart pick of the weakest correct unit.
//
// Sec. 4.2 step 1: unit k is correct iff its value exceeds alpha (strictly),
// here also requiring its correctness-mask bit.  Step 2 and Eq. (6): K_max
// counts the correct units from the start of the record up to the first one
// that is not, and k* is the argmin of the values among those K_max units.  Step 3 and Algorithm 1: the next rollout reuses K0 = k* - 1
// turns (1-based) as context; a task without a usable prefix starts from 0.
// The record is the rollout's units up to and including its stop (Algorithm 1
// records the generated turns).  Ties go to the lowest index.
//
// One workgroup per rollout.  Pass 1 finds the first non-correct unit of the
// record with a block-wide integer min over 2048-unit chunks, stopping at the
// first chunk that has one.  Pass 2 takes the lexicographic min of
// (value, index) over [0, K_max), so the pick is exact and deterministic.
#include <climits>

#include "common.hpp"

namespace stride {
namespace {

struct RestartArgs {
    stride_layout L;
    DomainTable alpha;
    int32_t n_dom;
    int32_t unit;
    const void *values;
    const int32_t *stop_unit;
    const uint8_t *mask;
    int32_t *k_star;
    int32_t *k0;
    int32_t *k_max;
    uint32_t *flags;
};

template <typename VT>
__global__ __launch_bounds__(256) void restart_kernel(RestartArgs a) {
    __shared__ int64_t s_min;
    __shared__ double s_val[256 / kWave];
    __shared__ int64_t s_idx[256 / kWave];
    const int64_t r = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int64_t T = a.L.n_turns;
    const int64_t t0 = a.L.rollout_turn_off[r], t1 = a.L.rollout_turn_off[r + 1];
    bool bad_off = t0 < 0 || t1 > T || t1 < t0;
    int64_t first = 0, n = 0;
    if (!bad_off) {
        if (a.unit == STRIDE_UNIT_TURN) {
            first = t0;
            n = t1 - t0;
        } else {
            first = a.L.turn_tok_off[t0];
            n = a.L.turn_tok_off[t1] - first;
            bad_off = first < 0 || n < 0 || first + n > a.L.n_tokens;
        }
    }
    const int32_t d = a.L.domain ? a.L.domain[r] : 0;
    const bool bad_dom = d < 0 || d >= a.n_dom;
    if (bad_off || bad_dom) {
        if (tid == 0) {
            a.k_star[r] = -1;
            a.k0[r] = 0;
            if (a.k_max) a.k_max[r] = 0;
            raise_flag(a.flags, bad_off ? STRIDE_FLAG_BAD_OFFSETS : STRIDE_FLAG_BAD_DOMAIN);
        }
        return;
    }
    int64_t len = n;
    if (a.stop_unit) {
        const int32_t s = a.stop_unit[r];
        if (s >= 0 && (int64_t)s + 1 < n) len = (int64_t)s + 1;
    }
    const double alpha = a.alpha.v[d];
    const VT *vals = static_cast<const VT *>(a.values);

    // ---- pass 1: K_max = first non-correct unit in [0, len), else len ----
    // chunks of 8 units per thread (eight loads in flight); the first chunk holding a
    // non-correct unit ends the search, and the min over it is exact
    constexpr int PU = 8;
    if (tid == 0) s_min = len;
    __syncthreads();
    for (int64_t c = 0; c < len; c += (int64_t)blockDim.x * PU) {
        int64_t local = LLONG_MAX;
#pragma unroll
        for (int k = 0; k < PU; ++k) {
            const int64_t u = c + (int64_t)k * blockDim.x + tid;
            if (u < len) {
                const double v = (double)vals[first + u];
                const bool ok = (a.mask == nullptr || a.mask[first + u] != 0) && (v > alpha);
                if (!ok && u < local) local = u;
            }
        }
        if (local != LLONG_MAX) atomicMin((unsigned long long *)&s_min, (unsigned long long)local);
        __syncthreads();
        const bool done = s_min < len;
        __syncthreads();  // every thread has read s_min before any thread updates it again
        if (done) break;
    }
    const int64_t kmax = s_min;

    // ---- pass 2: lowest index of the minimum over [0, K_max) ----
    double best = __builtin_inf();
    int64_t bidx = LLONG_MAX;
    for (int64_t c = 0; c < kmax; c += (int64_t)blockDim.x * PU) {
        double v[PU];
#pragma unroll
        for (int k = 0; k < PU; ++k) {
            const int64_t u = c + (int64_t)k * blockDim.x + tid;
            v[k] = u < kmax ? (double)vals[first + u] : __builtin_inf();
        }
#pragma unroll
        for (int k = 0; k < PU; ++k) {
            const int64_t u = c + (int64_t)k * blockDim.x + tid;
            // u increases, so the first hit per thread is its lowest index; the first unit
            // always counts, so values of +inf still give an index
            if (u < kmax && (v[k] < best || bidx == LLONG_MAX)) {
                best = v[k];
                bidx = u;
            }
        }
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const double v2 = __shfl_xor(best, off, kWave);
        const int64_t i2 = __shfl_xor(bidx, off, kWave);
        if (v2 < best || (v2 == best && i2 < bidx)) {
            best = v2;
            bidx = i2;
        }
    }
    if (lane == 0) {
        s_val[wave] = best;
        s_idx[wave] = bidx;
    }
    __syncthreads();
    if (tid == 0) {
        for (int w = 1; w < (int)(blockDim.x / kWave); ++w) {
            if (s_val[w] < best || (s_val[w] == best && s_idx[w] < bidx)) {
                best = s_val[w];
                bidx = s_idx[w];
            }
        }
        const int32_t ks = kmax > 0 ? (int32_t)bidx : -1;
        a.k_star[r] = ks;
        a.k0[r] = ks > 0 ? ks : 0;
        if (a.k_max) a.k_max[r] = (int32_t)kmax;
    }
}

}  // namespace

hipError_t launch_restart(const stride_layout &L, int32_t unit, const void *values,
                          const int32_t *stop_unit, const DomainTable &alpha, int32_t n_dom,
                          const uint8_t *mask, int32_t *k_star, int32_t *k0, int32_t *k_max,
                          uint32_t *flags, hipStream_t stream) {
    if (L.n_rollouts == 0) return hipSuccess;
    RestartArgs a;
    a.L = L;
    a.alpha = alpha;
    a.n_dom = n_dom;
    a.unit = unit;
    a.values = values;
    a.stop_unit = stop_unit;
    a.mask = mask;
    a.k_star = k_star;
    a.k0 = k0;
    a.k_max = k_max;
    a.flags = flags;
    if (unit == STRIDE_UNIT_TURN)
        hipLaunchKernelGGL(restart_kernel<double>, dim3((unsigned)L.n_rollouts), dim3(256), 0,
                           stream, a);
    else
        hipLaunchKernelGGL(restart_kernel<float>, dim3((unsigned)L.n_rollouts), dim3(256), 0,
                           stream, a);
    return hipGetLastError();
}

}  // namespace stride
