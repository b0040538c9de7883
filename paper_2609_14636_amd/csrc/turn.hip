// turn.hip -- mean teacher log-probability of each turn, and each token's KL estimate.
//
// Eq. (4) (Sec. 3.1): lbar_k = (1/n_k) sum over the rows of turn k of
// log pi_T(y).  Sec. 3.2: each token's KL estimate between student and teacher is
// log pi_S(y) - log pi_T(y) (= -r_t of Eq. 1), written for the same rows in the
// same pass.
//
// One workgroup per turn.  Thread j sums rows a+j, a+j+256, ... in double
// (four rows in flight at a time, added in that order);
// the 256 partial sums are combined by a fixed shuffle tree and a fixed
// cross-wave order, so the mean does not depend on scheduling.  The kernel
// reads 4 (or 8) bytes per row and is latency-bound; it sits next to the
// row-scoring kernel, which moves 2 V bytes per row.
#include "common.hpp"

namespace stride {
namespace {

__global__ __launch_bounds__(256) void turn_mean_kernel(stride_layout L,
                                                        const float *__restrict__ logp_t,
                                                        const float *__restrict__ logp_s,
                                                        float *__restrict__ kl,
                                                        double *turn_mean, uint32_t *flags) {
    __shared__ double part[256 / kWave];
    const int64_t t = blockIdx.x;
    const int64_t a = L.turn_tok_off[t], b = L.turn_tok_off[t + 1];
    const bool bad = a < 0 || b > L.n_tokens || b < a || (t == 0 && a != 0) ||
                     (t == L.n_turns - 1 && b != L.n_tokens);
    if (bad) {
        if (threadIdx.x == 0) {
            turn_mean[t] = __builtin_nan("");
            raise_flag(flags, STRIDE_FLAG_BAD_OFFSETS);
        }
        return;
    }
    // four rows per thread in flight; the additions keep the row order a+j, a+j+256, ...
    double acc = 0.0;
    constexpr int U = 4;
    const int64_t stride = blockDim.x;
    int64_t i = a + threadIdx.x;
    for (; i + (U - 1) * stride < b; i += U * stride) {
        float lt[U], ls[U];
#pragma unroll
        for (int u = 0; u < U; ++u) lt[u] = logp_t[i + u * stride];
        if (kl) {
#pragma unroll
            for (int u = 0; u < U; ++u) ls[u] = logp_s[i + u * stride];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) acc += (double)lt[u];
        if (kl) {
#pragma unroll
            for (int u = 0; u < U; ++u) kl[i + u * stride] = ls[u] - lt[u];
        }
    }
    for (; i < b; i += stride) {
        const float lt = logp_t[i];
        acc += (double)lt;
        if (kl) kl[i] = logp_s[i] - lt;
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, kWave);
    const int wave = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) part[wave] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        double s = part[0];
        for (int w = 1; w < (int)(blockDim.x / kWave); ++w) s += part[w];
        const int64_t n = b - a;
        if (n == 0) {
            turn_mean[t] = __builtin_nan("");
            raise_flag(flags, STRIDE_FLAG_EMPTY_TURN);
        } else {
            turn_mean[t] = s / (double)n;
        }
    }
}

}  // namespace

hipError_t launch_turn_mean(const stride_layout &L, const float *logp_t, const float *logp_s,
                            float *kl, double *turn_mean, uint32_t *flags, hipStream_t stream) {
    if (L.n_turns == 0) return hipSuccess;
    hipLaunchKernelGGL(turn_mean_kernel, dim3((unsigned)L.n_turns), dim3(256), 0, stream, L, logp_t,
                       logp_s, kl, turn_mean, flags);
    return hipGetLastError();
}

}  // namespace stride
