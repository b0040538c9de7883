// grad.hip -- token-level OPD loss and its gradient with respect to the student logits.
//
// Eq. (2) (Sec. 3.1): L = - sum_t log pi_S(y_t) r_t 1_trainable(t), with
// r_t = log pi_T(y_t) - log pi_S(y_t) held constant (stop-gradient).  The
// trainable rows are the retained ones: units K0 .. stop of each rollout,
// including the unit that triggered the stop (Sec. 4.1, Algorithm 1).  For a
// retained row,  dL/ds_v = scale * r_t * (p_S(v) - [v = y_t]),  and the row's
// log-normaliser comes for free from the scoring pass: LSE_S = s_y - log pi_S(y),
// so p_S(v) = exp(s_v - s_y + log pi_S(y)).
//
// Eight wavefronts per row stream the student row once (16-byte non-temporal
// loads) and write the gradient row once; a row that is not retained is
// written as zeros without being read.  Columns ld - vocab of padding are not
// touched.  A small kernel first marks the retained rows.
#include "common.hpp"

namespace stride {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
// Wavefronts per row.  Measured against one wavefront per row on V = 151,936 bf16 rows (gradient
// bits equal): eight are faster at every batch size, 26% at 1,024 rows and 4.4% at 131,072
// (14.94 against 15.62 ms for the whole read + write of 79.7 GB).
constexpr int kGradWaves = 8;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ uint32_t bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u) return (u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// mask[i] = 1 if row i lies in a retained unit of its rollout, else 0.
__global__ __launch_bounds__(256) void grad_mask_kernel(stride_layout L, int32_t unit,
                                                        const int32_t *start, const int32_t *stop,
                                                        uint8_t *mask, uint32_t *flags) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= L.n_tokens) return;
    uint8_t m = 0;
    if (L.n_turns > 0 && L.turn_tok_off[0] <= i) {
        int64_t lo = 0, hi = L.n_turns;
        while (hi - lo > 1) {
            const int64_t mid = (lo + hi) >> 1;
            if (L.turn_tok_off[mid] <= i) lo = mid; else hi = mid;
        }
        const int64_t t = lo;
        if (i < L.turn_tok_off[t + 1] && L.n_rollouts > 0 && L.rollout_turn_off[0] <= t) {
            int64_t rlo = 0, rhi = L.n_rollouts;
            while (rhi - rlo > 1) {
                const int64_t mid = (rlo + rhi) >> 1;
                if (L.rollout_turn_off[mid] <= t) rlo = mid; else rhi = mid;
            }
            const int64_t t0 = L.rollout_turn_off[rlo], t1 = L.rollout_turn_off[rlo + 1];
            if (t < t1) {
                int64_t local, n;
                if (unit == STRIDE_UNIT_TURN) {
                    local = t - t0;
                    n = t1 - t0;
                } else {
                    local = i - L.turn_tok_off[t0];
                    n = L.turn_tok_off[t1] - L.turn_tok_off[t0];
                }
                int64_t k0 = start ? (int64_t)start[rlo] : 0;
                k0 = k0 < 0 ? 0 : (k0 > n ? n : k0);
                const int32_t s = stop ? stop[rlo] : -1;
                const int64_t last = (s >= 0 && (int64_t)s < n) ? (int64_t)s : n - 1;
                m = (local >= k0 && local <= last) ? 1 : 0;
            }
        } else {
            raise_flag(flags, STRIDE_FLAG_BAD_OFFSETS);
        }
    } else {
        raise_flag(flags, STRIDE_FLAG_BAD_OFFSETS);
    }
    mask[i] = m;
}

struct GradArgs {
    const void *student;
    const int32_t *ids;
    const float *logp_t;
    const float *logp_s;
    const uint8_t *mask;
    void *grad;
    float *loss;
    uint32_t *flags;
    int64_t n_rows;
    int64_t ld;
    int32_t vocab;
    float scale;
};

// One row per workgroup of W = kGradWaves wavefronts: wavefront w handles the row's U-load chunks
// w, w + W, ... and every W-th word after the last whole chunk.  Every element's gradient depends
// only on that element, so nothing is merged and the bits do not depend on the split.
template <int DT>
__global__ __launch_bounds__(kGradWaves *kWave) void opd_grad_kernel(GradArgs a) {
    constexpr int E = (DT == STRIDE_BF16) ? 8 : 4;
    constexpr int ES = (DT == STRIDE_BF16) ? 2 : 4;
    constexpr int W = kGradWaves;
    const int lane = threadIdx.x & (kWave - 1);
    const int sub = threadIdx.x / kWave;  // this wavefront's share of the row
    const int64_t row = blockIdx.x;       // the grid has exactly n_rows workgroups
    if (row >= a.n_rows) return;
    const size_t off = (size_t)row * a.ld * ES;
    const u32x4 *src = reinterpret_cast<const u32x4 *>(static_cast<const char *>(a.student) + off);
    u32x4 *dst = reinterpret_cast<u32x4 *>(static_cast<char *>(a.grad) + off);
    const int64_t nvec = a.vocab / E;
    const int tail = a.vocab % E;
    const int32_t y = a.ids[row];
    const float lps = a.logp_s[row], lpt = a.logp_t[row];
    const bool retained = a.mask[row] != 0;
    const float r = lpt - lps;  // OPD reward, held constant
    const bool ok = (y >= 0) && (y < a.vocab) && (lps == lps) && (lpt == lpt) &&
                    (lps > -INFINITY) && (lpt > -INFINITY);
    if (sub == 0 && lane == 0) {
        if (a.loss) a.loss[row] = retained ? (ok ? -a.scale * lps * r : __builtin_nanf("")) : 0.0f;
        if (retained && !ok) raise_flag(a.flags, STRIDE_FLAG_NONFINITE);
    }
    if (!retained) {
        const u32x4 z = {0u, 0u, 0u, 0u};
        for (int64_t k = (int64_t)sub * kWave + lane; k < nvec; k += (int64_t)W * kWave)
            __builtin_nontemporal_store(z, dst + k);
        if (tail && sub == 0 && lane == 0) {
            for (int j = 0; j < tail; ++j) {
                if (DT == STRIDE_BF16)
                    reinterpret_cast<uint16_t *>(dst + nvec)[j] = 0;
                else
                    reinterpret_cast<float *>(dst + nvec)[j] = 0.0f;
            }
        }
        return;
    }
    // log-normaliser from the scoring pass: LSE_S = s_y - log pi_S(y)
    float sy = 0.0f;
    if (ok) {
        if (DT == STRIDE_BF16)
            sy = __uint_as_float((uint32_t)(reinterpret_cast<const uint16_t *>(src)[y]) << 16);
        else
            sy = reinterpret_cast<const float *>(src)[y];
    }
    const float c = ok ? a.scale * r : __builtin_nanf("");
    const float lse_l2 = (sy - lps) * kLog2e;
    const int64_t yv = ok ? (int64_t)(y / E) : -1;
    const int yj = ok ? y % E : 0;
    auto grad_vec = [&](const u32x4 v, int64_t vi) -> u32x4 {
        float x[E];
        if (DT == STRIDE_BF16) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                x[2 * i] = __uint_as_float(v[i] << 16);
                x[2 * i + 1] = __uint_as_float(v[i] & 0xFFFF0000u);
            }
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) x[i] = __uint_as_float(v[i]);
        }
        float g[E];
#pragma unroll
        for (int j = 0; j < E; ++j) g[j] = c * ex2(__builtin_fmaf(x[j], kLog2e, -lse_l2));
        if (vi == yv) {
#pragma unroll
            for (int j = 0; j < E; ++j)
                if (j == yj) g[j] -= c;
        }
        u32x4 o;
        if (DT == STRIDE_BF16) {
#pragma unroll
            for (int i = 0; i < 4; ++i) o[i] = bf16_rne(g[2 * i]) | (bf16_rne(g[2 * i + 1]) << 16);
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) o[i] = __float_as_uint(g[i]);
        }
        return o;
    };
    constexpr int U = 4;
    constexpr int64_t kStep = (int64_t)U * kWave;
    const int64_t nfull = nvec / kStep;  // whole U-load chunks
    for (int64_t c = sub; c < nfull; c += W) {
        const int64_t k = c * kStep;
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(src + k + u * kWave + lane);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t vi = k + u * kWave + lane;
            __builtin_nontemporal_store(grad_vec(v[u], vi), dst + vi);
        }
    }
    for (int64_t k = nfull * kStep + (int64_t)sub * kWave; k < nvec; k += (int64_t)W * kWave) {
        const int64_t vi = k + lane;
        if (vi < nvec) __builtin_nontemporal_store(grad_vec(__builtin_nontemporal_load(src + vi), vi), dst + vi);
    }
    if (tail && sub == 0 && lane == 0) {
        const u32x4 g = grad_vec(src[nvec], nvec);
        for (int j = 0; j < tail; ++j) {
            if (DT == STRIDE_BF16)
                reinterpret_cast<uint16_t *>(dst + nvec)[j] =
                    (uint16_t)(j & 1 ? (g[j >> 1] >> 16) : (g[j >> 1] & 0xFFFFu));
            else
                reinterpret_cast<float *>(dst + nvec)[j] = __uint_as_float(g[j]);
        }
    }
}

}  // namespace

hipError_t launch_opd_grad(const stride_layout &L, int32_t unit, int32_t dtype, int32_t vocab,
                           int64_t ld, const void *student, const int32_t *ids,
                           const float *logp_t, const float *logp_s, const int32_t *start,
                           const int32_t *stop, float scale, void *grad, float *loss,
                           uint32_t *flags, uint8_t *mask, hipStream_t stream) {
    if (L.n_tokens == 0) return hipSuccess;
    const unsigned mb = (unsigned)((L.n_tokens + 255) / 256);
    hipLaunchKernelGGL(grad_mask_kernel, dim3(mb), dim3(256), 0, stream, L, unit, start, stop,
                       mask, flags);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    GradArgs a;
    a.student = student;
    a.ids = ids;
    a.logp_t = logp_t;
    a.logp_s = logp_s;
    a.mask = mask;
    a.grad = grad;
    a.loss = loss;
    a.flags = flags;
    a.n_rows = L.n_tokens;
    a.ld = ld;
    a.vocab = vocab;
    a.scale = scale;
    const unsigned rows = (unsigned)L.n_tokens;  // one workgroup per row
    if (dtype == STRIDE_BF16)
        hipLaunchKernelGGL(opd_grad_kernel<STRIDE_BF16>, dim3(rows), dim3(kGradWaves * kWave), 0, stream, a);
    else
        hipLaunchKernelGGL(opd_grad_kernel<STRIDE_F32>, dim3(rows), dim3(kGradWaves * kWave), 0, stream, a);
    return hipGetLastError();
}

}  // namespace stride
