// score.hip -- sampled-token log-probabilities of teacher and student rows.
//
// Eq. (1) (Sec. 3.1): log pi(y_t | y_<t) = x[y_t] - log sum_v exp(x[v]) over the
// row's V logits.  Each row is read exactly once from HBM.
//
// Design (gfx950, wave64): one wavefront per row; a workgroup holds eight
// independent rows (small batches instead share each row among the eight
// wavefronts of a workgroup: score_rows_split_kernel).  Lanes stream the row
// with 16-byte non-temporal loads (8 bf16 or 4 fp32 per load, consecutive
// lanes on consecutive 16-byte words, so one wave instruction moves 1 KiB,
// fully coalesced).  Each lane keeps a
// running (max m, sum s) in fp32 registers and rescales once per chunk of
// U loads, not once per element (online normaliser, Milakov and Gimelshein
// 2018).  Per element the work is: unpack (shift or mask), max, one fma into
// the exp2 argument, v_exp_f32, add.  The 64 lane states are merged with a
// fixed butterfly of cross-lane shuffles, so the result does not depend on
// timing.  The sampled logit is fetched with one scalar-sized load per row.
#include "common.hpp"

namespace stride {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;
constexpr uint8_t kBadDomain = 0xFF;
// Row items (teacher and student rows) below which each row gets a workgroup of kSplitWaves
// wavefronts instead of one wavefront.  Measured on V = 151,936 bf16 rows: the shared rows read
// as fast or faster up to 16,384 items (64 rows: 14 us against 61 us) and 1-2% slower from
// 32,768 items on, where one wavefront per row already fills the chip.
constexpr int kSplitWaves = 8;
constexpr int64_t kSplitBelow = 16384;
// Tokens below which the paired pass (exact KL) shares each token's two rows the same way:
// measured, the shared form is as fast or faster up to 65,536 tokens (64 tokens: 25 us against
// 108 us) and 0.7-1.4% slower at 85,185 and 131,072.
constexpr int64_t kPairSplitBelow = 65536;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int DT>
struct Elem;
template <>
struct Elem<STRIDE_BF16> {
    static constexpr int kPerVec = 8;
    static constexpr int kSize = 2;
};
template <>
struct Elem<STRIDE_F32> {
    static constexpr int kPerVec = 4;
    static constexpr int kSize = 4;
};

template <int DT>
__device__ __forceinline__ void unpack(const u32x4 &v, float *x);

template <>
__device__ __forceinline__ void unpack<STRIDE_BF16>(const u32x4 &v, float *x) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[2 * i] = __uint_as_float(v[i] << 16);
        x[2 * i + 1] = __uint_as_float(v[i] & 0xFFFF0000u);
    }
}

template <>
__device__ __forceinline__ void unpack<STRIDE_F32>(const u32x4 &v, float *x) {
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = __uint_as_float(v[i]);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Fold n values into the lane's running (m, s0 + s1).  The reference point is
// the running maximum; a state that has only seen -inf keeps reference 0 so
// that -inf - -inf never appears.
template <int N>
__device__ __forceinline__ void fold(float &m, float &s0, float &s1, const float *x) {
    float cm = x[0];
#pragma unroll
    for (int i = 1; i < N; ++i) cm = fmaxf(cm, x[i]);
    const float mn = fmaxf(m, cm);
    const float ref = (mn == -INFINITY) ? 0.0f : mn;
    const float scale = fast_exp2((m - ref) * kLog2e);
    s0 *= scale;
    s1 *= scale;
    const float mref = ref * kLog2e;
#pragma unroll
    for (int i = 0; i < N; i += 2) {
        s0 += fast_exp2(__builtin_fmaf(x[i], kLog2e, -mref));
        if (i + 1 < N) s1 += fast_exp2(__builtin_fmaf(x[i + 1], kLog2e, -mref));
    }
    m = mn;
}

// Merge two (m, s) states.
__device__ __forceinline__ void merge(float &m, float &s, float m2, float s2) {
    const float mn = fmaxf(m, m2);
    const float ref = (mn == -INFINITY) ? 0.0f : mn;
    s = s * fast_exp2((m - ref) * kLog2e) + s2 * fast_exp2((m2 - ref) * kLog2e);
    m = mn;
}

struct ScoreArgs {
    PtrTable teachers;
    const void *student;
    const uint8_t *row_dom;
    const int32_t *ids;
    float *logp_t;
    float *logp_s;
    uint32_t *flags;
    int64_t n_rows;
    int64_t ld;
    int32_t vocab;
    int32_t n_teachers;
};

// Merge the 64 lane states of a wavefront with a fixed butterfly of cross-lane shuffles (every
// lane ends with the same result, so it does not depend on timing).
__device__ __forceinline__ void wave_merge(float &m, float &s) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const float m2 = __shfl_xor(m, off, kWave);
        const float s2 = __shfl_xor(s, off, kWave);
        merge(m, s, m2, s2);
    }
}

// The row's result from its (max, sum): log pi(y) = x_y - m - log s, NaN and a flag for a
// non-finite row or a token id outside [0, V).
template <int DT>
__device__ __forceinline__ void write_row(const ScoreArgs &a, int64_t row, const u32x4 *p, float m,
                                          float s, float *out) {
    const int32_t y = a.ids[row];
    float r;
    uint32_t bad = 0;
    const bool finite = (m > -INFINITY) && (m < INFINITY) && (s > 0.0f) && (s < INFINITY);
    if (!finite) bad |= STRIDE_FLAG_NONFINITE;
    if (y < 0 || y >= a.vocab) bad |= STRIDE_FLAG_TOKEN_OOB;
    if (bad) {
        r = __builtin_nanf("");
        raise_flag(a.flags, bad);
    } else {
        float xy;
        if (DT == STRIDE_BF16)
            xy = __uint_as_float((uint32_t)(reinterpret_cast<const uint16_t *>(p)[y]) << 16);
        else
            xy = reinterpret_cast<const float *>(p)[y];
        // At most 0: the maximum's own term is 1 in exact arithmetic.  Here it is exp2 of the
        // rounding residual of m * log2(e) (the exponent argument is one fma against that
        // rounded product), which can sit a few 1e-7 below 1; the clamp removes only that
        // excess (-inf stays -inf).
        r = fminf((xy - m) - __builtin_amdgcn_logf(s) * kLn2, 0.0f);
    }
    out[row] = r;
}

template <int DT, int U>
__global__ __launch_bounds__(kRowThreads) void score_rows_kernel(ScoreArgs a) {
    constexpr int E = Elem<DT>::kPerVec;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t item = (int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave);
    const bool two = a.student != nullptr;
    const int64_t n_items = two ? 2 * a.n_rows : a.n_rows;
    if (item >= n_items) return;
    const bool is_student = two && (item & 1);
    const int64_t row = two ? (item >> 1) : item;
    float *out = is_student ? a.logp_s : a.logp_t;

    const void *base;
    if (is_student) {
        base = a.student;
    } else {
        const int d = a.row_dom ? (int)a.row_dom[row] : 0;
        if (d >= a.n_teachers) {  // row not covered by the layout or bad domain (already flagged)
            if (lane == 0) out[row] = __builtin_nanf("");
            return;
        }
        base = a.teachers.p[d];
    }
    const u32x4 *p = reinterpret_cast<const u32x4 *>(static_cast<const char *>(base) +
                                                     row * a.ld * Elem<DT>::kSize);
    const int64_t nvec = a.vocab / E;  // 16-byte words lying wholly inside [0, vocab)
    const int tail = a.vocab % E;

    float m = -INFINITY, s0 = 0.0f, s1 = 0.0f;
    int64_t k = 0;
    constexpr int64_t kStep = (int64_t)U * kWave;
    for (; k + kStep <= nvec; k += kStep) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(p + k + u * kWave + lane);
        float x[U * E];
#pragma unroll
        for (int u = 0; u < U; ++u) unpack<DT>(v[u], x + u * E);
        fold<U * E>(m, s0, s1, x);
    }
    for (; k < nvec; k += kWave) {
        if (k + lane < nvec) {
            u32x4 v = __builtin_nontemporal_load(p + k + lane);
            float x[E];
            unpack<DT>(v, x);
            fold<E>(m, s0, s1, x);
        }
    }
    if (tail && lane == 0) {
        // The last word also holds ld - vocab padding elements: mask them out.
        u32x4 v = p[nvec];
        float x[E];
        unpack<DT>(v, x);
#pragma unroll
        for (int j = 0; j < E; ++j)
            if (j >= tail) x[j] = -INFINITY;
        fold<E>(m, s0, s1, x);
    }
    float s = s0 + s1;
    wave_merge(m, s);
    if (lane == 0) write_row<DT>(a, row, p, m, s, out);
}

// Batches too small to fill the chip with one wavefront per row (the online setting scores a
// few hundred rows per call): a workgroup of kSplitWaves wavefronts shares each row.  Wave w
// folds the row's U-load chunks w, w + kSplitWaves, ... and every kSplitWaves-th of the words
// after the last whole chunk; the waves' (max, sum) states are merged in wave order through
// LDS, so the result does not depend on timing (it differs from score_rows_kernel's only in
// the order of rounding).
template <int DT, int U>
__global__ __launch_bounds__(kSplitWaves *kWave) void score_rows_split_kernel(ScoreArgs a) {
    constexpr int E = Elem<DT>::kPerVec;
    __shared__ float s_m[kSplitWaves], s_s[kSplitWaves];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t item = blockIdx.x;  // one workgroup per item: the grid has exactly n_items
    const bool two = a.student != nullptr;
    const bool is_student = two && (item & 1);
    const int64_t row = two ? (item >> 1) : item;
    float *out = is_student ? a.logp_s : a.logp_t;

    const void *base;
    if (is_student) {
        base = a.student;
    } else {
        const int d = a.row_dom ? (int)a.row_dom[row] : 0;
        if (d >= a.n_teachers) {  // the same for the whole workgroup: it leaves before any barrier
            if (threadIdx.x == 0) out[row] = __builtin_nanf("");
            return;
        }
        base = a.teachers.p[d];
    }
    const u32x4 *p = reinterpret_cast<const u32x4 *>(static_cast<const char *>(base) +
                                                     row * a.ld * Elem<DT>::kSize);
    const int64_t nvec = a.vocab / E;
    const int tail = a.vocab % E;
    constexpr int64_t kStep = (int64_t)U * kWave;
    const int64_t nfull = nvec / kStep;  // whole U-load chunks

    float m = -INFINITY, s0 = 0.0f, s1 = 0.0f;
    for (int64_t c = wave; c < nfull; c += kSplitWaves) {
        const int64_t k = c * kStep;
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(p + k + u * kWave + lane);
        float x[U * E];
#pragma unroll
        for (int u = 0; u < U; ++u) unpack<DT>(v[u], x + u * E);
        fold<U * E>(m, s0, s1, x);
    }
    for (int64_t k = nfull * kStep + (int64_t)wave * kWave; k < nvec; k += (int64_t)kSplitWaves * kWave) {
        if (k + lane < nvec) {
            u32x4 v = __builtin_nontemporal_load(p + k + lane);
            float x[E];
            unpack<DT>(v, x);
            fold<E>(m, s0, s1, x);
        }
    }
    if (tail && wave == 0 && lane == 0) {
        u32x4 v = p[nvec];
        float x[E];
        unpack<DT>(v, x);
#pragma unroll
        for (int j = 0; j < E; ++j)
            if (j >= tail) x[j] = -INFINITY;
        fold<E>(m, s0, s1, x);
    }
    float s = s0 + s1;
    wave_merge(m, s);
    if (lane == 0) {
        s_m[wave] = m;
        s_s[wave] = s;
    }
    __syncthreads();
    if (threadIdx.x == 0) {  // wave 0's state, then waves 1, 2, ... in order
        for (int w = 1; w < kSplitWaves; ++w) merge(m, s, s_m[w], s_s[w]);
        write_row<DT>(a, row, p, m, s, out);
    }
}

// Exact reverse KL in the same pass: one wavefront per token streams the teacher
// and the student row together.  With p_S(v) = exp(s_v - LSE_S),
//   KL(pi_S || pi_T) = sum_v p_S(v) (s_v - t_v) - LSE_S + LSE_T
//                    = A / Z_S - LSE_S + LSE_T,  A = sum_v exp(s_v - m_S) (s_v - t_v),
// and A rescales with the student's running maximum exactly like Z_S.
template <int N>
__device__ __forceinline__ void fold_pair(float &mt, float &zt, float &ms, float &zs, float &am,
                                          const float *t, const float *x) {
    float ct = t[0], cs = x[0];
#pragma unroll
    for (int i = 1; i < N; ++i) {
        ct = fmaxf(ct, t[i]);
        cs = fmaxf(cs, x[i]);
    }
    const float mtn = fmaxf(mt, ct), msn = fmaxf(ms, cs);
    const float rt = (mtn == -INFINITY) ? 0.0f : mtn;
    const float rs = (msn == -INFINITY) ? 0.0f : msn;
    zt *= fast_exp2((mt - rt) * kLog2e);
    const float ss = fast_exp2((ms - rs) * kLog2e);
    zs *= ss;
    am *= ss;
    const float rtl = rt * kLog2e, rsl = rs * kLog2e;
#pragma unroll
    for (int i = 0; i < N; ++i) {
        zt += fast_exp2(__builtin_fmaf(t[i], kLog2e, -rtl));
        const float e = fast_exp2(__builtin_fmaf(x[i], kLog2e, -rsl));
        zs += e;
        // an entry with no student mass adds nothing, even where t - s is infinite
        if (e > 0.0f) am = __builtin_fmaf(e, x[i] - t[i], am);
    }
    mt = mtn;
    ms = msn;
}

struct PairArgs {
    PtrTable teachers;
    const void *student;
    const uint8_t *row_dom;
    const int32_t *ids;
    float *logp_t;
    float *logp_s;
    float *kl_full;
    uint32_t *flags;
    int64_t n_rows;
    int64_t ld;
    int32_t vocab;
    int32_t n_teachers;
};

// Merge two (max, sum) states of the teacher row and two of the student row, with the
// student's A rescaled like its sum.
__device__ __forceinline__ void pair_merge(float &mt, float &zt, float &ms, float &zs, float &am,
                                           float mt2, float zt2, float ms2, float zs2, float am2) {
    merge(mt, zt, mt2, zt2);
    const float mn = fmaxf(ms, ms2);
    const float ref = (mn == -INFINITY) ? 0.0f : mn;
    const float f1 = fast_exp2((ms - ref) * kLog2e), f2 = fast_exp2((ms2 - ref) * kLog2e);
    zs = zs * f1 + zs2 * f2;
    am = am * f1 + am2 * f2;
    ms = mn;
}

// The 64 lane states of a wavefront merged by a fixed butterfly of cross-lane shuffles.
__device__ __forceinline__ void pair_wave_merge(float &mt, float &zt, float &ms, float &zs, float &am) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        const float mt2 = __shfl_xor(mt, o, kWave), zt2 = __shfl_xor(zt, o, kWave);
        const float ms2 = __shfl_xor(ms, o, kWave), zs2 = __shfl_xor(zs, o, kWave);
        const float am2 = __shfl_xor(am, o, kWave);
        pair_merge(mt, zt, ms, zs, am, mt2, zt2, ms2, zs2, am2);
    }
}

// The token's exact KL and both sampled-token log-probabilities from the merged states.
template <int DT>
__device__ __forceinline__ void write_pair(const PairArgs &a, int64_t row, const u32x4 *pt,
                                           const u32x4 *ps, float mt, float zt, float ms, float zs,
                                           float am) {
    const int32_t y = a.ids[row];
    uint32_t bad = 0;
    const bool fin_t = (mt > -INFINITY) && (mt < INFINITY) && (zt > 0.0f) && (zt < INFINITY);
    const bool fin_s = (ms > -INFINITY) && (ms < INFINITY) && (zs > 0.0f) && (zs < INFINITY);
    if (!fin_t || !fin_s) bad |= STRIDE_FLAG_NONFINITE;
    const float lt = __builtin_amdgcn_logf(zt) * kLn2, ls = __builtin_amdgcn_logf(zs) * kLn2;
    // sum_v p_S (log p_S - log p_T) = A/Z_S - (m_S + log Z_S) + (m_T + log Z_T)
    // +inf when the teacher gives no mass where the student has some
    float kl = bad ? __builtin_nanf("") : (am / zs - (ms - mt)) - (ls - lt);
    if (!(kl == kl)) bad |= STRIDE_FLAG_NONFINITE;
    // KL >= 0 (Gibbs); when the two rows differ by a constant the fp32 terms cancel to a
    // rounding residue of either sign, and clamping only reduces that error (NaN stays NaN)
    if (kl < 0.0f) kl = 0.0f;
    a.kl_full[row] = kl;
    if (y < 0 || y >= a.vocab) bad |= STRIDE_FLAG_TOKEN_OOB;
    float rt, rs;
    if (bad & (STRIDE_FLAG_TOKEN_OOB | (fin_t && fin_s ? 0u : STRIDE_FLAG_NONFINITE))) {
        rt = rs = __builtin_nanf("");
    } else {
        float xt, xs;
        if (DT == STRIDE_BF16) {
            xt = __uint_as_float((uint32_t)(reinterpret_cast<const uint16_t *>(pt)[y]) << 16);
            xs = __uint_as_float((uint32_t)(reinterpret_cast<const uint16_t *>(ps)[y]) << 16);
        } else {
            xt = reinterpret_cast<const float *>(pt)[y];
            xs = reinterpret_cast<const float *>(ps)[y];
        }
        rt = fminf((xt - mt) - lt, 0.0f);  // at most 0, as in score_rows_kernel
        rs = fminf((xs - ms) - ls, 0.0f);
    }
    if (bad) raise_flag(a.flags, bad);
    a.logp_t[row] = rt;
    a.logp_s[row] = rs;
}

template <int DT, int U>
__global__ __launch_bounds__(256) void score_pairs_kernel(PairArgs a) {
    constexpr int E = Elem<DT>::kPerVec;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t row = (int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave);
    if (row >= a.n_rows) return;
    const int d = a.row_dom ? (int)a.row_dom[row] : 0;
    if (d >= a.n_teachers) {
        if (lane == 0) {
            a.logp_t[row] = __builtin_nanf("");
            a.kl_full[row] = __builtin_nanf("");
            a.logp_s[row] = __builtin_nanf("");
        }
        return;
    }
    const size_t off = (size_t)row * a.ld * Elem<DT>::kSize;
    const u32x4 *pt = reinterpret_cast<const u32x4 *>(static_cast<const char *>(a.teachers.p[d]) + off);
    const u32x4 *ps = reinterpret_cast<const u32x4 *>(static_cast<const char *>(a.student) + off);
    const int64_t nvec = a.vocab / E;
    const int tail = a.vocab % E;
    float mt = -INFINITY, zt = 0.0f, ms = -INFINITY, zs = 0.0f, am = 0.0f;
    int64_t k = 0;
    constexpr int64_t kStep = (int64_t)U * kWave;
    for (; k + kStep <= nvec; k += kStep) {
        u32x4 vt[U], vs[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            vt[u] = __builtin_nontemporal_load(pt + k + u * kWave + lane);
            vs[u] = __builtin_nontemporal_load(ps + k + u * kWave + lane);
        }
        float xt[U * E], xs[U * E];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            unpack<DT>(vt[u], xt + u * E);
            unpack<DT>(vs[u], xs + u * E);
        }
        fold_pair<U * E>(mt, zt, ms, zs, am, xt, xs);
    }
    for (; k < nvec; k += kWave) {
        if (k + lane < nvec) {
            float xt[E], xs[E];
            unpack<DT>(__builtin_nontemporal_load(pt + k + lane), xt);
            unpack<DT>(__builtin_nontemporal_load(ps + k + lane), xs);
            fold_pair<E>(mt, zt, ms, zs, am, xt, xs);
        }
    }
    if (tail && lane == 0) {
        float xt[E], xs[E];
        unpack<DT>(pt[nvec], xt);
        unpack<DT>(ps[nvec], xs);
#pragma unroll
        for (int j = 0; j < E; ++j)
            if (j >= tail) {
                xt[j] = -INFINITY;
                xs[j] = -INFINITY;
            }
        fold_pair<E>(mt, zt, ms, zs, am, xt, xs);
    }
    pair_wave_merge(mt, zt, ms, zs, am);
    if (lane == 0) write_pair<DT>(a, row, pt, ps, mt, zt, ms, zs, am);
}

// The paired pass for small batches, as score_rows_split_kernel does for single rows: the
// kSplitWaves wavefronts of a workgroup share one token's teacher and student rows (chunks w,
// w + kSplitWaves, ...) and merge their five-value states in wavefront order through LDS.
template <int DT, int U>
__global__ __launch_bounds__(kSplitWaves *kWave) void score_pairs_split_kernel(PairArgs a) {
    constexpr int E = Elem<DT>::kPerVec;
    __shared__ float s_st[5][kSplitWaves];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t row = blockIdx.x;  // one workgroup per token: the grid has exactly n_rows
    const int d = a.row_dom ? (int)a.row_dom[row] : 0;
    if (d >= a.n_teachers) {  // the same for the whole workgroup: it leaves before any barrier
        if (threadIdx.x == 0) {
            a.logp_t[row] = __builtin_nanf("");
            a.kl_full[row] = __builtin_nanf("");
            a.logp_s[row] = __builtin_nanf("");
        }
        return;
    }
    const size_t off = (size_t)row * a.ld * Elem<DT>::kSize;
    const u32x4 *pt = reinterpret_cast<const u32x4 *>(static_cast<const char *>(a.teachers.p[d]) + off);
    const u32x4 *ps = reinterpret_cast<const u32x4 *>(static_cast<const char *>(a.student) + off);
    const int64_t nvec = a.vocab / E;
    const int tail = a.vocab % E;
    constexpr int64_t kStep = (int64_t)U * kWave;
    const int64_t nfull = nvec / kStep;
    float mt = -INFINITY, zt = 0.0f, ms = -INFINITY, zs = 0.0f, am = 0.0f;
    for (int64_t c = wave; c < nfull; c += kSplitWaves) {
        const int64_t k = c * kStep;
        u32x4 vt[U], vs[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            vt[u] = __builtin_nontemporal_load(pt + k + u * kWave + lane);
            vs[u] = __builtin_nontemporal_load(ps + k + u * kWave + lane);
        }
        float xt[U * E], xs[U * E];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            unpack<DT>(vt[u], xt + u * E);
            unpack<DT>(vs[u], xs + u * E);
        }
        fold_pair<U * E>(mt, zt, ms, zs, am, xt, xs);
    }
    for (int64_t k = nfull * kStep + (int64_t)wave * kWave; k < nvec; k += (int64_t)kSplitWaves * kWave) {
        if (k + lane < nvec) {
            float xt[E], xs[E];
            unpack<DT>(__builtin_nontemporal_load(pt + k + lane), xt);
            unpack<DT>(__builtin_nontemporal_load(ps + k + lane), xs);
            fold_pair<E>(mt, zt, ms, zs, am, xt, xs);
        }
    }
    if (tail && wave == 0 && lane == 0) {
        float xt[E], xs[E];
        unpack<DT>(pt[nvec], xt);
        unpack<DT>(ps[nvec], xs);
#pragma unroll
        for (int j = 0; j < E; ++j)
            if (j >= tail) {
                xt[j] = -INFINITY;
                xs[j] = -INFINITY;
            }
        fold_pair<E>(mt, zt, ms, zs, am, xt, xs);
    }
    pair_wave_merge(mt, zt, ms, zs, am);
    if (lane == 0) {
        s_st[0][wave] = mt;
        s_st[1][wave] = zt;
        s_st[2][wave] = ms;
        s_st[3][wave] = zs;
        s_st[4][wave] = am;
    }
    __syncthreads();
    if (threadIdx.x == 0) {  // wave 0's state, then waves 1, 2, ... in order
        for (int w = 1; w < kSplitWaves; ++w)
            pair_merge(mt, zt, ms, zs, am, s_st[0][w], s_st[1][w], s_st[2][w], s_st[3][w], s_st[4][w]);
        write_pair<DT>(a, row, pt, ps, mt, zt, ms, zs, am);
    }
}

// Teacher index of every row: row -> turn (by offsets) -> rollout -> domain.
// Rows outside every turn, or whose rollout's domain is out of range, get
// kBadDomain and raise a flag, so the scoring kernel writes NaN for them.
__global__ __launch_bounds__(256) void row_domain_kernel(stride_layout L, int32_t n_teachers,
                                                         uint8_t *row_dom, uint32_t *flags) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= L.n_tokens) return;
    // last turn t with turn_tok_off[t] <= i
    int64_t lo = 0, hi = L.n_turns;  // answer in [0, T)
    if (L.n_turns == 0 || L.turn_tok_off[0] > i) {
        row_dom[i] = kBadDomain;
        raise_flag(flags, STRIDE_FLAG_BAD_OFFSETS);
        return;
    }
    while (hi - lo > 1) {
        const int64_t mid = (lo + hi) >> 1;
        if (L.turn_tok_off[mid] <= i) lo = mid; else hi = mid;
    }
    const int64_t t = lo;
    if (i >= L.turn_tok_off[t + 1]) {
        row_dom[i] = kBadDomain;
        raise_flag(flags, STRIDE_FLAG_BAD_OFFSETS);
        return;
    }
    int64_t rlo = 0, rhi = L.n_rollouts;
    if (L.n_rollouts == 0 || L.rollout_turn_off[0] > t) {
        row_dom[i] = kBadDomain;
        raise_flag(flags, STRIDE_FLAG_BAD_OFFSETS);
        return;
    }
    while (rhi - rlo > 1) {
        const int64_t mid = (rlo + rhi) >> 1;
        if (L.rollout_turn_off[mid] <= t) rlo = mid; else rhi = mid;
    }
    if (t >= L.rollout_turn_off[rlo + 1]) {
        row_dom[i] = kBadDomain;
        raise_flag(flags, STRIDE_FLAG_BAD_OFFSETS);
        return;
    }
    const int32_t d = L.domain ? L.domain[rlo] : 0;
    if (d < 0 || d >= n_teachers) {
        row_dom[i] = kBadDomain;
        raise_flag(flags, STRIDE_FLAG_BAD_DOMAIN);
        return;
    }
    row_dom[i] = (uint8_t)d;
}

}  // namespace

hipError_t launch_score_pairs(int32_t dtype, const PtrTable &teachers, int32_t n_teachers,
                              const uint8_t *row_dom, const void *student, const int32_t *ids,
                              float *logp_t, float *logp_s, float *kl_full, int64_t n_rows,
                              int32_t vocab, int64_t ld, uint32_t *flags, hipStream_t stream) {
    if (n_rows == 0) return hipSuccess;
    PairArgs a;
    a.teachers = teachers;
    a.student = student;
    a.row_dom = row_dom;
    a.ids = ids;
    a.logp_t = logp_t;
    a.logp_s = logp_s;
    a.kl_full = kl_full;
    a.flags = flags;
    a.n_rows = n_rows;
    a.ld = ld;
    a.vocab = vocab;
    a.n_teachers = n_teachers;
    if (n_rows < kPairSplitBelow) {
        if (dtype == STRIDE_BF16)
            hipLaunchKernelGGL((score_pairs_split_kernel<STRIDE_BF16, 4>), dim3((unsigned)n_rows),
                               dim3(kSplitWaves * kWave), 0, stream, a);
        else
            hipLaunchKernelGGL((score_pairs_split_kernel<STRIDE_F32, 4>), dim3((unsigned)n_rows),
                               dim3(kSplitWaves * kWave), 0, stream, a);
        return hipGetLastError();
    }
    const int64_t blocks = (n_rows + 3) / 4;
    if (dtype == STRIDE_BF16)
        hipLaunchKernelGGL((score_pairs_kernel<STRIDE_BF16, 4>), dim3((unsigned)blocks), dim3(256), 0,
                           stream, a);
    else
        hipLaunchKernelGGL((score_pairs_kernel<STRIDE_F32, 4>), dim3((unsigned)blocks), dim3(256), 0,
                           stream, a);
    return hipGetLastError();
}

hipError_t launch_row_domain(const stride_layout &L, int32_t n_teachers, uint8_t *row_dom,
                             uint32_t *flags, hipStream_t stream) {
    if (L.n_tokens == 0) return hipSuccess;
    const int64_t blocks = (L.n_tokens + 255) / 256;
    hipLaunchKernelGGL(row_domain_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, L,
                       n_teachers, row_dom, flags);
    return hipGetLastError();
}

hipError_t launch_score_rows(int32_t dtype, const PtrTable &teachers, int32_t n_teachers,
                             const uint8_t *row_dom, const void *student, const int32_t *ids,
                             float *logp_t, float *logp_s, int64_t n_rows, int32_t vocab,
                             int64_t ld, uint32_t *flags, hipStream_t stream) {
    if (n_rows == 0) return hipSuccess;
    ScoreArgs a;
    a.teachers = teachers;
    a.student = student;
    a.row_dom = row_dom;
    a.ids = ids;
    a.logp_t = logp_t;
    a.logp_s = logp_s;
    a.flags = flags;
    a.n_rows = n_rows;
    a.ld = ld;
    a.vocab = vocab;
    a.n_teachers = n_teachers;
    const int64_t items = student ? 2 * n_rows : n_rows;
    if (items < kSplitBelow) {
        if (dtype == STRIDE_BF16)
            hipLaunchKernelGGL((score_rows_split_kernel<STRIDE_BF16, 8>), dim3((unsigned)items),
                               dim3(kSplitWaves * kWave), 0, stream, a);
        else
            hipLaunchKernelGGL((score_rows_split_kernel<STRIDE_F32, 8>), dim3((unsigned)items),
                               dim3(kSplitWaves * kWave), 0, stream, a);
        return hipGetLastError();
    }
    constexpr int kRowsPerBlock = kRowThreads / kWave;
    const int64_t blocks = (items + kRowsPerBlock - 1) / kRowsPerBlock;
    if (dtype == STRIDE_BF16)
        hipLaunchKernelGGL((score_rows_kernel<STRIDE_BF16, 8>), dim3((unsigned)blocks), dim3(kRowThreads),
                           0, stream, a);
    else
        hipLaunchKernelGGL((score_rows_kernel<STRIDE_F32, 8>), dim3((unsigned)blocks), dim3(kRowThreads),
                           0, stream, a);
    return hipGetLastError();
}

}  // namespace stride
