/*
 * oracle.c -- plain float64 CPU oracle for the STRIDE scoring, early-stop and
 * restart path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may load, link or
 * call this file: only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no code, header, table or constant with the HIP
 * library; the only thing both sides consume is the seeded input generator.
 *
 * Paper: "Know When to Stop, Where to Restart: Accelerating Multi-Turn
 * Agentic On-Policy Distillation" (STRIDE).  Every function below cites the
 * passage it follows.  Arithmetic is IEEE binary64 with libm exp/log, summed
 * sequentially in index order; OpenMP only splits independent rows.
 *
 * Readings of points the paper leaves open (recorded with each function):
 *   - An out-of-range token id or a non-finite row gives NaN outputs.
 *   - An empty turn has no mean: NaN.
 *   - No crossing of the threshold: stop = -1, the whole rollout is kept.
 *   - Empty leading correct run (K_max = 0): k* = -1 and K0 = 0, which is the
 *     branch Algorithm 1 takes for a task without a usable record.
 *   - argmin ties go to the lowest index.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { OR_BF16 = 0, OR_F32 = 1, OR_F64 = 2 };
enum { OR_TOKEN_OOB = 1, OR_EMPTY_TURN = 2, OR_NONFINITE = 8 };

/* A bf16 value is the upper half of an IEEE binary32: widening is exact. */
static double bf16_bits_to_double(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static double load_logit(const void *base, int dtype, int64_t idx) {
    if (dtype == OR_BF16) return bf16_bits_to_double(((const uint16_t *)base)[idx]);
    if (dtype == OR_F32) return (double)((const float *)base)[idx];
    return ((const double *)base)[idx];
}

static int64_t elem_size(int dtype) {
    return dtype == OR_BF16 ? 2 : (dtype == OR_F32 ? 4 : 8);
}

/*
 * Log-normaliser of one row of logits, lse = log sum_v exp(x_v), returned as
 * its two parts: m = max_v x_v and log_s = log sum_v exp(x_v - m), so that
 * lse = m + log_s.  The model's next-token distribution is the softmax of the
 * row, hence log pi(v) = (x_v - m) - log_s; this is the log-probability that
 * enters r_t in Eq. (1) (Sec. 3.1), for the teacher and for the student.
 * Keeping m apart avoids losing log_s next to a large common offset.  Returns
 * 0 and NaN parts for a row holding NaN or +inf, or whose entries are all
 * -inf (no probability mass); 1 otherwise.
 */
static int row_lse(const void *row, int dtype, int64_t vocab, double *m_out, double *log_s_out) {
    double m = -INFINITY;
    *m_out = NAN;
    *log_s_out = NAN;
    for (int64_t v = 0; v < vocab; ++v) {
        double x = load_logit(row, dtype, v);
        if (isnan(x) || x == INFINITY) return 0;
        if (x > m) m = x;
    }
    if (m == -INFINITY) return 0;
    double s = 0.0;
    for (int64_t v = 0; v < vocab; ++v) s += exp(load_logit(row, dtype, v) - m);
    *m_out = m;
    *log_s_out = log(s);
    return 1;
}

/*
 * Sampled-token log-probabilities of n_rows rows (row i at logits + i*ld
 * elements): logp[i] = (x_i[y] - m_i) - log_s_i with y = ids[i], as in row_lse.
 * Eq. (1) (Sec. 3.1): log pi(y_t | y_<t) for the token y_t the student
 * sampled.  lse may be NULL.  Returns the OR of OR_TOKEN_OOB / OR_NONFINITE
 * over the rows; an affected row's logp is NaN.
 */
int oracle_logp_rows(int64_t n_rows, int64_t vocab, int64_t ld, int dtype,
                     const void *logits, const int32_t *ids, double *logp, double *lse) {
    int flags = 0;
    const char *base = (const char *)logits;
    int64_t es = elem_size(dtype);
#pragma omp parallel for schedule(dynamic, 4) reduction(| : flags)
    for (int64_t i = 0; i < n_rows; ++i) {
        const void *row = base + i * ld * es;
        double m, log_s;
        if (!row_lse(row, dtype, vocab, &m, &log_s)) flags |= OR_NONFINITE;
        int32_t y = ids[i];
        double lp;
        if (y < 0 || (int64_t)y >= vocab) {
            flags |= OR_TOKEN_OOB;
            lp = NAN;
        } else {
            lp = (load_logit(row, dtype, y) - m) - log_s;
        }
        logp[i] = lp;
        if (lse) lse[i] = m + log_s;
    }
    return flags;
}

/*
 * Per-token signals of Sec. 3.1-3.2 from the two sampled-token
 * log-probabilities: the OPD reward r_t = log pi_T - log pi_theta (Eq. 1) and
 * each token's KL estimate between student and teacher, log pi_theta - log pi_T = -r_t
 * (Sec. 3.2, analysis set-up).  kl may alias neither input.
 */
void oracle_token_kl(int64_t n, const double *logp_s, const double *logp_t, double *kl) {
    for (int64_t i = 0; i < n; ++i) kl[i] = logp_s[i] - logp_t[i];
}

/*
 * Exact full-vocabulary reverse KL per row, KL(pi_S || pi_T) =
 * sum_v p_S(v) (log p_S(v) - log p_T(v)): the divergence whose sequence-level
 * form OPD minimises (Sec. 3.1, following MiniLLM).  The sampled-token value
 * above is an unbiased one-sample estimate of it under pi_S.  NaN if either
 * row is non-finite.
 */
void oracle_exact_kl(int64_t n_rows, int64_t vocab, int64_t ld, int dtype,
                     const void *teacher, const void *student, double *out) {
    const char *tb = (const char *)teacher, *sb = (const char *)student;
    int64_t es = elem_size(dtype);
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t i = 0; i < n_rows; ++i) {
        const void *tr = tb + i * ld * es, *sr = sb + i * ld * es;
        double mt, lst, ms, lss;
        if (!row_lse(tr, dtype, vocab, &mt, &lst) || !row_lse(sr, dtype, vocab, &ms, &lss)) {
            out[i] = NAN;
            continue;
        }
        double acc = 0.0;
        for (int64_t v = 0; v < vocab; ++v) {
            double lps = (load_logit(sr, dtype, v) - ms) - lss;
            double lpt = (load_logit(tr, dtype, v) - mt) - lst;
            double ps = exp(lps);
            if (ps > 0.0) acc += ps * (lps - lpt);
        }
        out[i] = acc;
    }
}

/*
 * Mean teacher log-probability of each turn, Eq. (4) (Sec. 3.1): for turn k with
 * tokens [turn_tok_off[k], turn_tok_off[k+1]), lbar_k = (1/n_k) sum_i
 * logp_t[i].  An empty turn (n_k = 0) has no mean: NaN and OR_EMPTY_TURN.
 * Offsets that decrease also give NaN and OR_EMPTY_TURN.
 */
int oracle_turn_mean(int64_t n_turns, const int64_t *turn_tok_off, const double *logp_t,
                     double *out) {
    int flags = 0;
    for (int64_t k = 0; k < n_turns; ++k) {
        int64_t a = turn_tok_off[k], b = turn_tok_off[k + 1];
        if (b <= a) { out[k] = NAN; flags |= OR_EMPTY_TURN; continue; }
        double s = 0.0;
        for (int64_t i = a; i < b; ++i) s += logp_t[i];
        out[k] = s / (double)(b - a);
    }
    return flags;
}

/*
 * Early-stop test, Eq. (5) (Sec. 4.1) with the prefix-buffer offset of
 * Sec. 4.1 (its paragraph on combining the stop with the prefix buffer) and
 * Algorithm 1's inner loop.
 *
 * Rollout r owns units [unit_off[r], unit_off[r+1]); a unit is a turn (value =
 * lbar_k, the paper's rule) or a token (value = teacher log-prob, the
 * single-turn variant of Sec. 5.5).  Units before the reused prefix length
 * K0 = start[r] are excluded: C_u = sum_{j=K0}^{u} value_j for local index
 * u >= K0, and cum = 0 for u < K0.  stop[r] is the first local u >= K0 with
 * C_u < lambda[r] (strict), else -1; the triggering unit is retained for the
 * loss.  retained[r] counts the tokens of the newly generated, retained units
 * [K0, stop] (or [K0, end) without a stop), with unit u covering tokens
 * [unit_tok_off[g], unit_tok_off[g+1]) for global unit g.  start may be NULL
 * (all 0); retained and unit_tok_off may be NULL.
 */
void oracle_stop(int64_t n_roll, const int64_t *unit_off, const double *values,
                 const double *lambda, const int32_t *start, const int64_t *unit_tok_off,
                 double *cum, int32_t *stop, int64_t *retained) {
    for (int64_t r = 0; r < n_roll; ++r) {
        int64_t first = unit_off[r], n = unit_off[r + 1] - unit_off[r];
        int64_t k0 = start ? start[r] : 0;
        if (k0 < 0) k0 = 0;
        if (k0 > n) k0 = n;
        double c = 0.0;
        int32_t s = -1;
        for (int64_t u = 0; u < n; ++u) {
            if (u < k0) { cum[first + u] = 0.0; continue; }
            c += values[first + u];
            cum[first + u] = c;
            if (s < 0 && c < lambda[r]) s = (int32_t)u;
        }
        stop[r] = s;
        if (retained && unit_tok_off) {
            int64_t end = (s >= 0) ? (int64_t)s + 1 : n;
            retained[r] = unit_tok_off[first + end] - unit_tok_off[first + k0];
        }
    }
}

/*
 * Prefix-buffer restart pick, Sec. 4.2 steps 1-3, Eq. (6) and Algorithm 1.
 *
 * The record of rollout r is its first record_len[r] units (the units that
 * were generated: up to and including a stop, Algorithm 1), or all units if
 * record_len is NULL.  Unit u is correct iff mask[u] != 0 (mask NULL: all
 * set) and value_u > alpha[r] (strict; step 1).  K_max is the length of the
 * leading run of correct units, counted from unit 0 up to the first unit
 * that is not correct (step 2).  k* is the lowest index u < K_max attaining min value_u (Eq. 6,
 * 0-based), -1 if K_max = 0.  K0 = max(k*, 0): the next rollout reuses
 * units 0..k*-1 as context and resamples from k* (step 3), and a task without
 * a usable prefix starts from 0.  k_max may be NULL.
 */
void oracle_restart(int64_t n_roll, const int64_t *unit_off, const double *values,
                    const int32_t *record_len, const double *alpha, const uint8_t *mask,
                    int32_t *k_star, int32_t *k0, int32_t *k_max) {
    for (int64_t r = 0; r < n_roll; ++r) {
        int64_t first = unit_off[r], n = unit_off[r + 1] - unit_off[r];
        int64_t len = record_len ? record_len[r] : n;
        if (len < 0) len = 0;
        if (len > n) len = n;
        int64_t km = 0;
        while (km < len) {
            int64_t g = first + km;
            int ok = (mask == NULL || mask[g] != 0) && (values[g] > alpha[r]);
            if (!ok) break;
            ++km;
        }
        int32_t best = -1;
        for (int64_t u = 0; u < km; ++u) {
            if (best < 0 || values[first + u] < values[first + best]) best = (int32_t)u;
        }
        k_star[r] = best;
        k0[r] = best > 0 ? best : 0;
        if (k_max) k_max[r] = (int32_t)km;
    }
}

/*
 * Teacher log-probabilities when the teacher's logits come from its output
 * projection: z = h W with h the final hidden state of the row (bf16, [d])
 * and W the lm_head ([d, vocab] bf16, row-major), then the same log-softmax
 * at the sampled token as oracle_logp_rows (Eq. 1).  z is formed in binary64
 * (each bf16 x bf16 product is exact there) and is not rounded to bf16.
 */
int oracle_fused_logp(int64_t n_rows, int64_t d, int64_t vocab, const uint16_t *hidden,
                      const uint16_t *w, const int32_t *ids, double *logp, double *lse) {
    int flags = 0;
#pragma omp parallel reduction(| : flags)
    {
        double *z = (double *)malloc((size_t)(vocab > 0 ? vocab : 1) * sizeof(double));
#pragma omp for schedule(dynamic, 1)
        for (int64_t i = 0; i < n_rows; ++i) {
            for (int64_t v = 0; v < vocab; ++v) z[v] = 0.0;
            for (int64_t k = 0; k < d; ++k) {
                double h = bf16_bits_to_double(hidden[i * d + k]);
                const uint16_t *wrow = w + k * vocab;
                for (int64_t v = 0; v < vocab; ++v) z[v] += h * bf16_bits_to_double(wrow[v]);
            }
            double m, log_s;
            if (!row_lse(z, OR_F64, vocab, &m, &log_s)) flags |= OR_NONFINITE;
            int32_t y = ids[i];
            double lp;
            if (y < 0 || (int64_t)y >= vocab) {
                flags |= OR_TOKEN_OOB;
                lp = NAN;
            } else {
                lp = (z[y] - m) - log_s;
            }
            logp[i] = lp;
            if (lse) lse[i] = m + log_s;
        }
        free(z);
    }
    return flags;
}

/*
 * Token-level OPD loss and its gradient with respect to the student's logits,
 * Eq. (2) (Sec. 3.1): L = -scale * sum_t mask_t r_t log pi_S(y_t), where r_t
 * (Eq. 1, passed in) is held constant and mask_t marks the trainable rows.
 * Differentiating the log-softmax, d log pi_S(y) / d s_v = [v = y] - pi_S(v),
 * so grad[t, v] = -scale mask_t r_t ([v = y_t] - pi_S(v)) and
 * loss[t] = -scale mask_t r_t log pi_S(y_t).  pi_S is recomputed from the
 * row itself.  grad is [n_rows, vocab] (dense, no padding); rows with
 * mask 0 are all zero.  Returns the OR of flags as oracle_logp_rows.
 */
int oracle_opd_grad(int64_t n_rows, int64_t vocab, int64_t ld, int dtype, const void *student,
                    const int32_t *ids, const double *r, const uint8_t *mask, double scale,
                    double *grad, double *loss) {
    int flags = 0;
    const char *base = (const char *)student;
    int64_t es = elem_size(dtype);
#pragma omp parallel for schedule(dynamic, 4) reduction(| : flags)
    for (int64_t i = 0; i < n_rows; ++i) {
        double *g = grad + i * vocab;
        if (!mask[i]) {
            for (int64_t v = 0; v < vocab; ++v) g[v] = 0.0;
            loss[i] = 0.0;
            continue;
        }
        const void *row = base + i * ld * es;
        double m, log_s;
        int ok = row_lse(row, dtype, vocab, &m, &log_s);
        int32_t y = ids[i];
        if (!ok) flags |= OR_NONFINITE;
        if (y < 0 || (int64_t)y >= vocab) {
            flags |= OR_TOKEN_OOB;
            ok = 0;
        }
        if (!ok) {
            for (int64_t v = 0; v < vocab; ++v) g[v] = NAN;
            loss[i] = NAN;
            continue;
        }
        double c = -scale * r[i];
        for (int64_t v = 0; v < vocab; ++v) {
            double p = exp((load_logit(row, dtype, v) - m) - log_s);
            g[v] = c * (((int64_t)y == v ? 1.0 : 0.0) - p);
        }
        loss[i] = c * ((load_logit(row, dtype, y) - m) - log_s);
    }
    return flags;
}
