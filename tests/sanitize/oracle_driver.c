/*
 * Every entry point of the float64 oracle on small inputs, for a build with
 * AddressSanitizer and UndefinedBehaviorSanitizer: ragged and padded rows in
 * bf16, fp32 and fp64, empty and non-increasing turns, rollouts with no units,
 * out-of-range token ids, NaN / +inf / all -inf rows, start offsets past the
 * record, and NULL optional outputs.  Each buffer is allocated at exactly the
 * size the call may touch, so any read or write past it is reported.  The
 * values are only sanity-checked here; correctness is pinned elsewhere.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_logp_rows(int64_t n_rows, int64_t vocab, int64_t ld, int dtype, const void *logits,
                     const int32_t *ids, double *logp, double *lse);
void oracle_token_kl(int64_t n, const double *logp_s, const double *logp_t, double *kl);
void oracle_exact_kl(int64_t n_rows, int64_t vocab, int64_t ld, int dtype, const void *teacher,
                     const void *student, double *out);
int oracle_turn_mean(int64_t n_turns, const int64_t *turn_tok_off, const double *logp_t,
                     double *out);
void oracle_stop(int64_t n_roll, const int64_t *unit_off, const double *values,
                 const double *lambda, const int32_t *start, const int64_t *unit_tok_off,
                 double *cum, int32_t *stop, int64_t *retained);
void oracle_restart(int64_t n_roll, const int64_t *unit_off, const double *values,
                    const int32_t *record_len, const double *alpha, const uint8_t *mask,
                    int32_t *k_star, int32_t *k0, int32_t *k_max);
int oracle_fused_logp(int64_t n_rows, int64_t d, int64_t vocab, const uint16_t *hidden,
                      const uint16_t *w, const int32_t *ids, double *logp, double *lse);
int oracle_opd_grad(int64_t n_rows, int64_t vocab, int64_t ld, int dtype, const void *student,
                    const int32_t *ids, const double *r, const uint8_t *mask, double scale,
                    double *grad, double *loss);

static uint64_t state = 0x9E3779B97F4A7C15ull;
static double unif(void) { /* xorshift64*, in [0, 1) */
    state ^= state >> 12;
    state ^= state << 25;
    state ^= state >> 27;
    return (double)((state * 0x2545F4914F6CDD1Dull) >> 11) / 9007199254740992.0;
}

static void *exact(size_t bytes) { return malloc(bytes ? bytes : 1); }

static uint16_t to_bf16(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);
}

/* n_rows rows of `vocab` logits with row stride ld in the given dtype (0 bf16, 1 fp32, 2 fp64);
 * the buffer ends right after the last row's ld elements. */
static void *rows(int64_t n_rows, int64_t vocab, int64_t ld, int dtype) {
    const int64_t es = dtype == 0 ? 2 : (dtype == 1 ? 4 : 8);
    char *p = exact((size_t)(n_rows * ld * es));
    for (int64_t i = 0; i < n_rows; ++i)
        for (int64_t v = 0; v < ld; ++v) {
            const double x = v < vocab ? 4.0 * unif() - 2.0 : 1e30; /* padding must be ignored */
            char *q = p + (i * ld + v) * es;
            if (dtype == 0) { uint16_t b = to_bf16((float)x); memcpy(q, &b, 2); }
            else if (dtype == 1) { float f = (float)x; memcpy(q, &f, 4); }
            else memcpy(q, &x, 8);
        }
    return p;
}

static void poison_row(void *p, int64_t row, int64_t ld, int dtype, int kind) {
    const int64_t es = dtype == 0 ? 2 : (dtype == 1 ? 4 : 8);
    const double x = kind == 0 ? NAN : (kind == 1 ? INFINITY : -INFINITY);
    for (int64_t v = 0; v < (kind == 2 ? ld : 1); ++v) {
        char *q = (char *)p + (row * ld + v) * es;
        if (dtype == 0) { uint16_t b = to_bf16((float)x); memcpy(q, &b, 2); }
        else if (dtype == 1) { float f = (float)x; memcpy(q, &f, 4); }
        else memcpy(q, &x, 8);
    }
}

static int checks = 0;
#define EXPECT(c) do { ++checks; if (!(c)) { fprintf(stderr, "expectation failed at line %d: %s\n", __LINE__, #c); exit(2); } } while (0)

static void scoring(void) {
    const int64_t shapes[][3] = {{1, 1, 8}, {7, 9, 16}, {13, 1000, 1000}, {5, 257, 264}, {0, 10, 16}};
    for (int dt = 0; dt < 3; ++dt)
        for (size_t s = 0; s < sizeof shapes / sizeof shapes[0]; ++s) {
            const int64_t n = shapes[s][0], V = shapes[s][1], ld = shapes[s][2];
            void *t = rows(n, V, ld, dt), *st = rows(n, V, ld, dt);
            int32_t *ids = exact(sizeof(int32_t) * (size_t)n);
            for (int64_t i = 0; i < n; ++i) ids[i] = (int32_t)(unif() * (double)V);
            if (n >= 5) {
                ids[1] = -1;
                ids[2] = (int32_t)V;
                poison_row(t, 3, ld, dt, 0);
                poison_row(st, 4, ld, dt, 1);
                poison_row(t, 0, ld, dt, 2);
            }
            double *lt = exact(8 * (size_t)n), *ls = exact(8 * (size_t)n), *lse = exact(8 * (size_t)n),
                   *kl = exact(8 * (size_t)n), *kf = exact(8 * (size_t)n);
            const int ft = oracle_logp_rows(n, V, ld, dt, t, ids, lt, lse);
            const int fs = oracle_logp_rows(n, V, ld, dt, st, ids, ls, NULL);
            oracle_token_kl(n, ls, lt, kl);
            oracle_exact_kl(n, V, ld, dt, t, st, kf);
            if (n >= 5) {
                EXPECT(ft & 1);
                EXPECT(ft & 8);
                EXPECT(fs & 8);
                EXPECT(isnan(lt[1]) && isnan(lt[2]) && isnan(lt[3]) && isnan(lt[0]));
            } else {
                EXPECT(ft == 0 && fs == 0);
                for (int64_t i = 0; i < n; ++i) EXPECT(lt[i] <= 1e-12 && kf[i] >= -1e-12);
            }
            free(t); free(st); free(ids); free(lt); free(ls); free(lse); free(kl); free(kf);
        }
}

static void turns_stop_restart(void) {
    /* three rollouts: 4 turns, 0 turns, 3 turns (one of them empty, one with decreasing offsets) */
    const int64_t turn_tok_off[8] = {0, 3, 5, 5, 9, 12, 11, 14};
    double *logp = exact(8 * 14);
    for (int i = 0; i < 14; ++i) logp[i] = -3.0 * unif();
    double *tm = exact(8 * 7);
    const int f = oracle_turn_mean(7, turn_tok_off, logp, tm);
    EXPECT(f & 2);
    EXPECT(isnan(tm[2]) && isnan(tm[5]) && !isnan(tm[0]));
    EXPECT(oracle_turn_mean(0, turn_tok_off, logp, tm) == 0);

    const int64_t unit_off[4] = {0, 4, 4, 7};
    const int64_t unit_tok_off[8] = {0, 3, 5, 5, 9, 9, 11, 14};
    double vals[7] = {-1, -2, -0.5, -3, -1, -1, -1};
    const double lam[3] = {-3.2, -1e300, INFINITY};
    const int32_t start[3] = {1, 0, 9};  /* the third starts past its record */
    double *cum = exact(8 * 7);
    int32_t *stop = exact(4 * 3);
    int64_t *ret = exact(8 * 3);
    for (int k = 0; k < 3; ++k) {  /* one threshold per rollout */
        double *l3 = exact(8 * 3);
        for (int r = 0; r < 3; ++r) l3[r] = lam[(k + r) % 3];
        oracle_stop(3, unit_off, vals, l3, start, unit_tok_off, cum, stop, ret);
        EXPECT(stop[1] == -1 && ret[1] == 0 && ret[2] == 0);
        oracle_stop(3, unit_off, vals, l3, NULL, NULL, cum, stop, NULL);
        free(l3);
    }
    const int32_t rec[3] = {4, 0, 2};
    const uint8_t mask[7] = {1, 1, 0, 1, 1, 1, 1};
    int32_t *ks = exact(4 * 3), *k0 = exact(4 * 3), *km = exact(4 * 3);
    const double al[4] = {-10.0, -1.5, NAN, -INFINITY};
    for (int k = 0; k < 4; ++k) {  /* one threshold per rollout */
        double *a3 = exact(8 * 3);
        for (int r = 0; r < 3; ++r) a3[r] = al[(k + r) % 4];
        oracle_restart(3, unit_off, vals, rec, a3, mask, ks, k0, km);
        EXPECT(ks[1] == -1 && k0[1] == 0 && km[1] == 0);
        oracle_restart(3, unit_off, vals, NULL, a3, NULL, ks, k0, NULL);
        free(a3);
    }
    free(logp); free(tm); free(cum); free(stop); free(ret); free(ks); free(k0); free(km);
}

static void fused_and_grad(void) {
    const int64_t n = 6, d = 64, V = 130;
    uint16_t *h = exact(2 * (size_t)(n * d)), *w = exact(2 * (size_t)(V * d));
    for (int64_t i = 0; i < n * d; ++i) h[i] = to_bf16((float)(2.0 * unif() - 1.0));
    for (int64_t i = 0; i < V * d; ++i) w[i] = to_bf16((float)(0.1 * unif() - 0.05));
    int32_t ids[6] = {0, 129, 5, -1, 130, 64};
    int32_t *idp = exact(sizeof ids);
    memcpy(idp, ids, sizeof ids);
    double *lp = exact(8 * (size_t)n), *lse = exact(8 * (size_t)n);
    const int f = oracle_fused_logp(n, d, V, h, w, idp, lp, lse);
    EXPECT(f & 1);
    EXPECT(isnan(lp[3]) && isnan(lp[4]) && lp[0] <= 0.0);
    EXPECT(oracle_fused_logp(0, d, V, h, w, idp, lp, NULL) == 0);

    for (int dt = 0; dt < 3; ++dt) {
        const int64_t ld = 136;
        void *s = rows(n, V, ld, dt);
        double r[6] = {0.5, -0.25, 1.0, 0.0, 2.0, -1.0};
        double *rp = exact(sizeof r);
        memcpy(rp, r, sizeof r);
        uint8_t mk[6] = {1, 1, 0, 1, 1, 0};
        uint8_t *mp = exact(sizeof mk);
        memcpy(mp, mk, sizeof mk);
        double *g = exact(8 * (size_t)(n * V)), *loss = exact(8 * (size_t)n);  /* dense [n, V] */
        const int fg = oracle_opd_grad(n, V, ld, dt, s, idp, rp, mp, 0.5, g, loss);
        EXPECT(fg & 1);
        EXPECT(loss[2] == 0.0 && g[2 * V] == 0.0 && isnan(loss[3]) && isnan(loss[4]));
        free(s); free(rp); free(mp); free(g); free(loss);
    }
    free(h); free(w); free(idp); free(lp); free(lse);
}

int main(void) {
    scoring();
    turns_stop_restart();
    fused_and_grad();
    printf("oracle driver ok: %d expectations\n", checks);
    return 0;
}
