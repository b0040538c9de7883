// stride_abi.cpp -- the extern "C" entry points of libstride.so.
//
// Host-side argument checking (synchronous, before any launch), workspace
// carving and the launch sequence of each call.  Every launch is asynchronous
// on the caller's stream; nothing here synchronises or allocates.
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "common.hpp"

namespace stride {

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

WsLayout ws_layout(int64_t n_rollouts, int64_t n_tokens, int64_t n_units, int64_t fused_partials) {
    WsLayout w;
    size_t off = 0;
    w.counter = off;
    off += 256;
    w.unit_off = off;
    off += align256(sizeof(int64_t) * (size_t)(n_rollouts + 1));
    w.desc = off;
    const int64_t tiles = n_units > 0 ? (n_units + kScanTile - 1) / kScanTile : 0;
    off += align256(sizeof(TileDesc) * (size_t)tiles);
    w.stop_end = off;
    w.row_dom = off;
    off += align256((size_t)(n_tokens > 0 ? n_tokens : 0));
    w.fused = off;
    off += align256(8 * (size_t)(fused_partials > 0 ? fused_partials : 0));
    w.total = off;
    return w;
}

}  // namespace stride

using namespace stride;

namespace {

thread_local char g_err[512] = "";

stride_status fail(stride_status st, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

stride_status ok() {
    g_err[0] = '\0';
    return STRIDE_OK;
}

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

stride_status check_layout(const stride_layout *L) {
    if (!L) return fail(STRIDE_ERR_INVALID_ARG, "layout is NULL");
    if (L->n_rollouts < 0 || L->n_turns < 0 || L->n_tokens < 0)
        return fail(STRIDE_ERR_INVALID_ARG, "negative layout size (R=%d T=%d N=%lld)", L->n_rollouts,
                    L->n_turns, (long long)L->n_tokens);
    if (!L->rollout_turn_off) return fail(STRIDE_ERR_INVALID_ARG, "rollout_turn_off is NULL");
    if (!L->turn_tok_off) return fail(STRIDE_ERR_INVALID_ARG, "turn_tok_off is NULL");
    if (L->n_tokens > 0 && L->n_turns == 0)
        return fail(STRIDE_ERR_INVALID_ARG, "N = %lld rows but no turns", (long long)L->n_tokens);
    if (L->n_turns > 0 && L->n_rollouts == 0)
        return fail(STRIDE_ERR_INVALID_ARG, "T = %d turns but no rollouts", L->n_turns);
    return STRIDE_OK;
}

stride_status check_ws(size_t need, void *ws, size_t ws_bytes) {
    if (!ws) return fail(STRIDE_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", need);
    if (!aligned(ws, 256)) return fail(STRIDE_ERR_WORKSPACE, "workspace is not 256-byte aligned");
    if (ws_bytes < need)
        return fail(STRIDE_ERR_WORKSPACE, "workspace has %zu bytes, need %zu", ws_bytes, need);
    return STRIDE_OK;
}

// Bytes of workspace the row-domain table (scoring) or retained-row mask (gradient) needs.
size_t rows_ws_bytes(const stride_layout &L) { return ws_layout(L.n_rollouts, L.n_tokens, 0, 0).total; }

// Bytes of workspace the stop test needs: tile counter, unit offsets, tile descriptors.
size_t stop_ws_bytes(const stride_layout &L, int64_t n_units) {
    return ws_layout(L.n_rollouts, 0, n_units, 0).stop_end;
}

stride_status check_domains(const double *table, int32_t n_dom, const char *name) {
    if (!table) return fail(STRIDE_ERR_INVALID_ARG, "%s is NULL", name);
    if (n_dom < 1 || n_dom > STRIDE_MAX_DOMAINS)
        return fail(STRIDE_ERR_UNSUPPORTED, "n_dom = %d outside 1..%d", n_dom, STRIDE_MAX_DOMAINS);
    return STRIDE_OK;
}

stride_status hip_fail(hipError_t e, const char *what) {
    return fail(STRIDE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace

extern "C" {

size_t stride_workspace_size(const stride_layout *layout, int32_t unit) {
    if (!layout) return 0;
    const int64_t n_units = (unit == STRIDE_UNIT_TOKEN) ? layout->n_tokens : layout->n_turns;
    return ws_layout(layout->n_rollouts, layout->n_tokens, n_units, 0).total;
}

const char *stride_last_error(void) { return g_err; }

stride_status stride_score(const stride_layout *layout, int32_t vocab, int64_t ld, int32_t dtype,
                           int32_t n_teachers, const void *const *teacher_logits,
                           const void *student_logits, const int32_t *token_ids, float *logp_t,
                           float *logp_s, float *kl, float *kl_full, double *turn_mean,
                           uint32_t *dev_flags, void *ws, size_t ws_bytes, hipStream_t stream) {
    stride_status st = check_layout(layout);
    if (st != STRIDE_OK) return st;
    const stride_layout &L = *layout;
    if (vocab < 1) return fail(STRIDE_ERR_INVALID_ARG, "vocab = %d < 1", vocab);
    if (ld < vocab) return fail(STRIDE_ERR_INVALID_ARG, "ld = %lld < vocab = %d", (long long)ld, vocab);
    if (dtype != STRIDE_BF16 && dtype != STRIDE_F32)
        return fail(STRIDE_ERR_UNSUPPORTED, "dtype %d is neither STRIDE_BF16 nor STRIDE_F32", dtype);
    const int64_t esize = dtype == STRIDE_BF16 ? 2 : 4;
    if ((ld * esize) % 16 != 0)
        return fail(STRIDE_ERR_UNSUPPORTED, "row stride %lld bytes is not a multiple of 16",
                    (long long)(ld * esize));
    if (n_teachers < 1 || n_teachers > STRIDE_MAX_DOMAINS)
        return fail(STRIDE_ERR_UNSUPPORTED, "n_teachers = %d outside 1..%d", n_teachers,
                    STRIDE_MAX_DOMAINS);
    if (!student_logits && (logp_s || kl || kl_full))
        return fail(STRIDE_ERR_INVALID_ARG, "logp_s / kl / kl_full requested without student logits");
    // the student rows' results are written to logp_s, and kl is formed from it
    if (student_logits && !logp_s && L.n_tokens > 0)
        return fail(STRIDE_ERR_INVALID_ARG, "student_logits given without logp_s");
    if ((kl || kl_full) && !logp_s && L.n_tokens > 0)
        return fail(STRIDE_ERR_INVALID_ARG, "kl / kl_full need logp_s as well");
    if (L.n_tokens > 0) {
        if (!teacher_logits) return fail(STRIDE_ERR_INVALID_ARG, "teacher_logits is NULL");
        for (int d = 0; d < n_teachers; ++d) {
            if (!teacher_logits[d])
                return fail(STRIDE_ERR_INVALID_ARG, "teacher_logits[%d] is NULL", d);
            if (!aligned(teacher_logits[d], 16))
                return fail(STRIDE_ERR_UNSUPPORTED, "teacher_logits[%d] is not 16-byte aligned", d);
        }
        if (student_logits && !aligned(student_logits, 16))
            return fail(STRIDE_ERR_UNSUPPORTED, "student_logits is not 16-byte aligned");
        if (!token_ids) return fail(STRIDE_ERR_INVALID_ARG, "token_ids is NULL");
        if (!logp_t) return fail(STRIDE_ERR_INVALID_ARG, "logp_t is NULL");
    }
    if (L.n_turns > 0 && !turn_mean) return fail(STRIDE_ERR_INVALID_ARG, "turn_mean is NULL");
    const bool routed = n_teachers > 1 && L.domain != nullptr;
    if (routed) {
        st = check_ws(rows_ws_bytes(L), ws, ws_bytes);
        if (st != STRIDE_OK) return st;
    }

    PtrTable tp{};
    for (int d = 0; d < n_teachers && teacher_logits; ++d) tp.p[d] = teacher_logits[d];
    uint8_t *row_dom = nullptr;
    hipError_t e;
    if (routed && L.n_tokens > 0) {
        const WsLayout w = ws_layout(L.n_rollouts, L.n_tokens, 0, 0);
        row_dom = static_cast<uint8_t *>(ws) + w.row_dom;
        e = launch_row_domain(L, n_teachers, row_dom, dev_flags, stream);
        if (e != hipSuccess) return hip_fail(e, "row-domain launch");
    }
    if (kl_full)
        e = launch_score_pairs(dtype, tp, n_teachers, row_dom, student_logits, token_ids, logp_t,
                               logp_s, kl_full, L.n_tokens, vocab, ld, dev_flags, stream);
    else
        e = launch_score_rows(dtype, tp, n_teachers, row_dom, student_logits, token_ids, logp_t,
                              logp_s, L.n_tokens, vocab, ld, dev_flags, stream);
    if (e != hipSuccess) return hip_fail(e, "row-scoring launch");
    e = launch_turn_mean(L, logp_t, logp_s, kl, turn_mean, dev_flags, stream);
    if (e != hipSuccess) return hip_fail(e, "turn-mean launch");
    return ok();
}

size_t stride_fused_workspace_size(const stride_layout *layout, int32_t vocab) {
    if (!layout || vocab < 1 || layout->n_tokens < 0) return 0;
    return fused_ws_bytes(layout->n_tokens, vocab);
}

stride_status stride_score_fused(const stride_layout *layout, int32_t vocab, int32_t d,
                                 const void *hidden_t, const void *w_t, const void *student_logits,
                                 int64_t ld, const int32_t *token_ids, float *logp_t, float *logp_s,
                                 float *kl, double *turn_mean, uint32_t *dev_flags, void *ws,
                                 size_t ws_bytes, hipStream_t stream) {
    stride_status st = check_layout(layout);
    if (st != STRIDE_OK) return st;
    const stride_layout &L = *layout;
    if (vocab < 1) return fail(STRIDE_ERR_INVALID_ARG, "vocab = %d < 1", vocab);
    if (d < 64 || d % 64 != 0 || d > kMaxFusedD)
        return fail(STRIDE_ERR_UNSUPPORTED,
                    "hidden size d = %d is not a multiple of 64 in [64, %d]", d, kMaxFusedD);
    if (!student_logits && (logp_s || kl))
        return fail(STRIDE_ERR_INVALID_ARG, "logp_s / kl requested without student logits");
    if (student_logits && !logp_s && L.n_tokens > 0)
        return fail(STRIDE_ERR_INVALID_ARG, "student_logits given without logp_s");
    if (L.n_tokens > 0) {
        if (!hidden_t || !w_t) return fail(STRIDE_ERR_INVALID_ARG, "hidden_t or w_t is NULL");
        if (!aligned(hidden_t, 16) || !aligned(w_t, 16))
            return fail(STRIDE_ERR_UNSUPPORTED, "hidden_t and w_t must be 16-byte aligned");
        if (!token_ids || !logp_t) return fail(STRIDE_ERR_INVALID_ARG, "token_ids or logp_t is NULL");
        if (student_logits) {
            if (ld < vocab)
                return fail(STRIDE_ERR_INVALID_ARG, "ld = %lld < vocab = %d", (long long)ld, vocab);
            if ((ld * 2) % 16 != 0 || !aligned(student_logits, 16))
                return fail(STRIDE_ERR_UNSUPPORTED, "student rows must be 16-byte aligned");
        }
    }
    if (L.n_turns > 0 && !turn_mean) return fail(STRIDE_ERR_INVALID_ARG, "turn_mean is NULL");
    const size_t need = fused_ws_bytes(L.n_tokens, vocab);
    if (!ws) return fail(STRIDE_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", need);
    if (!aligned(ws, 256)) return fail(STRIDE_ERR_WORKSPACE, "workspace is not 256-byte aligned");
    if (ws_bytes < need)
        return fail(STRIDE_ERR_WORKSPACE, "workspace has %zu bytes, need %zu", ws_bytes, need);

    hipError_t e = launch_fused_teacher(static_cast<const uint16_t *>(hidden_t),
                                        static_cast<const uint16_t *>(w_t), token_ids, logp_t,
                                        L.n_tokens, vocab, d, dev_flags, ws, stream);
    if (e != hipSuccess) return hip_fail(e, "fused projection launch");
    if (student_logits) {
        PtrTable sp{};
        sp.p[0] = student_logits;
        e = launch_score_rows(STRIDE_BF16, sp, 1, nullptr, nullptr, token_ids, logp_s, nullptr,
                              L.n_tokens, vocab, ld, dev_flags, stream);
        if (e != hipSuccess) return hip_fail(e, "student scoring launch");
    }
    e = launch_turn_mean(L, logp_t, logp_s, kl, turn_mean, dev_flags, stream);
    if (e != hipSuccess) return hip_fail(e, "turn-mean launch");
    return ok();
}

stride_status stride_stop(const stride_layout *layout, int32_t unit, const void *values,
                          const double *lambda, int32_t n_dom, const int32_t *start_unit,
                          double *cum, int32_t *stop_unit, int64_t *n_retained_tokens,
                          uint32_t *dev_flags, void *ws, size_t ws_bytes, hipStream_t stream) {
    stride_status st = check_layout(layout);
    if (st != STRIDE_OK) return st;
    const stride_layout &L = *layout;
    if (unit != STRIDE_UNIT_TURN && unit != STRIDE_UNIT_TOKEN)
        return fail(STRIDE_ERR_INVALID_ARG, "unit %d is neither STRIDE_UNIT_TURN nor STRIDE_UNIT_TOKEN",
                    unit);
    st = check_domains(lambda, n_dom, "lambda");
    if (st != STRIDE_OK) return st;
    const int64_t n_units = (unit == STRIDE_UNIT_TURN) ? L.n_turns : L.n_tokens;
    if (n_units > 0 && (!values || !cum))
        return fail(STRIDE_ERR_INVALID_ARG, "values or cum is NULL");
    if (L.n_rollouts > 0 && !stop_unit) return fail(STRIDE_ERR_INVALID_ARG, "stop_unit is NULL");
    st = check_ws(stop_ws_bytes(L, n_units), ws, ws_bytes);
    if (st != STRIDE_OK) return st;
    DomainTable lt{};
    for (int i = 0; i < n_dom; ++i) lt.v[i] = lambda[i];
    const hipError_t e = launch_stop(L, unit, values, lt, n_dom, start_unit, cum, stop_unit,
                                     n_retained_tokens, dev_flags, ws, stream);
    if (e != hipSuccess) return hip_fail(e, "stop launch");
    return ok();
}

stride_status stride_stop_noalloc(const stride_layout *layout, int32_t unit, const void *values,
                                  const double *lambda, int32_t n_dom, const int32_t *start_unit,
                                  double *cum, int32_t *stop_unit, int64_t *n_retained_tokens,
                                  uint32_t *dev_flags, hipStream_t stream) {
    stride_status st = check_layout(layout);
    if (st != STRIDE_OK) return st;
    const stride_layout &L = *layout;
    if (unit != STRIDE_UNIT_TURN && unit != STRIDE_UNIT_TOKEN)
        return fail(STRIDE_ERR_INVALID_ARG, "unit %d is neither STRIDE_UNIT_TURN nor STRIDE_UNIT_TOKEN",
                    unit);
    st = check_domains(lambda, n_dom, "lambda");
    if (st != STRIDE_OK) return st;
    const int64_t n_units = (unit == STRIDE_UNIT_TURN) ? L.n_turns : L.n_tokens;
    if (n_units > 0 && (!values || !cum))
        return fail(STRIDE_ERR_INVALID_ARG, "values or cum is NULL");
    if (L.n_rollouts > 0 && !stop_unit) return fail(STRIDE_ERR_INVALID_ARG, "stop_unit is NULL");
    const size_t need = stop_ws_bytes(L, n_units);
    if (need > (size_t)STRIDE_NOALLOC_SCRATCH_BYTES)
        return fail(STRIDE_ERR_UNSUPPORTED,
                    "layout needs %zu bytes of scratch (R = %d, %lld units); the fixed scratch "
                    "holds %zu: use stride_stop with a workspace",
                    need, L.n_rollouts, (long long)n_units, (size_t)STRIDE_NOALLOC_SCRATCH_BYTES);
    void *scratch = nullptr;
    hipError_t e = noalloc_scratch(&scratch);
    if (e != hipSuccess) return hip_fail(e, "scratch address lookup");
    DomainTable lt{};
    for (int i = 0; i < n_dom; ++i) lt.v[i] = lambda[i];
    e = launch_stop(L, unit, values, lt, n_dom, start_unit, cum, stop_unit, n_retained_tokens,
                    dev_flags, scratch, stream);
    if (e != hipSuccess) return hip_fail(e, "stop launch");
    return ok();
}

stride_status stride_stop_step(int32_t n_active, const int32_t *slot, const int64_t *new_off,
                               int32_t unit, const void *values, const int32_t *domain,
                               const double *lambda, int32_t n_dom, double *state_cum,
                               int32_t *state_units, int32_t *stop_unit, uint32_t *dev_flags,
                               hipStream_t stream) {
    if (n_active < 0) return fail(STRIDE_ERR_INVALID_ARG, "n_active = %d < 0", n_active);
    if (unit != STRIDE_UNIT_TURN && unit != STRIDE_UNIT_TOKEN)
        return fail(STRIDE_ERR_INVALID_ARG, "unit %d is neither STRIDE_UNIT_TURN nor STRIDE_UNIT_TOKEN",
                    unit);
    stride_status st = check_domains(lambda, n_dom, "lambda");
    if (st != STRIDE_OK) return st;
    if (n_active > 0 && (!slot || !new_off || !values || !state_cum || !state_units || !stop_unit))
        return fail(STRIDE_ERR_INVALID_ARG, "slot, new_off, values and the state arrays are required");
    DomainTable lt{};
    for (int i = 0; i < n_dom; ++i) lt.v[i] = lambda[i];
    const hipError_t e = launch_stop_step(n_active, slot, new_off, unit, values, domain, lt, n_dom,
                                          state_cum, state_units, stop_unit, dev_flags, stream);
    if (e != hipSuccess) return hip_fail(e, "stop-step launch");
    return ok();
}

stride_status stride_restart_turn(const stride_layout *layout, int32_t unit, const void *values,
                                  const int32_t *stop_unit, const double *alpha, int32_t n_dom,
                                  const uint8_t *correct_mask, int32_t *k_star, int32_t *k0,
                                  int32_t *k_max, uint32_t *dev_flags, hipStream_t stream) {
    stride_status st = check_layout(layout);
    if (st != STRIDE_OK) return st;
    const stride_layout &L = *layout;
    if (unit != STRIDE_UNIT_TURN && unit != STRIDE_UNIT_TOKEN)
        return fail(STRIDE_ERR_INVALID_ARG, "unit %d is neither STRIDE_UNIT_TURN nor STRIDE_UNIT_TOKEN",
                    unit);
    st = check_domains(alpha, n_dom, "alpha");
    if (st != STRIDE_OK) return st;
    const int64_t n_units = (unit == STRIDE_UNIT_TURN) ? L.n_turns : L.n_tokens;
    if (n_units > 0 && !values) return fail(STRIDE_ERR_INVALID_ARG, "values is NULL");
    if (L.n_rollouts > 0 && (!k_star || !k0))
        return fail(STRIDE_ERR_INVALID_ARG, "k_star or k0 is NULL");
    DomainTable at{};
    for (int i = 0; i < n_dom; ++i) at.v[i] = alpha[i];
    const hipError_t e = launch_restart(L, unit, values, stop_unit, at, n_dom, correct_mask, k_star,
                                        k0, k_max, dev_flags, stream);
    if (e != hipSuccess) return hip_fail(e, "restart launch");
    return ok();
}

stride_status stride_opd_grad(const stride_layout *layout, int32_t unit, int32_t vocab, int64_t ld,
                              int32_t dtype, const void *student_logits, const int32_t *token_ids,
                              const float *logp_t, const float *logp_s, const int32_t *start_unit,
                              const int32_t *stop_unit, float scale, void *grad, float *loss,
                              uint32_t *dev_flags, void *ws, size_t ws_bytes, hipStream_t stream) {
    stride_status st = check_layout(layout);
    if (st != STRIDE_OK) return st;
    const stride_layout &L = *layout;
    if (unit != STRIDE_UNIT_TURN && unit != STRIDE_UNIT_TOKEN)
        return fail(STRIDE_ERR_INVALID_ARG, "unit %d is neither STRIDE_UNIT_TURN nor STRIDE_UNIT_TOKEN",
                    unit);
    if (vocab < 1) return fail(STRIDE_ERR_INVALID_ARG, "vocab = %d < 1", vocab);
    if (ld < vocab) return fail(STRIDE_ERR_INVALID_ARG, "ld = %lld < vocab = %d", (long long)ld, vocab);
    if (dtype != STRIDE_BF16 && dtype != STRIDE_F32)
        return fail(STRIDE_ERR_UNSUPPORTED, "dtype %d is neither STRIDE_BF16 nor STRIDE_F32", dtype);
    const int64_t esize = dtype == STRIDE_BF16 ? 2 : 4;
    if ((ld * esize) % 16 != 0)
        return fail(STRIDE_ERR_UNSUPPORTED, "row stride %lld bytes is not a multiple of 16",
                    (long long)(ld * esize));
    if (L.n_tokens > 0) {
        if (!student_logits || !grad || !token_ids || !logp_t || !logp_s)
            return fail(STRIDE_ERR_INVALID_ARG, "student_logits, grad, token_ids, logp_t and logp_s are required");
        if (!aligned(student_logits, 16) || !aligned(grad, 16))
            return fail(STRIDE_ERR_UNSUPPORTED, "student_logits and grad must be 16-byte aligned");
    }
    st = check_ws(rows_ws_bytes(L), ws, ws_bytes);
    if (st != STRIDE_OK) return st;
    const WsLayout w = ws_layout(L.n_rollouts, L.n_tokens, 0, 0);
    uint8_t *mask = static_cast<uint8_t *>(ws) + w.row_dom;
    const hipError_t e = launch_opd_grad(L, unit, dtype, vocab, ld, student_logits, token_ids,
                                         logp_t, logp_s, start_unit, stop_unit, scale, grad, loss,
                                         dev_flags, mask, stream);
    if (e != hipSuccess) return hip_fail(e, "gradient launch");
    return ok();
}

stride_status stride_probe_read(const void *a, const void *b, int64_t n_rows, int64_t row_bytes,
                                int64_t read_bytes, uint32_t *sink, hipStream_t stream) {
    if (n_rows < 0) return fail(STRIDE_ERR_INVALID_ARG, "n_rows = %lld < 0", (long long)n_rows);
    if (n_rows == 0) return ok();
    if (!a || !sink) return fail(STRIDE_ERR_INVALID_ARG, "a or sink is NULL");
    if (read_bytes < 16 || read_bytes > row_bytes)
        return fail(STRIDE_ERR_INVALID_ARG, "read_bytes = %lld outside [16, row_bytes = %lld]",
                    (long long)read_bytes, (long long)row_bytes);
    if (row_bytes % 16 != 0 || !aligned(a, 16) || (b && !aligned(b, 16)))
        return fail(STRIDE_ERR_UNSUPPORTED, "rows must be 16-byte aligned");
    hipError_t e = launch_probe_read(a, b, n_rows, row_bytes, read_bytes, sink, stream);
    if (e != hipSuccess) return hip_fail(e, "probe launch");
    return ok();
}

stride_status stride_probe_read_flat(const void *a, const void *b, int64_t n_bytes, uint32_t *sink,
                                     int64_t sink_len, hipStream_t stream) {
    if (n_bytes < 0) return fail(STRIDE_ERR_INVALID_ARG, "n_bytes = %lld < 0", (long long)n_bytes);
    if (n_bytes == 0) return ok();
    if (!a || !sink) return fail(STRIDE_ERR_INVALID_ARG, "a or sink is NULL");
    if (sink_len < 4) return fail(STRIDE_ERR_INVALID_ARG, "sink_len = %lld < 4", (long long)sink_len);
    if (n_bytes % 16 != 0 || !aligned(a, 16) || (b && !aligned(b, 16)))
        return fail(STRIDE_ERR_UNSUPPORTED, "ranges must be 16-byte aligned multiples of 16 bytes");
    hipError_t e = launch_probe_flat(a, b, n_bytes, sink, sink_len, stream);
    if (e != hipSuccess) return hip_fail(e, "probe launch");
    return ok();
}

stride_status stride_probe_copy(const void *src, void *dst, const uint8_t *row_mask, int64_t n_rows,
                                int64_t row_bytes, int64_t copy_bytes, hipStream_t stream) {
    if (n_rows < 0) return fail(STRIDE_ERR_INVALID_ARG, "n_rows = %lld < 0", (long long)n_rows);
    if (n_rows == 0) return ok();
    if (!src || !dst) return fail(STRIDE_ERR_INVALID_ARG, "src or dst is NULL");
    if (copy_bytes < 16 || copy_bytes > row_bytes)
        return fail(STRIDE_ERR_INVALID_ARG, "copy_bytes = %lld outside [16, row_bytes = %lld]",
                    (long long)copy_bytes, (long long)row_bytes);
    if (row_bytes % 16 != 0 || !aligned(src, 16) || !aligned(dst, 16))
        return fail(STRIDE_ERR_UNSUPPORTED, "rows must be 16-byte aligned");
    hipError_t e = launch_probe_copy(src, dst, row_mask, n_rows, row_bytes, copy_bytes, stream);
    if (e != hipSuccess) return hip_fail(e, "probe launch");
    return ok();
}

}  // extern "C"
