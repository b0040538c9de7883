/*
 * stride.h -- C ABI of libstride.so: the data-parallel hot path of STRIDE's
 * on-policy distillation step on one AMD Instinct MI355X (gfx950).
 *
 * Paper: "Know When to Stop, Where to Restart: Accelerating Multi-Turn Agentic
 * On-Policy Distillation" (STRIDE).  The path scores student rollouts with the
 * teacher and the student (Eq. 1, Sec. 3.1-3.2), averages the teacher
 * log-probability per turn (Eq. 4), applies the early-stop test (Eq. 5,
 * Sec. 4.1, with token units for the single-turn variant of Sec. 5.5) and
 * picks the restart turn of the prefix buffer (Sec. 4.2, Eq. 6, Algorithm 1).
 *
 * Conventions shared by every entry point
 *   - Pointers are device pointers unless marked (host).  The caller owns every
 *     buffer; the library keeps no state between calls and allocates nothing.
 *     Scratch memory is the caller's workspace `ws` of at least
 *     stride_workspace_size() bytes, 256-byte aligned, used in stream order.
 *   - Calls are asynchronous on `stream` and never synchronise.  Two calls that
 *     share a workspace must be ordered (same stream, or events).
 *   - Argument errors (null pointers, negative sizes, misaligned rows, too small
 *     a workspace, unsupported dtype) are found on the host before anything is
 *     launched: the call returns a non-OK status, launches nothing, and
 *     stride_last_error() describes the problem.
 *   - Data errors found on the device are OR-ed into *dev_flags (a device
 *     uint32, may be NULL) and the call still completes; the affected outputs
 *     are NaN (or -1 for indices).  Read dev_flags after synchronising.
 *   - Layout: the scored tokens of all rollouts form one stream of N rows in
 *     rollout order.  Rollout r owns turns [rollout_turn_off[r],
 *     rollout_turn_off[r+1]); turn k owns rows [turn_tok_off[k],
 *     turn_tok_off[k+1]).  Only tokens the student generated are rows: the
 *     environment's observation tokens are masked out of the loss (Eq. 2) and
 *     are not part of the stream.  Indices of turns and units returned per
 *     rollout are 0-based and local to the rollout; the paper's 1-based k*
 *     is k_star + 1, and its K0 = k* - 1 equals k0.
 *   - Units: STRIDE_UNIT_TURN makes each turn a unit whose value is its mean
 *     teacher log-probability (Eq. 4, Eq. 5); STRIDE_UNIT_TOKEN makes each row
 *     a unit whose value is its teacher log-probability (Sec. 5.5).
 */
#ifndef STRIDE_H
#define STRIDE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    STRIDE_OK = 0,
    STRIDE_ERR_INVALID_ARG = 1, /* a null pointer, a negative size, inconsistent sizes   */
    STRIDE_ERR_UNSUPPORTED = 2, /* dtype, alignment or a size past the library limits    */
    STRIDE_ERR_WORKSPACE = 3,   /* ws is NULL, misaligned or smaller than required       */
    STRIDE_ERR_HIP = 4          /* a HIP launch failed; the message names the HIP error  */
} stride_status;

enum { STRIDE_BF16 = 0, STRIDE_F32 = 1 };          /* logits element type         */
enum { STRIDE_UNIT_TURN = 0, STRIDE_UNIT_TOKEN = 1 };

/* Device data-error flags, OR-ed into *dev_flags. */
enum {
    STRIDE_FLAG_TOKEN_OOB = 1,   /* token id outside [0, vocab): that row's outputs are NaN        */
    STRIDE_FLAG_EMPTY_TURN = 2,  /* a turn with no rows: its mean is NaN                            */
    STRIDE_FLAG_BAD_OFFSETS = 4, /* offsets not monotone, not starting at 0 or not ending at N/T    */
    STRIDE_FLAG_NONFINITE = 8,   /* a row holds NaN or +inf, or only -inf: its outputs are NaN      */
    STRIDE_FLAG_BAD_DOMAIN = 16, /* domain[r] outside [0, n_dom), or [0, n_teachers) when routing  */
    STRIDE_FLAG_SPIN_LIMIT = 32  /* a cross-workgroup wait gave up; the scan results are not valid  */
};

#define STRIDE_MAX_DOMAINS 64

typedef struct {
    int32_t n_rollouts;              /* R >= 0                                        */
    int32_t n_turns;                 /* T >= 0                                        */
    int64_t n_tokens;                /* N >= 0, rows of every logits matrix           */
    const int32_t *rollout_turn_off; /* [R+1], 0 .. T, non-decreasing                 */
    const int64_t *turn_tok_off;     /* [T+1], 0 .. N, non-decreasing                 */
    const int32_t *domain;           /* [R] teacher / lambda / alpha index, NULL => 0 */
} stride_layout;

/*
 * Bytes of workspace the calls below need for this layout and unit (the
 * maximum over stride_score, stride_stop, stride_restart_turn and
 * stride_opd_grad, so one buffer serves them all; stride_score_fused sizes its
 * own with stride_fused_workspace_size).  Host-only; reads only the sizes in
 * *layout.  Returns 0 for a NULL layout.
 */
size_t stride_workspace_size(const stride_layout *layout, int32_t unit);

/*
 * Teacher and student scoring of every row, then the per-turn mean.
 * Eq. (1) (Sec. 3.1): log pi(y_t | y_<t) is the log-softmax of the row's
 * logits at the sampled token y_t, for the teacher (T) and the student (S);
 * Sec. 3.2: the per-token KL estimate is log pi_S(y_t) - log pi_T(y_t) = -r_t;
 * Eq. (4): lbar_k = (1/n_k) sum over turn k's rows of log pi_T.
 *
 *   vocab            V >= 1 logits per row; rows have ld >= V elements, row-major
 *   ld               row stride in elements; ld * element size must be a multiple
 *                    of 16 bytes, and every logits pointer 16-byte aligned
 *   dtype            STRIDE_BF16 or STRIDE_F32
 *   n_teachers       1 .. STRIDE_MAX_DOMAINS
 *   teacher_logits   (host) array of n_teachers device pointers, each [N, ld];
 *                    with n_teachers > 1 the rows of rollout r are read from
 *                    teacher domain[r] (rows of rollouts routed elsewhere are
 *                    never read) and a domain id outside [0, n_teachers) raises
 *                    STRIDE_FLAG_BAD_DOMAIN with NaN outputs for its rows; with
 *                    n_teachers = 1 every row reads teacher 0 and the domain ids
 *                    are not used here (they select lambda and alpha in
 *                    stride_stop and stride_restart_turn, which check them)
 *   student_logits   [N, ld] or NULL (then logp_s, kl and kl_full must be NULL)
 *   token_ids        [N] int32, the sampled tokens
 *   logp_t, logp_s   [N] float outputs; logp_s is required with student_logits
 *                    (STRIDE_ERR_INVALID_ARG otherwise) and must be NULL without
 *   kl               [N] float output log pi_S - log pi_T, or NULL
 *   kl_full          [N] float output or NULL: the exact reverse KL over the whole
 *                    vocabulary, KL(pi_S || pi_T) = sum_v pi_S(v) log(pi_S(v) / pi_T(v)),
 *                    the divergence whose sequence-level form OPD minimises (Sec. 3.1);
 *                    needs student_logits.  Computed in the same single pass over both
 *                    rows (one wavefront reads the token's teacher and student rows).
 *   turn_mean        [T] double output
 *   dev_flags        device uint32 or NULL
 *
 * Values: -inf logits carry no mass; NaN, +inf or an all -inf row raise
 * STRIDE_FLAG_NONFINITE and give NaN outputs for that row.  Finite logits are
 * supported up to |x| = 2^127 (the exponent is formed as x * log2(e) in fp32);
 * rows with larger finite values are outside the supported range.
 */
stride_status stride_score(const stride_layout *layout, int32_t vocab, int64_t ld, int32_t dtype,
                           int32_t n_teachers, const void *const *teacher_logits,
                           const void *student_logits, const int32_t *token_ids, float *logp_t,
                           float *logp_s, float *kl, float *kl_full, double *turn_mean,
                           uint32_t *dev_flags, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * As stride_score, with the teacher's logits produced by its output
 * projection inside the kernel and never written to memory: z = h W^T with h
 * the teacher's final hidden state of the row and W its lm_head weight, then
 * the same log-softmax at the sampled token (Eq. 1).  The projection runs on
 * the matrix cores (bf16 inputs, fp32 accumulation).  The student's logits
 * are given as in stride_score.
 *
 *   d                hidden size, a multiple of 64 in [64, 65536]
 *   hidden_t         [N, d] bf16 row-major, 16-byte aligned
 *   w_t              [vocab, d] bf16 row-major (a linear layer's weight: row v
 *                    holds the weights of vocabulary entry v), 16-byte aligned
 *   student_logits   [N, ld] bf16 or NULL; logp_s is required with it and kl
 *                    needs it (as in stride_score)
 *   ws               at least stride_fused_workspace_size(layout, vocab) bytes
 */
stride_status stride_score_fused(const stride_layout *layout, int32_t vocab, int32_t d,
                                 const void *hidden_t, const void *w_t, const void *student_logits,
                                 int64_t ld, const int32_t *token_ids, float *logp_t, float *logp_s,
                                 float *kl, double *turn_mean, uint32_t *dev_flags, void *ws,
                                 size_t ws_bytes, hipStream_t stream);

/*
 * Bytes of workspace stride_score_fused needs: a table of per-row partial
 * (max, sum) pairs, one per 128 vocabulary entries, plus one float per row.
 * Host-only; 0 for a NULL layout.
 */
size_t stride_fused_workspace_size(const stride_layout *layout, int32_t vocab);

/*
 * Early-stop test, Eq. (5) (Sec. 4.1), over the new units of each rollout:
 * C_u = sum_{j=K0}^{u} value_j for u >= K0 = start_unit[r] (the prefix reused
 * from an earlier rollout is left out of the sum, Sec. 4.1 and Algorithm 1);
 * stop_unit[r] is the first u >= K0 with C_u < lambda[domain[r]], strictly,
 * or -1.  The triggering unit is kept for the loss.
 *
 *   unit              STRIDE_UNIT_TURN (values = turn_mean, double [T]) or
 *                     STRIDE_UNIT_TOKEN (values = logp_t, float [N])
 *   lambda            (host) [n_dom] thresholds, n_dom in 1 .. STRIDE_MAX_DOMAINS
 *   start_unit        [R] int32 K0 per rollout (clamped to [0, units]), or NULL => 0
 *   cum               [U] double output: C_u, and 0 for u < K0
 *   stop_unit         [R] int32 output
 *   n_retained_tokens [R] int64 output or NULL: rows of units K0 .. stop
 *                     (K0 .. last unit without a stop), the newly generated rows
 *                     that join the loss
 * Sums are carried in double; results do not depend on scheduling.
 */
stride_status stride_stop(const stride_layout *layout, int32_t unit, const void *values,
                          const double *lambda, int32_t n_dom, const int32_t *start_unit,
                          double *cum, int32_t *stop_unit, int64_t *n_retained_tokens,
                          uint32_t *dev_flags, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * stride_stop without a workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation).  Arguments, outputs and errors are those of stride_stop without
 * ws / ws_bytes.  The call allocates nothing: its scratch (tile counter, unit
 * offsets, scan tile descriptors; 256 + 8 (R + 1) + 16 ceil(U / 2048) bytes, each
 * part rounded up to 256) lives in a fixed device array of
 * STRIDE_NOALLOC_SCRATCH_BYTES per GPU, which the library holds until the process
 * ends (for example R = 65,536 rollouts with up to 67 million units fit).  A layout
 * that needs more returns STRIDE_ERR_UNSUPPORTED before any launch.  The first call
 * on each device looks up that device's array address.  Every call on one GPU
 * shares the array, which keeps the last call's contents; the call clears what must
 * start at zero with its own kernel, in stream order.  Calls that overlap on one
 * GPU (unordered streams, or several host threads) race: order them.
 */
#define STRIDE_NOALLOC_SCRATCH_BYTES (1u << 20)
stride_status stride_stop_noalloc(const stride_layout *layout, int32_t unit, const void *values,
                                  const double *lambda, int32_t n_dom, const int32_t *start_unit,
                                  double *cum, int32_t *stop_unit, int64_t *n_retained_tokens,
                                  uint32_t *dev_flags, hipStream_t stream);

/*
 * Online form of the stop test, for use while rollouts are being generated
 * (Algorithm 1's inner loop: after each new turn the teacher scores it and the
 * sum over the new turns is tested against lambda, Eq. 5).  Each call appends new
 * units to some rollouts and updates their stop state in place; feeding a
 * rollout's units in any split gives the stride_stop result for the whole rollout.
 *
 *   n_active          number of rollouts receiving units in this call
 *   slot              [n_active] int32 state index of each (0 .. size of the state arrays)
 *   new_off           [n_active+1] int64 CSR offsets into values
 *   unit, values      STRIDE_UNIT_TURN: double turn means (from stride_score on the
 *                     new turns); STRIDE_UNIT_TOKEN: float teacher log-probabilities
 *   domain            [slots] int32 or NULL => 0;  lambda (host) [n_dom]
 *   state_cum         [slots] double, running sum over the new units (0 at the start)
 *   state_units       [slots] int32, local index of the next unit (K0 at the start)
 *   stop_unit         [slots] int32, -1 while running; set to the local index of
 *                     the triggering unit, after which the rollout ignores new units
 * The caller initialises the three state arrays for a rollout before its first
 * call; slots not named in a call are untouched.  Calls naming the same slot twice
 * race.
 */
stride_status stride_stop_step(int32_t n_active, const int32_t *slot, const int64_t *new_off,
                               int32_t unit, const void *values, const int32_t *domain,
                               const double *lambda, int32_t n_dom, double *state_cum,
                               int32_t *state_units, int32_t *stop_unit, uint32_t *dev_flags,
                               hipStream_t stream);

/*
 * Prefix-buffer restart pick (Sec. 4.2 steps 1-3, Eq. 6, Algorithm 1) from the
 * record of each rollout: its units 0 .. stop_unit[r] (all units when
 * stop_unit is NULL or stop_unit[r] = -1).  Unit u is correct iff
 * correct_mask[u] != 0 (NULL => every unit) and value_u > alpha[domain[r]],
 * strictly.  k_max[r] is the length of the leading run of correct units;
 * k_star[r] is the lowest index u < k_max attaining the minimum value (-1 if
 * k_max = 0); k0[r] = max(k_star, 0) is the number of units the next rollout
 * reuses as context.
 *
 *   unit, values      as in stride_stop
 *   alpha             (host) [n_dom]; -INFINITY disables the gate
 *   correct_mask      [U] uint8 or NULL
 *   k_star, k0        [R] int32 outputs;  k_max [R] int32 output or NULL
 */
stride_status stride_restart_turn(const stride_layout *layout, int32_t unit, const void *values,
                                  const int32_t *stop_unit, const double *alpha, int32_t n_dom,
                                  const uint8_t *correct_mask, int32_t *k_star, int32_t *k0,
                                  int32_t *k_max, uint32_t *dev_flags, hipStream_t stream);

/*
 * Token-level OPD loss and its gradient with respect to the student's logits,
 * Eq. (2) (Sec. 3.1): L = -scale * sum_t log pi_S(y_t) r_t 1_trainable(t), with
 * r_t = log pi_T(y_t) - log pi_S(y_t) held constant.  The trainable rows are the
 * retained ones: units start_unit[r] .. stop_unit[r] of each rollout (to its last
 * unit without a stop), the trigger included (Sec. 4.1, Algorithm 1).  For those
 * rows  grad[t, v] = scale * r_t * (pi_S(v) - [v = y_t]);  other rows get zeros.
 * pi_S comes from the row and log pi_S(y_t): LSE_S = s_y - log pi_S(y_t).
 *
 *   unit              STRIDE_UNIT_TURN or STRIDE_UNIT_TOKEN, as given to stride_stop
 *   student_logits    [N, ld] (dtype as in stride_score), read once per retained row
 *   logp_t, logp_s    [N] from stride_score
 *   start_unit        [R] K0 or NULL => 0;  stop_unit  [R] from stride_stop or NULL => none
 *   scale             multiplies loss and gradient (e.g. 1 / number of retained rows)
 *   grad              [N, ld] output, same dtype as the logits; columns >= vocab untouched
 *   loss              [N] float output (0 on rows that are not retained) or NULL
 *   ws                at least stride_workspace_size(layout, unit) bytes
 */
stride_status stride_opd_grad(const stride_layout *layout, int32_t unit, int32_t vocab, int64_t ld,
                              int32_t dtype, const void *student_logits, const int32_t *token_ids,
                              const float *logp_t, const float *logp_s, const int32_t *start_unit,
                              const int32_t *stop_unit, float scale, void *grad, float *loss,
                              uint32_t *dev_flags, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * Per-task trajectory record H(x) of the prefix buffer (Algorithm 1), kept on
 * the host.  After a rollout of task x, put() stores its per-unit values (turn
 * means, or token log-probabilities in the single-turn setting) and optional
 * correctness mask, replacing the previous record.  Before the next rollout,
 * plan() returns for each task the restart pick of Sec. 4.2 / Eq. (6) on its
 * record -- K_max (leading correct run, value > alpha and mask set), k* (lowest
 * index of its minimum, -1 if K_max = 0) and K0 = max(k*, 0) units of reused
 * context -- or k* = -1, K0 = 0, K_max = 0 for a task without a record.
 * All pointers here are host pointers.  The store is an object the caller
 * creates and destroys (host memory only); its calls are thread-safe.
 * get() copies up to `capacity` values (and mask bytes, 1 where none was
 * stored) and returns the record length, or -1 if the task has none.
 */
typedef struct stride_records stride_records;
stride_records *stride_records_create(void);
void stride_records_destroy(stride_records *rec);
stride_status stride_records_put(stride_records *rec, int64_t task, int32_t n_units,
                                 const double *values, const uint8_t *mask);
int32_t stride_records_get(stride_records *rec, int64_t task, int32_t capacity, double *values,
                           uint8_t *mask);
int64_t stride_records_size(stride_records *rec);
stride_status stride_records_plan(stride_records *rec, int32_t n_tasks, const int64_t *tasks,
                                  const double *alpha, int32_t *k_star, int32_t *k0,
                                  int32_t *k_max);

/* Streaming-read reference (a measurement aid, not a step of the method).
 *
 * Reads n_rows rows of `a` (and, when b is not NULL, the same rows of `b`,
 * interleaved row by row) with the scoring kernel's access pattern for batches of
 * 16,384 row items or more -- one wavefront per row, 16-byte non-temporal loads
 * -- and does no arithmetic, so
 * timing it gives the read bandwidth that pattern reaches; the scoring kernel's
 * bandwidth is reported as a fraction of it next to the fraction of peak.
 *   a, b        device rows, 16-byte aligned; b may be NULL
 *   n_rows      rows to read from each matrix (>= 0)
 *   row_bytes   row stride in bytes, a multiple of 16
 *   read_bytes  bytes read from the start of each row, <= row_bytes (rounded
 *               down to a multiple of 16)
 *   sink        [n_rows, or 2 * n_rows with b] uint32 written with an XOR of
 *               each row's words (keeps the loads live)
 * Errors: STRIDE_ERR_INVALID_ARG for NULL pointers or inconsistent sizes,
 * STRIDE_ERR_UNSUPPORTED for misaligned rows. */
stride_status stride_probe_read(const void *a, const void *b, int64_t n_rows, int64_t row_bytes,
                                int64_t read_bytes, uint32_t *sink, hipStream_t stream);

/* Streaming-read reference in the plainest order (a measurement aid, not a step of
 * the method): reads the first n_bytes of a, then of b (when not NULL), as one
 * contiguous range each, in a grid-stride order with 16-byte non-temporal loads,
 * so that its rate, next to stride_probe_read's on the same bytes, separates the
 * effect of the row-per-wavefront pattern from that of the footprint.
 *   n_bytes     a multiple of 16 (>= 0); a, b 16-byte aligned
 *   sink        [sink_len >= 4] uint32; min(2048, sink_len / 4) workgroups write
 *               one XOR word per wavefront
 * Errors: STRIDE_ERR_INVALID_ARG for NULL pointers or sizes out of range,
 * STRIDE_ERR_UNSUPPORTED for misaligned ranges. */
stride_status stride_probe_read_flat(const void *a, const void *b, int64_t n_bytes, uint32_t *sink,
                                     int64_t sink_len, hipStream_t stream);

/* Streaming read+write reference for the OPD gradient's roofline (a measurement aid,
 * not a step of the method): moves n_rows rows as stride_opd_grad does -- eight
 * wavefronts per row, a 16-byte non-temporal load and store per word -- copying the
 * first copy_bytes of each row of src to dst; a row whose row_mask byte is 0 is
 * written as zeros without being read (row_mask may be NULL: every row copied).
 *   src, dst    device rows of row_bytes (a multiple of 16), 16-byte aligned
 *   copy_bytes  in [16, row_bytes], rounded down to a multiple of 16
 * Errors as stride_probe_read. */
stride_status stride_probe_copy(const void *src, void *dst, const uint8_t *row_mask, int64_t n_rows,
                                int64_t row_bytes, int64_t copy_bytes, hipStream_t stream);

/* Test hook of the stop test's cross-workgroup look-back (not a step of the method).
 *
 * In the library built for testing (libstride_debug.so, scan compiled with
 * STRIDE_SCAN_DELAY_HOOK), later stride_stop / stride_stop_noalloc calls make the scan tiles
 * picked by a hash of (seed, tile) -- about one in `one_in` -- sleep 1 .. `sleeps` times
 * s_sleep(127) (about 8,000 cycles each) before publishing their aggregate, so that their
 * successors look back over descriptors that are not yet published.  The waits stay far below
 * the look-back spin limit, so every wave exits normally and the results must equal the
 * undelayed ones bit for bit.  one_in = 0 switches the delays off.  Process-wide setting.
 * Returns STRIDE_ERR_INVALID_ARG for sleeps outside 1 .. 1000 (with one_in > 0), and
 * STRIDE_ERR_UNSUPPORTED in the product library (libstride.so), which has no delay code. */
stride_status stride_debug_scan_delay(uint64_t seed, uint32_t one_in, uint32_t sleeps);

/* Test hook of the look-back's bounded wait (not a step of the method).
 *
 * In libstride_debug.so, later stride_stop / stride_stop_noalloc calls let a scan tile wait at
 * most `limit` rounds of s_sleep(1) for each predecessor's descriptor instead of the library's
 * own bound (2^22 rounds); limit = 0 restores that bound.  With a tiny limit and the delays of
 * stride_debug_scan_delay, successors give up: the call still completes, raises
 * STRIDE_FLAG_SPIN_LIMIT and writes NaN to the cumulative values that needed the missing carry,
 * so the error path can be tested while every wave exits normally.  Process-wide setting.
 * Returns STRIDE_ERR_UNSUPPORTED in the product library (libstride.so). */
stride_status stride_debug_scan_spin_limit(uint32_t limit);

/* Test hook of the fused projection's tile order (not a step of the method).
 *
 * In libstride_debug.so (fused projection compiled with STRIDE_FUSED_BAND_HOOK), later
 * stride_score_fused calls group `band` super-rows of 4,096 rows per band instead of the
 * library's own choice (as many as fit 128 MiB of h; band = 0 restores it).  The band only
 * orders the tiles, so every output must be the same bit for bit at any band; the hook lets a
 * test check that and a benchmark time one order against another.  Process-wide setting.
 * Returns STRIDE_ERR_INVALID_ARG for band < 0, and STRIDE_ERR_UNSUPPORTED in the product
 * library (libstride.so). */
stride_status stride_debug_fused_band(int32_t band);

/* Message for the last non-OK status returned on this thread ("" if none). */
const char *stride_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* STRIDE_H */
