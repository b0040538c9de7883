/*
 * c_client.c -- a plain C caller of libstride.so: score -> stop -> restart on inputs read from
 * files, outputs written to files.  No Python and no torch on this side of the boundary: device
 * memory comes from hipMalloc, and every call goes through the declarations in stride.h.
 *
 * usage: c_client DIR [--graph]
 *   DIR/meta.txt      "R T N V n_dom unit has_start has_mask has_domain"
 *   DIR/rto.i32       [R+1] rollout -> turn offsets      DIR/tto.i64   [T+1] turn -> row offsets
 *   DIR/teacher.bf16  [N][V] teacher logits (bf16 bits)  DIR/student.bf16 [N][V]
 *   DIR/ids.i32       [N] sampled tokens                 DIR/lambda.f64, DIR/alpha.f64 [n_dom]
 *   DIR/start.i32     [R] K0 per rollout (has_start)     DIR/mask.u8 [U] (has_mask)
 *   DIR/domain.i32    [R] (has_domain)
 * writes DIR/out_<name> for logp_t, logp_s, kl (f32 [N]), turn_mean (f64 [T]), cum (f64 [U]),
 * stop, k_star, k0, k_max (i32 [R]), retained (i64 [R]) and flags (u32).
 * With --graph the same three calls are then captured into a HIP graph on the stream
 * (hipStreamBeginCapture / hipStreamEndCapture), the outputs are overwritten with a sentinel,
 * and the graph is replayed three times; every output must equal the eager run's bit for bit.
 */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "stride.h"

static const char *g_dir;

static void die(const char *what, const char *detail) {
    fprintf(stderr, "c_client: %s: %s\n", what, detail);
    exit(1);
}

static void hip_ok(hipError_t e, const char *what) {
    if (e != hipSuccess) die(what, hipGetErrorString(e));
}

static void stride_ok(stride_status s, const char *what) {
    if (s != STRIDE_OK) die(what, stride_last_error());
}

static void *read_file(const char *name, size_t bytes) {
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", g_dir, name);
    FILE *f = fopen(path, "rb");
    if (!f) die("open", path);
    void *p = malloc(bytes ? bytes : 1);
    if (!p) die("malloc", path);
    if (bytes && fread(p, 1, bytes, f) != bytes) die("short read", path);
    fclose(f);
    return p;
}

static void write_file(const char *name, const void *p, size_t bytes) {
    char path[4096];
    snprintf(path, sizeof path, "%s/out_%s", g_dir, name);
    FILE *f = fopen(path, "wb");
    if (!f) die("create", path);
    if (bytes && fwrite(p, 1, bytes, f) != bytes) die("short write", path);
    fclose(f);
}

/* host buffer -> new device buffer of the same size */
static void *to_device(const void *h, size_t bytes) {
    void *d = NULL;
    hip_ok(hipMalloc(&d, bytes ? bytes : 16), "hipMalloc");
    if (bytes) hip_ok(hipMemcpy(d, h, bytes, hipMemcpyHostToDevice), "hipMemcpy H2D");
    return d;
}

static void *device_alloc(size_t bytes) {
    void *d = NULL;
    hip_ok(hipMalloc(&d, bytes ? bytes : 16), "hipMalloc");
    return d;
}

static void *to_host(const void *d, size_t bytes) {
    void *h = malloc(bytes ? bytes : 1);
    if (!h) die("malloc", "output");
    if (bytes) hip_ok(hipMemcpy(h, d, bytes, hipMemcpyDeviceToHost), "hipMemcpy D2H");
    return h;
}

/* device buffer equal, byte for byte, to a host copy */
static int same_as(const void *d, const void *h, size_t bytes) {
    void *x = to_host(d, bytes);
    const int eq = bytes == 0 || memcmp(x, h, bytes) == 0;
    free(x);
    return eq;
}

int main(int argc, char **argv) {
    const int graph = argc == 3 && strcmp(argv[2], "--graph") == 0;
    if (argc != 2 && !graph) die("usage", "c_client DIR [--graph]");
    g_dir = argv[1];
    int R, T, V, n_dom, unit, has_start, has_mask, has_domain;
    long long N;
    {
        char path[4096];
        snprintf(path, sizeof path, "%s/meta.txt", g_dir);
        FILE *f = fopen(path, "r");
        if (!f) die("open", path);
        if (fscanf(f, "%d %d %lld %d %d %d %d %d %d", &R, &T, &N, &V, &n_dom, &unit, &has_start,
                   &has_mask, &has_domain) != 9)
            die("parse", path);
        fclose(f);
    }
    const long long U = unit == STRIDE_UNIT_TURN ? T : N;
    /* rows padded so that every row starts 16-byte aligned */
    const long long ld = (V + 7) / 8 * 8;

    int32_t *rto = read_file("rto.i32", sizeof(int32_t) * (R + 1));
    int64_t *tto = read_file("tto.i64", sizeof(int64_t) * (T + 1));
    uint16_t *teacher = read_file("teacher.bf16", sizeof(uint16_t) * N * V);
    uint16_t *student = read_file("student.bf16", sizeof(uint16_t) * N * V);
    int32_t *ids = read_file("ids.i32", sizeof(int32_t) * N);
    double *lambda = read_file("lambda.f64", sizeof(double) * n_dom);
    double *alpha = read_file("alpha.f64", sizeof(double) * n_dom);
    int32_t *start = has_start ? read_file("start.i32", sizeof(int32_t) * R) : NULL;
    uint8_t *mask = has_mask ? read_file("mask.u8", U) : NULL;
    int32_t *domain = has_domain ? read_file("domain.i32", sizeof(int32_t) * R) : NULL;

    uint16_t *tpad = calloc((size_t)(N * ld) + 1, sizeof(uint16_t));
    uint16_t *spad = calloc((size_t)(N * ld) + 1, sizeof(uint16_t));
    if (!tpad || !spad) die("calloc", "padded rows");
    for (long long i = 0; i < N; ++i) {
        memcpy(tpad + i * ld, teacher + i * V, sizeof(uint16_t) * V);
        memcpy(spad + i * ld, student + i * V, sizeof(uint16_t) * V);
    }

    stride_layout L;
    L.n_rollouts = R;
    L.n_turns = T;
    L.n_tokens = N;
    L.rollout_turn_off = to_device(rto, sizeof(int32_t) * (R + 1));
    L.turn_tok_off = to_device(tto, sizeof(int64_t) * (T + 1));
    L.domain = has_domain ? to_device(domain, sizeof(int32_t) * R) : NULL;

    const void *d_teacher = to_device(tpad, sizeof(uint16_t) * N * ld);
    const void *d_student = to_device(spad, sizeof(uint16_t) * N * ld);
    int32_t *d_ids = to_device(ids, sizeof(int32_t) * N);
    int32_t *d_start = has_start ? to_device(start, sizeof(int32_t) * R) : NULL;
    uint8_t *d_mask = has_mask ? to_device(mask, U) : NULL;
    float *d_logp_t = device_alloc(sizeof(float) * N);
    float *d_logp_s = device_alloc(sizeof(float) * N);
    float *d_kl = device_alloc(sizeof(float) * N);
    double *d_turn_mean = device_alloc(sizeof(double) * T);
    double *d_cum = device_alloc(sizeof(double) * U);
    int32_t *d_stop = device_alloc(sizeof(int32_t) * R);
    int64_t *d_retained = device_alloc(sizeof(int64_t) * R);
    int32_t *d_kstar = device_alloc(sizeof(int32_t) * R);
    int32_t *d_k0 = device_alloc(sizeof(int32_t) * R);
    int32_t *d_kmax = device_alloc(sizeof(int32_t) * R);
    uint32_t zero = 0;
    uint32_t *d_flags = to_device(&zero, sizeof zero);

    const size_t ws_bytes = stride_workspace_size(&L, unit);
    void *d_ws = device_alloc(ws_bytes);
    hipStream_t stream;
    hip_ok(hipStreamCreate(&stream), "hipStreamCreate");

    const void *teachers[1] = {d_teacher};
    const void *values = unit == STRIDE_UNIT_TURN ? (const void *)d_turn_mean : (const void *)d_logp_t;
    /* score -> stop -> restart, issued on the stream without waiting */
#define STEP()                                                                                     \
    do {                                                                                           \
        stride_ok(stride_score(&L, V, ld, STRIDE_BF16, 1, teachers, d_student, d_ids, d_logp_t,   \
                               d_logp_s, d_kl, NULL, d_turn_mean, d_flags, d_ws, ws_bytes, stream), \
                  "stride_score");                                                                 \
        stride_ok(stride_stop(&L, unit, values, lambda, n_dom, d_start, d_cum, d_stop, d_retained, \
                              d_flags, d_ws, ws_bytes, stream),                                    \
                  "stride_stop");                                                                  \
        stride_ok(stride_restart_turn(&L, unit, values, d_stop, alpha, n_dom, d_mask, d_kstar,     \
                                      d_k0, d_kmax, d_flags, stream),                              \
                  "stride_restart_turn");                                                          \
    } while (0)
    STEP();
    hip_ok(hipStreamSynchronize(stream), "hipStreamSynchronize");

    struct { const char *name; void *dev; size_t bytes; void *host; } out[] = {
        {"logp_t", d_logp_t, sizeof(float) * N, NULL},     {"logp_s", d_logp_s, sizeof(float) * N, NULL},
        {"kl", d_kl, sizeof(float) * N, NULL},             {"turn_mean", d_turn_mean, sizeof(double) * T, NULL},
        {"cum", d_cum, sizeof(double) * U, NULL},          {"stop", d_stop, sizeof(int32_t) * R, NULL},
        {"retained", d_retained, sizeof(int64_t) * R, NULL}, {"k_star", d_kstar, sizeof(int32_t) * R, NULL},
        {"k0", d_k0, sizeof(int32_t) * R, NULL},           {"k_max", d_kmax, sizeof(int32_t) * R, NULL},
        {"flags", d_flags, sizeof(uint32_t), NULL},
    };
    const int n_out = (int)(sizeof out / sizeof out[0]);
    for (int i = 0; i < n_out; ++i) {
        out[i].host = to_host(out[i].dev, out[i].bytes);
        write_file(out[i].name, out[i].host, out[i].bytes);
    }

    if (graph) {
        /* the same three calls captured once; the library allocates, synchronises and memsets
           nothing, so the captured graph holds only its kernels */
        hipGraph_t g;
        hipGraphExec_t exec;
        hip_ok(hipStreamBeginCapture(stream, hipStreamCaptureModeGlobal), "hipStreamBeginCapture");
        STEP();
        hip_ok(hipStreamEndCapture(stream, &g), "hipStreamEndCapture");
        hip_ok(hipGraphInstantiate(&exec, g, NULL, NULL, 0), "hipGraphInstantiate");
        for (int rep = 0; rep < 3; ++rep) {
            /* outputs overwritten outside the graph: a sentinel, and the flag word cleared */
            for (int i = 0; i < n_out; ++i)
                if (out[i].bytes)
                    hip_ok(hipMemset(out[i].dev, i == n_out - 1 ? 0 : 0xA5, out[i].bytes), "hipMemset");
            hip_ok(hipGraphLaunch(exec, stream), "hipGraphLaunch");
            hip_ok(hipStreamSynchronize(stream), "hipStreamSynchronize");
            for (int i = 0; i < n_out; ++i)
                if (!same_as(out[i].dev, out[i].host, out[i].bytes)) die("graph replay differs", out[i].name);
        }
        hip_ok(hipGraphExecDestroy(exec), "hipGraphExecDestroy");
        hip_ok(hipGraphDestroy(g), "hipGraphDestroy");
        printf("c_client: graph of the step replayed 3 times, every output equal to the eager run\n");
    }
#undef STEP
    hip_ok(hipStreamDestroy(stream), "hipStreamDestroy");
    /* the caller owns every buffer the library was handed: release them */
    for (int i = 0; i < n_out; ++i) {
        free(out[i].host);
        hip_ok(hipFree(out[i].dev), "hipFree");
    }
    const void *inputs[] = {L.rollout_turn_off, L.turn_tok_off, L.domain, d_teacher, d_student,
                            d_ids, d_start, d_mask, d_ws};
    for (size_t i = 0; i < sizeof inputs / sizeof inputs[0]; ++i)
        if (inputs[i]) hip_ok(hipFree((void *)inputs[i]), "hipFree");
    free(rto), free(tto), free(teacher), free(student), free(ids), free(lambda), free(alpha);
    free(start), free(mask), free(domain), free(tpad), free(spad);
    printf("c_client: R=%d T=%d N=%lld V=%d unit=%d ws=%zu bytes: ok\n", R, T, N, V, unit, ws_bytes);
    return 0;
}
