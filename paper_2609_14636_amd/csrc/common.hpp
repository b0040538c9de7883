// common.hpp -- declarations shared by the HIP sources of libstride.so.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/stride.h"

namespace stride {

constexpr int kWave = 64;
// Threads per workgroup of the one-row-per-wave streaming kernels (the row scoring kernel and
// the read reference that mirrors it): eight rows per workgroup read about 0.6% faster from
// HBM than four.
constexpr int kRowThreads = 512;

// Device-side view of the host's per-domain tables, passed by value.
struct DomainTable {
    double v[STRIDE_MAX_DOMAINS];
};
struct PtrTable {
    const void *p[STRIDE_MAX_DOMAINS];
};

// Scan tile descriptor published by one tile and read by its successors.
struct alignas(16) TileDesc {
    double value;     // sum of the tile's values after its last segment head
    uint32_t head;    // 1 if a segment starts inside the tile
    uint32_t status;  // 0 = not yet published, 1 = aggregate ready
};

// Workspace layout (byte offsets from ws, each region 256-byte aligned).
struct WsLayout {
    size_t counter;   // uint32 tile counter + spare words
    size_t unit_off;  // int64 [R+1] first unit of each rollout
    size_t desc;      // TileDesc [tiles]
    size_t stop_end;  // end of the regions the stop test uses
    size_t row_dom;   // uint8 [N] teacher index per row (multi-teacher scoring) or
                      // retained-row mask (gradient)
    size_t fused;     // float2 [N, vocab tiles] partial (max, sum) of the fused projection
    size_t total;
};

// Largest delay the scan's test hook may add before a tile publishes: this many
// s_sleep(127) (about 8,000 cycles each), about 4 ms, far below the look-back spin limit of
// 4 million waits of at least 64 cycles each.
constexpr uint32_t kMaxDelaySleeps = 1000;

constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int64_t kScanTile = (int64_t)kScanThreads * kScanItems;
// Largest hidden size of the fused projection: a 256-row operand tile (256 * d * 2
// bytes) must fit the 32-bit range of one buffer descriptor.
constexpr int32_t kMaxFusedD = 65536;

WsLayout ws_layout(int64_t n_rollouts, int64_t n_tokens, int64_t n_units, int64_t fused_partials);

__device__ inline void raise_flag(uint32_t *flags, uint32_t bits) {
    if (flags) atomicOr(flags, bits);
}

// ---- launchers (one per source file); all asynchronous on `stream` ----

// score.hip
hipError_t launch_row_domain(const stride_layout &L, int32_t n_teachers, uint8_t *row_dom,
                             uint32_t *flags, hipStream_t stream);
hipError_t launch_score_rows(int32_t dtype, const PtrTable &teachers, int32_t n_teachers,
                             const uint8_t *row_dom, const void *student, const int32_t *ids,
                             float *logp_t, float *logp_s, int64_t n_rows, int32_t vocab,
                             int64_t ld, uint32_t *flags, hipStream_t stream);

hipError_t launch_score_pairs(int32_t dtype, const PtrTable &teachers, int32_t n_teachers,
                              const uint8_t *row_dom, const void *student, const int32_t *ids,
                              float *logp_t, float *logp_s, float *kl_full, int64_t n_rows,
                              int32_t vocab, int64_t ld, uint32_t *flags, hipStream_t stream);

// turn.hip
hipError_t launch_turn_mean(const stride_layout &L, const float *logp_t, const float *logp_s,
                            float *kl, double *turn_mean, uint32_t *flags, hipStream_t stream);

// scan.hip
hipError_t launch_stop(const stride_layout &L, int32_t unit, const void *values,
                       const DomainTable &lambda, int32_t n_dom, const int32_t *start,
                       double *cum, int32_t *stop_unit, int64_t *retained, uint32_t *flags,
                       void *ws, hipStream_t stream);
// Device address of this GPU's fixed scratch array (STRIDE_NOALLOC_SCRATCH_BYTES), looked
// up on the first call per device.
hipError_t noalloc_scratch(void **ptr);

// fused.hip
size_t fused_ws_bytes(int64_t n_rows, int32_t vocab);
hipError_t launch_fused_teacher(const uint16_t *h, const uint16_t *w, const int32_t *ids,
                                float *logp_t, int64_t n_rows, int32_t vocab, int32_t d,
                                uint32_t *flags, void *ws, hipStream_t stream);

// grad.hip
hipError_t launch_opd_grad(const stride_layout &L, int32_t unit, int32_t dtype, int32_t vocab,
                           int64_t ld, const void *student, const int32_t *ids,
                           const float *logp_t, const float *logp_s, const int32_t *start,
                           const int32_t *stop, float scale, void *grad, float *loss,
                           uint32_t *flags, uint8_t *mask, hipStream_t stream);

hipError_t launch_stop_step(int32_t n_active, const int32_t *rid, const int64_t *new_off,
                            int32_t unit, const void *values, const int32_t *domain,
                            const DomainTable &lambda, int32_t n_dom, double *state_cum,
                            int32_t *state_units, int32_t *stop_unit, uint32_t *flags,
                            hipStream_t stream);

// probe.hip
hipError_t launch_probe_flat(const void *a, const void *b, int64_t n_bytes, uint32_t *sink,
                             int64_t sink_len, hipStream_t stream);
hipError_t launch_probe_copy(const void *src, void *dst, const uint8_t *mask, int64_t n_rows,
                             int64_t row_bytes, int64_t copy_bytes, hipStream_t stream);
hipError_t launch_probe_read(const void *a, const void *b, int64_t n_rows, int64_t row_bytes,
                             int64_t read_bytes, uint32_t *sink, hipStream_t stream);

// restart.hip
hipError_t launch_restart(const stride_layout &L, int32_t unit, const void *values,
                          const int32_t *stop_unit, const DomainTable &alpha, int32_t n_dom,
                          const uint8_t *mask, int32_t *k_star, int32_t *k0, int32_t *k_max,
                          uint32_t *flags, hipStream_t stream);

}  // namespace stride
