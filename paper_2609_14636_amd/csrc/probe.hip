// probe.hip -- streaming references for the rooflines of the row kernels.
//
// Not part of the method.  probe_read_kernel reads rows exactly as the scoring
// kernel does (one wavefront per row, 16-byte non-temporal loads with eight per
// lane in flight, rows of the two matrices interleaved item by item) and does no
// arithmetic beyond an XOR, so its rate is the read bandwidth this access pattern
// reaches on the device; the scoring kernel's bandwidth divided by this rate says
// how much of the reachable bandwidth the softmax arithmetic leaves on the table.
// probe_flat_kernel reads the same bytes as one contiguous range per matrix in a
// grid-stride order (the plainest streaming order), to tell the access pattern
// apart from the footprint.  probe_copy_kernel moves rows as the OPD gradient
// kernel does: eight wavefronts per row (wavefront w takes the row's 4-load chunks
// w, w + 8, ...), a 16-byte non-temporal load and store per word; rows whose mask
// byte is 0 are written as zeros without being read.
#include "common.hpp"

namespace stride {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kUnroll = 8;

__global__ __launch_bounds__(kRowThreads) void probe_read_kernel(const char *a, const char *b,
                                                         int64_t n_rows, int64_t row_bytes,
                                                         int64_t nvec, uint32_t *sink) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t item = (int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave);
    const int64_t n_items = b ? 2 * n_rows : n_rows;
    if (item >= n_items) return;
    const bool second = b && (item & 1);
    const int64_t row = b ? (item >> 1) : item;
    const u32x4 *p = reinterpret_cast<const u32x4 *>((second ? b : a) + row * row_bytes);
    uint32_t x = 0;
    int64_t k = 0;
    constexpr int64_t kStep = (int64_t)kUnroll * kWave;
    for (; k + kStep <= nvec; k += kStep) {
        u32x4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) v[u] = __builtin_nontemporal_load(p + k + u * kWave + lane);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) x ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
    }
    for (; k < nvec; k += kWave)
        if (k + lane < nvec) {
            const u32x4 v = __builtin_nontemporal_load(p + k + lane);
            x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
        }
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) x ^= __shfl_xor(x, o, kWave);
    if (lane == 0) sink[item] = x;
}

// Grid-stride over the 16-byte words of a (then b): block i reads words i*256+t,
// (i+G)*256+t, ...; eight loads per lane in flight.
__global__ __launch_bounds__(256) void probe_flat_kernel(const u32x4 *a, const u32x4 *b,
                                                         int64_t nvec, uint32_t *sink) {
    uint32_t x = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int m = 0; m < (b ? 2 : 1); ++m) {
        const u32x4 *p = m ? b : a;
        int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
        for (; i + (kUnroll - 1) * stride < nvec; i += kUnroll * stride) {
            u32x4 v[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) x ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
        }
        for (; i < nvec; i += stride) {
            const u32x4 v = __builtin_nontemporal_load(p + i);
            x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
        }
    }
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) x ^= __shfl_xor(x, o, kWave);
    if ((threadIdx.x & (kWave - 1)) == 0) sink[(int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave] = x;
}

constexpr int kCopyWaves = 8;

__global__ __launch_bounds__(kCopyWaves *kWave) void probe_copy_kernel(const char *src, char *dst,
                                                                       const uint8_t *mask,
                                                                       int64_t n_rows,
                                                                       int64_t row_bytes,
                                                                       int64_t nvec) {
    const int lane = threadIdx.x & (kWave - 1);
    const int sub = threadIdx.x / kWave;
    const int64_t row = blockIdx.x;  // the grid has exactly n_rows workgroups
    if (row >= n_rows) return;
    const u32x4 *s = reinterpret_cast<const u32x4 *>(src + row * row_bytes);
    u32x4 *d = reinterpret_cast<u32x4 *>(dst + row * row_bytes);
    if (mask && !mask[row]) {
        const u32x4 z = {0u, 0u, 0u, 0u};
        for (int64_t k = (int64_t)sub * kWave + lane; k < nvec; k += (int64_t)kCopyWaves * kWave)
            __builtin_nontemporal_store(z, d + k);
        return;
    }
    constexpr int U = 4;
    constexpr int64_t kStep = (int64_t)U * kWave;
    const int64_t nfull = nvec / kStep;
    for (int64_t c = sub; c < nfull; c += kCopyWaves) {
        const int64_t k = c * kStep;
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(s + k + u * kWave + lane);
#pragma unroll
        for (int u = 0; u < U; ++u) __builtin_nontemporal_store(v[u], d + k + u * kWave + lane);
    }
    for (int64_t k = nfull * kStep + (int64_t)sub * kWave; k < nvec; k += (int64_t)kCopyWaves * kWave)
        if (k + lane < nvec) __builtin_nontemporal_store(__builtin_nontemporal_load(s + k + lane), d + k + lane);
}

}  // namespace

hipError_t launch_probe_flat(const void *a, const void *b, int64_t n_bytes, uint32_t *sink,
                             int64_t sink_len, hipStream_t stream) {
    if (n_bytes == 0) return hipSuccess;
    // 2048 workgroups of four waves (eight per CU) or fewer when the sink is shorter
    int64_t blocks = sink_len / 4;
    if (blocks > 2048) blocks = 2048;
    if (blocks < 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL(probe_flat_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                       static_cast<const u32x4 *>(a), static_cast<const u32x4 *>(b), n_bytes / 16,
                       sink);
    return hipGetLastError();
}

hipError_t launch_probe_copy(const void *src, void *dst, const uint8_t *mask, int64_t n_rows,
                             int64_t row_bytes, int64_t copy_bytes, hipStream_t stream) {
    if (n_rows == 0) return hipSuccess;
    hipLaunchKernelGGL(probe_copy_kernel, dim3((unsigned)n_rows), dim3(kCopyWaves * kWave), 0, stream,
                       static_cast<const char *>(src), static_cast<char *>(dst), mask, n_rows,
                       row_bytes, copy_bytes / 16);
    return hipGetLastError();
}

hipError_t launch_probe_read(const void *a, const void *b, int64_t n_rows, int64_t row_bytes,
                             int64_t read_bytes, uint32_t *sink, hipStream_t stream) {
    const int64_t items = b ? 2 * n_rows : n_rows;
    if (items == 0) return hipSuccess;
    constexpr int kRowsPerBlock = kRowThreads / kWave;
    const int64_t blocks = (items + kRowsPerBlock - 1) / kRowsPerBlock;
    hipLaunchKernelGGL(probe_read_kernel, dim3((unsigned)blocks), dim3(kRowThreads), 0, stream,
                       static_cast<const char *>(a), static_cast<const char *>(b), n_rows, row_bytes,
                       read_bytes / 16, sink);
    return hipGetLastError();
}

}  // namespace stride
