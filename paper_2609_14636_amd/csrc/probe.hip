// probe.hip -- streaming-read reference for the scoring kernel's roofline.
//
// Not part of the method: it reads rows exactly as the scoring kernel does (one
// wavefront per row, 16-byte non-temporal loads with eight per lane in flight,
// rows of the two matrices interleaved item by item) and does no arithmetic
// beyond an XOR, so its rate is the read bandwidth this access pattern reaches
// on the device.  The scoring kernel's bandwidth divided by this rate says how
// much of the reachable bandwidth the softmax arithmetic leaves on the table.
#include "common.hpp"

namespace stride {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kUnroll = 8;

__global__ __launch_bounds__(256) void probe_read_kernel(const char *a, const char *b,
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

}  // namespace

hipError_t launch_probe_read(const void *a, const void *b, int64_t n_rows, int64_t row_bytes,
                             int64_t read_bytes, uint32_t *sink, hipStream_t stream) {
    const int64_t items = b ? 2 * n_rows : n_rows;
    if (items == 0) return hipSuccess;
    const int64_t blocks = (items + 3) / 4;
    hipLaunchKernelGGL(probe_read_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                       static_cast<const char *>(a), static_cast<const char *>(b), n_rows, row_bytes,
                       read_bytes / 16, sink);
    return hipGetLastError();
}

}  // namespace stride
