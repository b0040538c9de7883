// synth.hip -- seeded synthetic logits, hidden states and weights, on the host
// and on the device, bit-identical.
//
// This is the only code the float64 oracle and the HIP library have in common:
// it makes inputs and holds none of the method's arithmetic.  The tests fill
// host arrays for the oracle with synth_fill_host and device buffers for the
// library with synth_fill_device; both evaluate the same element function.
//
// Element definition.  For tensor stream s, row i, column v (0 <= v < cols):
//   key  = mix(seed + mix(s + 1))
//   c    = 3 (i cols + v)
//   w_j  = mix(key + (c + j + 1) * GAMMA)                        j = 0, 1, 2
//   S    = sum of the twelve 16-bit fields of w_0, w_1, w_2
//   z    = (S - 393210) * 2^-16          (exact: Irwin-Hall sum of 12 uniforms,
//                                          mean 0, variance ~1, range +-6)
//   x    = sigma * z                      (one binary32 multiply)
//   x    = x + boost[i]   if v == tok[i]  (one binary32 add)
//   out  = x as binary32, or x rounded to bf16 (nearest, ties to even)
// mix() is the splitmix64 output function and GAMMA its increment (Steele, Lea
// and Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014),
// so w_j is the splitmix64 sequence started at `key`, read at position c + j.
// The file is compiled with -ffp-contract=off so that no multiply-add is fused.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

constexpr uint64_t GAMMA = 0x9E3779B97F4A7C15ull;

__host__ __device__ inline uint64_t mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__host__ __device__ inline uint32_t sum16(uint64_t w) {
    return (uint32_t)(w & 0xFFFF) + (uint32_t)((w >> 16) & 0xFFFF) + (uint32_t)((w >> 32) & 0xFFFF) +
           (uint32_t)(w >> 48);
}

__host__ __device__ inline float element(uint64_t key, int64_t row, int64_t col, int64_t cols,
                                         float sigma, int32_t tok, float boost) {
    uint64_t c = 3ull * ((uint64_t)row * (uint64_t)cols + (uint64_t)col);
    uint32_t s = sum16(mix(key + (c + 1) * GAMMA)) + sum16(mix(key + (c + 2) * GAMMA)) +
                 sum16(mix(key + (c + 3) * GAMMA));
    float z = (float)((int32_t)s - 393210) * (1.0f / 65536.0f);
    float x = sigma * z;
    if (col == (int64_t)tok) x = x + boost;
    return x;
}

__host__ __device__ inline uint16_t to_bf16(float f) {
    uint32_t u;
    __builtin_memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__host__ __device__ inline uint64_t stream_key(uint64_t seed, uint64_t stream) {
    return mix(seed + mix(stream + 1));
}

// One thread per (row, group of 8 columns).
__global__ __launch_bounds__(256) void fill_kernel(void *dst, int dtype, int64_t ld, int64_t cols,
                                                   int64_t row0, int64_t n_rows, uint64_t key,
                                                   float sigma, const int32_t *tok,
                                                   const float *boost) {
    int64_t groups = (cols + 7) / 8;
    int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t i = blockIdx.y + (int64_t)gridDim.y * blockIdx.z;
    if (g >= groups || i >= n_rows) return;
    int32_t t = tok ? tok[i] : -1;
    float b = boost ? boost[i] : 0.0f;
    int64_t v0 = g * 8;
    for (int k = 0; k < 8; ++k) {
        int64_t v = v0 + k;
        if (v >= cols) break;
        float x = element(key, row0 + i, v, cols, sigma, t, b);
        if (dtype == 0)
            ((uint16_t *)dst)[i * ld + v] = to_bf16(x);
        else
            ((float *)dst)[i * ld + v] = x;
    }
}

}  // namespace

extern "C" {

// Fill rows row0 .. row0+n_rows-1 of a [*, cols] tensor into dst (dst points at
// row row0; row stride ld elements; dtype 0 = bf16 bits, 1 = float).  tok and
// boost are per filled row (index i = 0 .. n_rows-1) and may be NULL (no
// boost).  Host memory; single-threaded (callers split rows across threads).
// Returns 0, or -1 on a bad argument.
int synth_fill_host(void *dst, int dtype, int64_t ld, int64_t cols, int64_t row0, int64_t n_rows,
                    uint64_t seed, uint64_t stream, float sigma, const int32_t *tok,
                    const float *boost) {
    if (!dst || ld < cols || cols < 0 || n_rows < 0 || (dtype != 0 && dtype != 1)) return -1;
    uint64_t key = stream_key(seed, stream);
    for (int64_t i = 0; i < n_rows; ++i) {
        int32_t t = tok ? tok[i] : -1;
        float b = boost ? boost[i] : 0.0f;
        for (int64_t v = 0; v < cols; ++v) {
            float x = element(key, row0 + i, v, cols, sigma, t, b);
            if (dtype == 0)
                ((uint16_t *)dst)[i * ld + v] = to_bf16(x);
            else
                ((float *)dst)[i * ld + v] = x;
        }
    }
    return 0;
}

// Same rows on the device, asynchronously on `stream_h`; tok and boost are
// device arrays.  Returns 0, -1 on a bad argument, or the HIP error code.
int synth_fill_device(void *dst, int dtype, int64_t ld, int64_t cols, int64_t row0, int64_t n_rows,
                      uint64_t seed, uint64_t stream, float sigma, const int32_t *tok,
                      const float *boost, hipStream_t stream_h) {
    if (!dst || ld < cols || cols < 0 || n_rows < 0 || (dtype != 0 && dtype != 1)) return -1;
    if (n_rows == 0 || cols == 0) return 0;
    int64_t groups = (cols + 7) / 8;
    int64_t ny = n_rows < 65535 ? n_rows : 65535;
    int64_t nz = (n_rows + ny - 1) / ny;
    if (nz > 65535) return -1;
    dim3 grid((unsigned)((groups + 255) / 256), (unsigned)ny, (unsigned)nz);
    hipLaunchKernelGGL(fill_kernel, grid, dim3(256), 0, stream_h, dst, dtype, ld, cols, row0,
                       n_rows, stream_key(seed, stream), sigma, tok, boost);
    return (int)hipGetLastError();
}

}  // extern "C"
