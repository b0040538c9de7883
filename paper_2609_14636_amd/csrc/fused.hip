// fused.hip -- teacher log-probabilities from the output projection, logits never stored.
//
// Eq. (1) (Sec. 3.1) with the teacher's logits z = h W^T, h the teacher's final
// hidden state of the row ([N, d] bf16) and W its lm_head weight as stored by a
// linear layer ([V, d] bf16, row v = the weights of vocabulary entry v):
// log pi_T(y) = z_y - log sum_v exp(z_v).  The [N, V] logits (40 GB at the
// fused workload) exist only tile by tile in registers.
//
// Kernel 1 (MFMA): a 256 x 256 tile of z per workgroup of eight waves, two per
//   SIMD, each wave holding a 128 (vocabulary) x 64 (token) fp32 accumulator
//   (32 v_mfma_f32_16x16x32_bf16 tiles, 128 registers).  The 16 x 16 form reads and
//   writes half as many accumulator registers per product as the 32 x 32 one, and
//   under this load the chip's power, not its issue rate, sets the pace.  The waves
//   form two groups of four (one wave per SIMD) that alternate every 32-wide K step: while one
//   group multiplies from registers, the other reads its next fragments from LDS
//   and issues loads, then a barrier swaps them (ping-pong), so each SIMD's matrix
//   unit always has a wave with work.  K = d streams in 64-wide stages through a
//   ring of five 32 KB LDS buffers (the whole 160 KB LDS), each holding one
//   operand of one stage, filled by direct buffer->LDS loads (buffer_load_dwordx4
//   ... lds, no register staging): H of stage j in buffer 2j mod 5, W in 2j+1 mod 5.
//   Every memory phase issues one operand's loads -- W(j+1) in the first half of
//   stage j, H(j+2) in the second -- so the loads are spread evenly over the
//   phases and each has two to four phases to land.  Eight lanes load one row's
//   128 bytes, a whole cache line, and rows are XOR-swizzled so the 16-byte
//   fragment reads are free of bank conflicts.  No vector ALU work remains in the
//   loop: wave-uniform values are scalar and the fragment addresses are fixed per
//   buffer.  Both operands are K-contiguous, so each MFMA operand is one 16-byte
//   LDS read.  W is the A operand and H the B operand, so each lane's
//   accumulators hold 32 of one token's 128 logits and the lanes l ^ 16, l ^ 32 and
//   l ^ 48 the other 96: the epilogue reduces a token to (max, sum of exp(z - max))
//   with two exchanges and writes it to a partial table [V/128][N] (tokens
//   contiguous).
//   Workgroups are numbered so that the 32 resident on one XCD (dispatch is
//   round-robin over the 8 XCDs) cover a 4 x 8 block of tiles of a 16 x 16
//   super-tile: each XCD's L2 serves every H panel slice to 8 tiles and every
//   W slice to 4.  Super-rows are grouped in bands (up to 128 MiB of H, eight
//   super-rows at d = 2,048) and a band is walked one super-column at a time:
//   the band's H and the current W slab both stay in the 256 MB last-level
//   cache, so each W slab comes from HBM once per band instead of once per
//   super-row.  With fewer than 16 (or 8) row tiles the super-tile is 8 x 32
//   (or 4 x 64) tiles, so every XCD still has tiles.
// Kernel 2: z_y = h . w_y per row (one wave per row, fp32).
// Kernel 3: four waves per 64 rows merge each row's V/128 partials (reads
//   coalesced across rows) and write log pi_T(y) = (z_y - m) - log s.
#include <atomic>

#include "common.hpp"

namespace stride {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#define LDS_PTR(p) ((__attribute__((address_space(3))) void *)(p))

constexpr int kBM = 256, kBN = 256, kBK = 64;      // tile and stage width along K
constexpr int kThreads = 512;                      // eight waves
constexpr int kRowB = kBK * 2;                     // 128 bytes per LDS row
constexpr int kBufB = kBM * kRowB;                 // 32 KB: one operand of one stage
constexpr int kBuffers = 5;                        // LDS ring of operand buffers
constexpr size_t kLdsBytes = (size_t)kBuffers * kBufB;  // 160 KB, the whole LDS
constexpr int kHalf = 128;                         // vocabulary entries per partial
// H bytes a band of super-rows may hold in the 256 MB last-level cache beside the W slab
// it is reading: 128 MiB, eight 4,096-row super-rows at d = 2,048
constexpr int64_t kBandHBytes = 128ll << 20;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;
// Third word of a raw buffer descriptor: 32-bit data format, no swizzle; accesses
// at or beyond num_records bytes return zeros.
constexpr int kBufferFlags = 0x00020000;

struct FusedArgs {
    const uint16_t *h;     // [N, d]
    const uint16_t *w;     // [V, d]
    float2 *partial;       // [n_half, N]
    int64_t n_rows;
    int32_t vocab;
    int32_t d;
    int32_t n_half;
    int32_t tiles_m, tiles_n, super_rows, super_cols;
    int32_t xcd_cols;      // XCD blocks per super-tile row: 2, 4 or 8 (the super-tile is
                           // 32 / xcd_cols row tiles by 8 * xcd_cols vocabulary tiles)
    int32_t band;          // super-rows per band; a band is walked one super-column at a time
};

__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

// 16-byte chunk c of LDS row r is stored at position c ^ swz(r).  The LDS has 64
// banks (256 B per cycle) and serves a 16-byte-per-lane read in four cycles of 16
// lanes; on gfx950 a cycle takes four lane quads of one half-wave, quads 0, 3, 5, 6
// or quads 1, 2, 4, 7 (the quads whose index has even or odd parity; measured with
// the bank-conflict counter).  Rows are 128 B, so a row's place in the 256-byte bank
// row is r % 2.  Fragment lane l reads row l % 16 (of a 16-row block) at chunk
// 4 * hf + l / 16 for the half hf of the stage; over the 16 lanes of either kind of
// cycle the pairs (r % 2, chunk ^ swz(r)) are all distinct, so every read is free of
// conflicts.
__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

// Wait until at most N vector-memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmem() {
    __builtin_amdgcn_s_waitcnt((N & 0xF) | (7 << 4) | (0xF << 8) | ((N >> 4) << 14));
}

// Wait until this wave's LDS reads have returned.
__device__ __forceinline__ void wait_lds() {
    __builtin_amdgcn_s_waitcnt(0xF | (7 << 4) | (0 << 8) | (3 << 14));
}

__device__ __forceinline__ void barrier() {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

__global__ __launch_bounds__(kThreads, 1) void fused_lse_kernel(FusedArgs a) {
    extern __shared__ __attribute__((aligned(1024))) char lds[];
    const int tid = threadIdx.x, lane = tid & 63;
    // wave-uniform values in scalar registers: the LDS-DMA destinations are scalar arithmetic
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = wave >> 2;                   // ping-pong group (one wave per SIMD)
    const int wv = wave & 1, wt = wave >> 1;     // vocabulary half, token quarter

    // ---- tile of this workgroup (XCD-aware order) ----
    const int b = blockIdx.x;
    const int xcd = b & 7, s = b >> 3;
    const int S = s >> 5, q = s & 31;
    const int xc = a.xcd_cols, xr = 8 / xc;
    // super-tile S -> (super-row, super-column): bands of a.band super-rows, each band
    // walked column by column, so a W slab read from HBM serves the whole band from the
    // last-level cache while the band's H stays there too
    const int per_band = a.band * a.super_cols;
    const int bi = S / per_band, r0 = bi * a.band, idx = S - bi * per_band;
    const int rows_b = (a.super_rows - r0) < a.band ? (a.super_rows - r0) : a.band;
    const int sr = r0 + idx % rows_b, sc = idx / rows_b;
    const int tm = sr * (4 * xr) + (xcd / xc) * 4 + (q & 3);
    const int tn = sc * (8 * xc) + (xcd % xc) * 8 + (q >> 2);
    if (tm >= a.tiles_m || tn >= a.tiles_n) return;
    const int64_t m0 = (int64_t)tm * kBM;
    const int64_t n0 = (int64_t)tn * kBN;
    const int d = a.d, ns = d / kBK;

    // ---- direct global -> LDS loads (buffer_load_dwordx4 ... lds): for each operand and
    // stage, each wave fills 32 rows of that operand's buffer, 8 rows per instruction (lane l
    // -> row l >> 3, position l & 7 of the swizzled row).  Each operand's descriptor spans
    // only the rows of this tile that exist, so rows past N or V read as zeros (their results
    // are never used) and no load can leave the operand.  Lane offsets are 32-bit; the K
    // position goes in the scalar offset.
    const int64_t h_rows = (a.n_rows - m0) < kBM ? (a.n_rows - m0) : kBM;
    const int64_t w_rows = (a.vocab - n0) < kBN ? (a.vocab - n0) : kBN;
    const __amdgpu_buffer_rsrc_t rh = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(a.h + m0 * d), (short)0, (int)(h_rows * d * 2), kBufferFlags);
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(a.w + n0 * d), (short)0, (int)(w_rows * d * 2), kBufferFlags);
    const int lr = lane >> 3, lp = lane & 7;
    int voff[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int R = 32 * wave + 8 * i + lr;
        voff[i] = (R * d + ((lp ^ swz(R)) * 8)) * 2;
    }
    auto issue = [&](const __amdgpu_buffer_rsrc_t &rsrc, int j, int buf) __attribute__((always_inline)) {
        char *dst = lds + buf * kBufB;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rsrc, LDS_PTR(dst + (32 * wave + 8 * i) * kRowB), 16, voff[i], j * kRowB, 0, 0);
    };

    // ---- MFMA fragments: W is the A operand and H the B operand of 16 x 16 x 32 products,
    // so lane l's accumulators hold token jj*16 + l%16 and 4 vocabulary entries of each
    // 16-row block.  Lane l reads row l % 16 of a block at chunk 4*hf + l/16; the fragment
    // addresses are fixed per buffer pair {0,1}, {2,3}, {4} and stage half: the buffer's
    // place in its pair and the 16-row block go in the read's immediate offset.
    const int fr = lane & 15, kg = lane >> 4;
    int wb[3][2], hb[3][2];
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
        const int f = fr * kRowB + (((4 * hf + kg) ^ swz(fr)) * 16);
#pragma unroll
        for (int g = 0; g < 3; ++g) {
            wb[g][hf] = g * 2 * kBufB + (wv * 128) * kRowB + f;
            hb[g][hf] = g * 2 * kBufB + (wt * 64) * kRowB + f;
            // opaque to the compiler: it would otherwise fold the pair's 64 KB step into the
            // reads' offsets, overflow their 16-bit immediate and keep a register per read
            asm volatile("" : "+v"(wb[g][hf]), "+v"(hb[g][hf]));
        }
    }
    bf16x8 FA[8], FB[4];
    f32x4 acc[8][4];  // the first K step's MFMAs start from zero, so no vector moves clear it

    // One 32-wide K step of this wave (half hf of stage j, whose H and W operands sit in
    // buffers hbuf and wbuf): fragments from LDS and one operand's loads, then the MFMAs.
    // The two groups are one phase apart, so every barrier is met by all eight waves: group
    // 0 at the end of a memory phase when group 1 ends a compute phase, and the other way
    // round.  The first half-stage loads W(j+1) into the buffer of H(j-1); the second loads
    // H(j+2) into the buffer of W(j-1) (both read for the last time in stage j-1) and waits
    // until this wave's shares of H(j+1) and W(j+1) have landed, so stage j+1 is complete in
    // LDS at the barrier that ends stage j.
    // may_start: this call site can be the tile's first K step (stage 0 sits at ring position 0),
    // whose MFMAs take zero as their accumulator input.
    auto phase = [&](int j, int hf, int hbuf, int wbuf, bool may_start) __attribute__((always_inline)) {
#pragma unroll
        for (int t = 0; t < 8; ++t)
            FA[t] = *reinterpret_cast<const bf16x8 *>(lds + wb[wbuf >> 1][hf] + (wbuf & 1) * kBufB +
                                                      t * 16 * kRowB);
#pragma unroll
        for (int t = 0; t < 4; ++t)
            FB[t] = *reinterpret_cast<const bf16x8 *>(lds + hb[hbuf >> 1][hf] + (hbuf & 1) * kBufB +
                                                      t * 16 * kRowB);
        if (hf == 0) {
            const int nb = wbuf + 2 >= kBuffers ? wbuf + 2 - kBuffers : wbuf + 2;
            if (j + 1 < ns) issue(rw, j + 1, nb);
        } else {
            const int nb = hbuf + 4 >= kBuffers ? hbuf + 4 - kBuffers : hbuf + 4;
            if (j + 2 < ns) {
                issue(rh, j + 2, nb);
                wait_vmem<4>();
            } else {
                wait_vmem<0>();
            }
        }
        wait_lds();
        barrier();
        if (may_start && j == 0) {
            const f32x4 zero = {};
#pragma unroll
            for (int i = 0; i < 8; ++i)
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
                    acc[i][jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(FA[i], FB[jj], zero, 0, 0, 0);
        } else {
#pragma unroll
            for (int i = 0; i < 8; ++i)
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
                    acc[i][jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(FA[i], FB[jj], acc[i][jj], 0, 0, 0);
        }
        barrier();
    };
    // H(j) lives in buffer 2j mod 5 and W(j) in buffer 2j+1 mod 5; r = j mod 5 is a
    // compile-time value at every call, so every buffer index is.
    auto stage = [&](int j, int r) __attribute__((always_inline)) {
        const int hbuf = (2 * r) % kBuffers, wbuf = (2 * r + 1) % kBuffers;
        phase(j, 0, hbuf, wbuf, r == 0);
        phase(j, 1, hbuf, wbuf, false);
    };
    // prologue: H(0), W(0), H(1) in flight, H(0) and W(0) landed
    issue(rh, 0, 0);
    issue(rw, 0, 1);
    if (ns > 1) {
        issue(rh, 1, 2);
        wait_vmem<4>();
    } else {
        wait_vmem<0>();
    }
    barrier();
    if (grp == 1) barrier();  // group 1 runs one phase behind
    int j = 0;
    for (; j + 4 < ns; j += 5) {
        stage(j, 0);
        stage(j + 1, 1);
        stage(j + 2, 2);
        stage(j + 3, 3);
        stage(j + 4, 4);
    }
    if (j < ns) stage(j, 0);  // j is a multiple of 5 here
    if (j + 1 < ns) stage(j + 1, 1);
    if (j + 2 < ns) stage(j + 2, 2);
    if (j + 3 < ns) stage(j + 3, 3);
    if (grp == 0) barrier();  // both groups meet the same number of barriers

    // ---- epilogue: per token of this wave, (max, sum exp(z - max)) over its 128 entries;
    // lane l holds entries i*16 + 4*(l/16) + e of token jj*16 + l%16, and the lanes l, l^16,
    // l^32, l^48 that share a token combine theirs with two exchanges ----
    const int q4 = lane >> 4;
    const int64_t v_base = n0 + wv * 128;
    const int vlim = (int)((a.vocab - v_base) < 128 ? (a.vocab - v_base) : 128);  // valid entries
    const int hidx = tn * 2 + wv;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
        if (vlim < 128) {
#pragma unroll
            for (int i = 0; i < 8; ++i)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (i * 16 + q4 * 4 + e >= vlim) acc[i][jj][e] = -INFINITY;
        }
        float m = acc[0][jj][0];
#pragma unroll
        for (int x = 1; x < 32; ++x) m = fmaxf(m, acc[x >> 2][jj][x & 3]);
        m = fmaxf(m, __shfl_xor(m, 16, 64));
        m = fmaxf(m, __shfl_xor(m, 32, 64));
        const float ref = (m == -INFINITY) ? 0.0f : m;
        const float mref = ref * kLog2e;
        float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
        for (int x = 0; x < 32; x += 2) {
            s0 += ex2(__builtin_fmaf(acc[x >> 2][jj][x & 3], kLog2e, -mref));
            s1 += ex2(__builtin_fmaf(acc[(x + 1) >> 2][jj][(x + 1) & 3], kLog2e, -mref));
        }
        float sum = s0 + s1;
        sum += __shfl_xor(sum, 16, 64);
        sum += __shfl_xor(sum, 32, 64);
        const int64_t row = m0 + wt * 64 + jj * 16 + (lane & 15);
        if (q4 == 0 && hidx < a.n_half && row < a.n_rows)
            a.partial[(int64_t)hidx * a.n_rows + row] = make_float2(m, sum);
    }
}

// z_y = h . w_y, one wave per row, fp32.
__global__ __launch_bounds__(256) void fused_gather_kernel(const uint16_t *h, const uint16_t *w,
                                                           const int32_t *ids, float *zy,
                                                           int64_t n_rows, int32_t vocab, int32_t d) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= n_rows) return;
    const int32_t y = ids[row];
    if (y < 0 || y >= vocab) {
        if (lane == 0) zy[row] = __builtin_nanf("");
        return;
    }
    const u32x4 *hp = reinterpret_cast<const u32x4 *>(h + row * d);
    const u32x4 *wp = reinterpret_cast<const u32x4 *>(w + (int64_t)y * d);
    float acc = 0.0f;
    for (int c = lane; c < d / 8; c += 64) {
        const u32x4 x = hp[c], z = wp[c];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            acc = __builtin_fmaf(__uint_as_float(x[e] << 16), __uint_as_float(z[e] << 16), acc);
            acc = __builtin_fmaf(__uint_as_float(x[e] & 0xFFFF0000u), __uint_as_float(z[e] & 0xFFFF0000u), acc);
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
    if (lane == 0) zy[row] = acc;
}

// Fold one partial (max p.x, sum p.y of exp(z - p.x)) into a running (m, s).
__device__ __forceinline__ void fold_partial(float &m, float &s, const float2 p) {
    const float mn = fmaxf(m, p.x);
    const float ref = (mn == -INFINITY) ? 0.0f : mn;
    s = s * ex2((m - ref) * kLog2e) + p.y * ex2((p.x - ref) * kLog2e);
    m = mn;
}

constexpr int kMergeRows = 64;   // rows per workgroup, one per lane
constexpr int kMergeSplit = 4;   // waves per workgroup, each folding every 4th partial

// Merge the V/128 partials of each row and finish log pi_T(y).  Wave w of a workgroup
// folds partials w, w+4, w+8, ... of its 64 rows (each load is 64 consecutive rows,
// 512 contiguous bytes, eight loads in flight); the four wave results are combined in
// LDS in wave order, so the result does not depend on timing.
__global__ __launch_bounds__(256) void fused_merge_kernel(const float2 *partial, const float *zy,
                                                          const int32_t *ids, float *logp_t,
                                                          int64_t n_rows, int32_t n_half,
                                                          int32_t vocab, uint32_t *flags) {
    __shared__ float2 red[kMergeSplit][kMergeRows];
    const int r = threadIdx.x & (kMergeRows - 1), sp = threadIdx.x / kMergeRows;
    const int64_t row = (int64_t)blockIdx.x * kMergeRows + r;
    float m = -INFINITY, s = 0.0f;
    if (row < n_rows) {
        const float2 *col = partial + row;
        int j = sp;
        constexpr int U = 8;
        for (; j + (U - 1) * kMergeSplit < n_half; j += U * kMergeSplit) {
            float2 p[U];
#pragma unroll
            for (int u = 0; u < U; ++u) p[u] = col[(int64_t)(j + u * kMergeSplit) * n_rows];
#pragma unroll
            for (int u = 0; u < U; ++u) fold_partial(m, s, p[u]);
        }
        for (; j < n_half; j += kMergeSplit) fold_partial(m, s, col[(int64_t)j * n_rows]);
    }
    red[sp][r] = make_float2(m, s);
    __syncthreads();
    if (sp != 0 || row >= n_rows) return;
#pragma unroll
    for (int k = 1; k < kMergeSplit; ++k) fold_partial(m, s, red[k][r]);
    const int32_t y = ids[row];
    uint32_t bad = 0;
    if (!((m > -INFINITY) && (m < INFINITY) && (s > 0.0f) && (s < INFINITY))) bad |= STRIDE_FLAG_NONFINITE;
    if (y < 0 || y >= vocab) bad |= STRIDE_FLAG_TOKEN_OOB;
    const float z = zy[row];
    if (!bad && !(z > -INFINITY && z < INFINITY)) bad |= STRIDE_FLAG_NONFINITE;
    if (bad) {
        raise_flag(flags, bad);
        logp_t[row] = __builtin_nanf("");
    } else {
        // z_y comes from its own fp32 dot product and (m, s) from the MFMA accumulators, so
        // their rounding differs by ~1e-6 relative; a log-probability is at most 0, and
        // clamping there only moves a rounding excess toward the true value.
        logp_t[row] = fminf(0.0f, (z - m) - __builtin_amdgcn_logf(s) * kLn2);
    }
}

}  // namespace

namespace {

#ifdef STRIDE_FUSED_BAND_HOOK
std::atomic<int32_t> g_band_override{0};  // super-rows per band; 0: the library's choice
#endif

// The projection kernel's dynamic LDS (160 KB) is above the default limit; the limit is
// raised once per device, so later calls (and calls under stream capture) make no
// attribute call.
hipError_t ensure_lds_limit() {
    static std::atomic<uint64_t> done{0};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const uint64_t bit = (dev >= 0 && dev < 64) ? (1ull << dev) : 0;
    if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(fused_lse_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsBytes);
    if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_release);
    return e;
}

}  // namespace

size_t fused_ws_bytes(int64_t n_rows, int32_t vocab) {
    const int64_t n_half = ((int64_t)vocab + kHalf - 1) / kHalf;
    return (size_t)n_half * n_rows * sizeof(float2) + (size_t)n_rows * sizeof(float) + 256;
}

hipError_t launch_fused_teacher(const uint16_t *h, const uint16_t *w, const int32_t *ids,
                                float *logp_t, int64_t n_rows, int32_t vocab, int32_t d,
                                uint32_t *flags, void *ws, hipStream_t stream) {
    if (n_rows == 0) return hipSuccess;
    FusedArgs a;
    a.h = h;
    a.w = w;
    a.n_rows = n_rows;
    a.vocab = vocab;
    a.d = d;
    a.n_half = (vocab + kHalf - 1) / kHalf;
    a.tiles_m = (int)((n_rows + kBM - 1) / kBM);
    a.tiles_n = (vocab + kBN - 1) / kBN;
    // Few row tiles (small batches): lay the eight XCD blocks out along V instead, so
    // every XCD still gets work.
    a.xcd_cols = a.tiles_m >= 16 ? 2 : (a.tiles_m >= 8 ? 4 : 8);
    const int xr = 8 / a.xcd_cols;
    a.super_cols = (a.tiles_n + 8 * a.xcd_cols - 1) / (8 * a.xcd_cols);
    const int super_rows = (a.tiles_m + 4 * xr - 1) / (4 * xr);
    a.super_rows = super_rows;
    const int64_t h_super_row = (int64_t)4 * xr * kBM * d * 2;  // H bytes of one super-row
    int64_t band = kBandHBytes / h_super_row;
#ifdef STRIDE_FUSED_BAND_HOOK
    if (const int32_t o = g_band_override.load()) band = o;
#endif
    a.band = (int)(band < 1 ? 1 : (band > super_rows ? super_rows : band));
    a.partial = static_cast<float2 *>(ws);
    float *zy = reinterpret_cast<float *>(static_cast<char *>(ws) +
                                          (size_t)a.n_half * n_rows * sizeof(float2));
    hipError_t e = ensure_lds_limit();
    if (e != hipSuccess) return e;
    const int64_t blocks = (int64_t)super_rows * a.super_cols * 256;
    if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;  // grid past the 32-bit limit
    hipLaunchKernelGGL(fused_lse_kernel, dim3((unsigned)blocks), dim3(kThreads), kLdsBytes, stream, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fused_gather_kernel, dim3((unsigned)((n_rows + 3) / 4)), dim3(256), 0, stream,
                       h, w, ids, zy, n_rows, vocab, d);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fused_merge_kernel, dim3((unsigned)((n_rows + kMergeRows - 1) / kMergeRows)),
                       dim3(kMergeRows * kMergeSplit), 0,
                       stream, a.partial, zy, ids, logp_t, n_rows, a.n_half, vocab, flags);
    return hipGetLastError();
}

}  // namespace stride

extern "C" stride_status stride_debug_fused_band(int32_t band) {
#ifdef STRIDE_FUSED_BAND_HOOK
    if (band < 0) return STRIDE_ERR_INVALID_ARG;
    stride::g_band_override.store(band);
    return STRIDE_OK;
#else
    (void)band;
    return STRIDE_ERR_UNSUPPORTED;
#endif
}
