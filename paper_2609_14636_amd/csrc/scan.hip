// scan.hip -- the early-stop test: per-rollout cumulative sums and first crossing.
//
// Eq. (5) (Sec. 4.1): stop at the first unit K* whose cumulative value is
// strictly below lambda; with a reused prefix of K0 units the sum starts at
// unit K0 (Sec. 4.1, prefix-buffer synergy; Algorithm 1).  Units are turns
// (values = lbar_k, Eq. 4) or tokens (values = teacher log-probabilities, the
// single-turn variant of Sec. 5.5), so one rollout can hold tens of thousands
// of units.
//
// Single-pass segmented scan (Merrill and Garland, "Single-pass Parallel Prefix
// Scan with Decoupled Look-back", 2016), specialised for determinism:
//   1. A workgroup takes the next tile id from a counter (tiles start in id
//      order, so every tile waited on is already running: forward progress).
//   2. It loads 2048 units, zeroes those before K0, and scans them in double
//      (per-thread sequential, then a fixed shuffle tree, then waves in order),
//      with the segmented operator (f1,v1)+(f2,v2) = (f1|f2, f2 ? v2 : v1+v2).
//   3. It publishes its aggregate (value after its last rollout start, and
//      whether one occurs) with a release store, before waiting on anything.
//   4. If its first unit continues a rollout, it looks back over predecessor
//      aggregates only, nearest first, until the tile holding that rollout's
//      start.  Inclusive prefixes are never used, so every sum is associated
//      in the same order on every run: cum is bit-reproducible.
//   5. The first crossing per rollout is an integer min, reduced in LDS and
//      then with one global atomicMin per rollout per tile.
// Waits are bounded: past the spin limit the tile gives up, raises
// STRIDE_FLAG_SPIN_LIMIT and writes NaN, so no wave can hang.
#include <atomic>
#include <climits>
#include <mutex>

#include "common.hpp"

namespace stride {
namespace {

constexpr int kSlots = 256;            // rollouts per tile reduced in LDS
constexpr uint32_t kSpinLimit = 1u << 22;

struct StopArgs {
    stride_layout L;
    DomainTable lambda;
    int32_t n_dom;
    int32_t unit;
    int64_t n_units;
    int64_t n_tiles;
    const void *values;
    const int32_t *start;
    const int64_t *unit_off;  // [R+1] in the workspace
    double *cum;
    int32_t *stop_unit;
    int64_t *retained;
    uint32_t *counter;
    TileDesc *desc;
    uint32_t *flags;
    // Test hook (the library built with STRIDE_SCAN_DELAY_HOOK only): tiles picked by a
    // seeded hash sleep a bounded time before publishing their aggregate, so successors
    // must wait on unpublished descriptors.  Zero in the product build.
    uint64_t delay_seed;
    uint32_t delay_one_in;
    uint32_t delay_sleeps;
    // Test hook, same build only: a look-back wait bound other than kSpinLimit (0: kSpinLimit),
    // so that the give-up path can be forced from the host.
    uint32_t spin_limit;
};

#ifdef STRIDE_SCAN_DELAY_HOOK
std::atomic<uint64_t> g_delay_seed{0};
std::atomic<uint32_t> g_delay_one_in{0};
std::atomic<uint32_t> g_delay_sleeps{0};
std::atomic<uint32_t> g_spin_limit{0};
#endif

// unit_off, stop_unit sentinels, descriptor reset, tile counter reset.
__global__ __launch_bounds__(256) void stop_prep_kernel(StopArgs a, int64_t *unit_off) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t R = a.L.n_rollouts, T = a.L.n_turns;
    if (i <= R) {
        int64_t t = a.L.rollout_turn_off[i];
        bool bad = t < 0 || t > T;
        if (i == 0 && t != 0) bad = true;
        if (i == R && t != T) bad = true;
        if (i < R && a.L.rollout_turn_off[i + 1] < t) bad = true;
        t = t < 0 ? 0 : (t > T ? T : t);
        unit_off[i] = (a.unit == STRIDE_UNIT_TURN) ? t : a.L.turn_tok_off[t];
        if (bad) raise_flag(a.flags, STRIDE_FLAG_BAD_OFFSETS);
    }
    if (i < R) a.stop_unit[i] = INT_MAX;
    if (i < a.n_tiles) {
        a.desc[i].status = 0;
        a.desc[i].head = 0;
        a.desc[i].value = 0.0;
    }
    if (i == 0) *a.counter = 0;
}

struct Seg {
    uint32_t f;
    double v;
};

__device__ __forceinline__ Seg combine(Seg a, Seg b) {
    return Seg{a.f | b.f, b.f ? b.v : a.v + b.v};
}

__device__ __forceinline__ int64_t find_rollout(const int64_t *off, int64_t R, int64_t u) {
    // last r in [0, R) with off[r] <= u; -1 if none
    if (R == 0 || off[0] > u) return -1;
    int64_t lo = 0, hi = R;
    while (hi - lo > 1) {
        const int64_t mid = (lo + hi) >> 1;
        if (off[mid] <= u) lo = mid; else hi = mid;
    }
    return lo;
}

template <typename VT>
__global__ __launch_bounds__(kScanThreads) void stop_scan_kernel(StopArgs a) {
    __shared__ int64_t s_tile;
    __shared__ Seg s_wave[kScanThreads / kWave];
    __shared__ double s_carry;
    __shared__ int32_t s_first[kSlots];
    __shared__ int64_t s_r0;

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    if (tid == 0) s_tile = (int64_t)atomicAdd(a.counter, 1u);
    for (int i = tid; i < kSlots; i += blockDim.x) s_first[i] = INT_MAX;
    __syncthreads();
    const int64_t tile = s_tile;
    const int64_t u0 = tile * kScanTile;
    const int64_t R = a.L.n_rollouts;
    const VT *vals = static_cast<const VT *>(a.values);

    // ---- load and thread-local segmented scan ----
    const int64_t ubase = u0 + (int64_t)tid * kScanItems;
    int64_t r = find_rollout(a.unit_off, R, ubase);
    if (tid == 0) s_r0 = find_rollout(a.unit_off, R, u0);
    double run[kScanItems];
    uint8_t head[kScanItems];
    int64_t rr[kScanItems];
    Seg tagg{0u, 0.0};
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        const int64_t u = ubase + j;
        double v = 0.0;
        uint8_t h = 0;
        int64_t rj = -1;  // rollout holding unit u, -1 if none (only with bad offsets)
        if (u < a.n_units && r >= 0) {
            while (r + 1 < R && a.unit_off[r + 1] <= u) ++r;
            const int64_t first = a.unit_off[r];
            const int64_t n = a.unit_off[r + 1] - first;
            const int64_t local = u - first;
            if (local >= 0 && local < n) {
                int64_t k0 = a.start ? (int64_t)a.start[r] : 0;
                k0 = k0 < 0 ? 0 : (k0 > n ? n : k0);
                h = (local == 0);
                if (local >= k0) v = (double)vals[u];
                rj = r;
            }
        }
        rr[j] = rj;
        head[j] = h;
        tagg = combine(tagg, Seg{h, v});
        run[j] = tagg.v;
    }

    // ---- block-level exclusive scan of the thread aggregates ----
    Seg inc = tagg;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const uint32_t f2 = __shfl_up(inc.f, off, kWave);
        const double v2 = __shfl_up(inc.v, off, kWave);
        if (lane >= off) inc = combine(Seg{f2, v2}, inc);
    }
    if (lane == kWave - 1) s_wave[wave] = inc;
    __syncthreads();
    Seg wpre{0u, 0.0};
    for (int w = 0; w < wave; ++w) wpre = combine(wpre, s_wave[w]);
    Seg excl;
    {
        const uint32_t f2 = __shfl_up(inc.f, 1, kWave);
        const double v2 = __shfl_up(inc.v, 1, kWave);
        excl = (lane == 0) ? wpre : combine(wpre, Seg{f2, v2});
    }

    // ---- publish the tile aggregate, then look back ----
    if (tid == 0) {
        Seg total{0u, 0.0};
        for (int w = 0; w < kScanThreads / kWave; ++w) total = combine(total, s_wave[w]);
#ifdef STRIDE_SCAN_DELAY_HOOK
        if (a.delay_one_in) {
            // splitmix64 step (Steele, Lea and Flood 2014) of (seed, tile): picks the tile
            // and its sleep count
            uint64_t z = a.delay_seed + 0x9E3779B97F4A7C15ull * (uint64_t)(tile + 1);
            z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
            z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
            z ^= z >> 31;
            if ((z % a.delay_one_in) == 0) {
                const uint32_t n = 1 + (uint32_t)((z >> 32) % a.delay_sleeps);
                for (uint32_t i = 0; i < n; ++i) __builtin_amdgcn_s_sleep(127);
            }
        }
#endif
        a.desc[tile].value = total.v;
        a.desc[tile].head = total.f;
        __hip_atomic_store(&a.desc[tile].status, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);

        double carry = 0.0;
        const int64_t r0 = s_r0;
        const bool continues = tile > 0 && r0 >= 0 && a.unit_off[r0] < u0;
        if (continues) {
#ifdef STRIDE_SCAN_DELAY_HOOK
            const uint32_t limit = a.spin_limit ? a.spin_limit : kSpinLimit;
#else
            constexpr uint32_t limit = kSpinLimit;
#endif
            for (int64_t p = tile - 1; p >= 0; --p) {
                uint32_t spins = 0;
                while (__hip_atomic_load(&a.desc[p].status, __ATOMIC_ACQUIRE,
                                         __HIP_MEMORY_SCOPE_AGENT) == 0u) {
                    if (++spins > limit) break;
                    __builtin_amdgcn_s_sleep(1);
                }
                if (spins > limit) {
                    raise_flag(a.flags, STRIDE_FLAG_SPIN_LIMIT);
                    carry = __builtin_nan("");
                    break;
                }
                carry = a.desc[p].value + carry;
                if (a.desc[p].head) break;
            }
        }
        s_carry = carry;
    }
    __syncthreads();
    const double carry = s_carry;
    const int64_t r0 = s_r0;

    // ---- cumulative values and first crossings ----
    uint32_t seen = excl.f;
    int64_t last_r = -2;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        const int64_t u = ubase + j;
        if (u >= a.n_units) break;
        const int64_t rj = rr[j];
        seen |= head[j];
        double c;
        if (rj < 0) {
            c = __builtin_nan("");
        } else {
            // thread-local running sum restarted at a head inside this thread's items
            bool head_in_thread = false;
            for (int q = 0; q <= j; ++q) head_in_thread |= (head[q] != 0);
            c = head_in_thread ? run[j] : excl.v + run[j];
            if (!seen) c += carry;
        }
        a.cum[u] = c;
        if (rj < 0 || rj == last_r) continue;
        const int64_t first = a.unit_off[rj];
        const int64_t local = u - first;
        int64_t k0 = a.start ? (int64_t)a.start[rj] : 0;
        const int64_t n = a.unit_off[rj + 1] - first;
        k0 = k0 < 0 ? 0 : (k0 > n ? n : k0);
        const int32_t d = a.L.domain ? a.L.domain[rj] : 0;
        const double lam = (d >= 0 && d < a.n_dom) ? a.lambda.v[d] : __builtin_nan("");
        if (local >= k0 && c < lam) {
            last_r = rj;  // later units of this rollout in this thread cannot be earlier
            const int64_t slot = rj - r0;
            if (r0 >= 0 && slot >= 0 && slot < kSlots)
                atomicMin(&s_first[slot], (int32_t)local);
            else
                atomicMin(&a.stop_unit[rj], (int32_t)local);
        }
    }
    __syncthreads();
    if (r0 >= 0) {
        for (int i = tid; i < kSlots; i += blockDim.x) {
            if (s_first[i] != INT_MAX) atomicMin(&a.stop_unit[r0 + i], s_first[i]);
        }
    }
}

// stop_unit sentinel -> -1, retained row counts, bad domains.
__global__ __launch_bounds__(256) void stop_finish_kernel(StopArgs a) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= a.L.n_rollouts) return;
    const int32_t d = a.L.domain ? a.L.domain[r] : 0;
    if (d < 0 || d >= a.n_dom) raise_flag(a.flags, STRIDE_FLAG_BAD_DOMAIN);
    int32_t s = a.stop_unit[r];
    if (s == INT_MAX) s = -1;
    a.stop_unit[r] = s;
    if (!a.retained) return;
    const int64_t first = a.unit_off[r];
    int64_t n = a.unit_off[r + 1] - first;
    if (n < 0) n = 0;
    int64_t k0 = a.start ? (int64_t)a.start[r] : 0;
    k0 = k0 < 0 ? 0 : (k0 > n ? n : k0);
    int64_t end = (s >= 0) ? (int64_t)s + 1 : n;
    if (end < k0) end = k0;
    if (a.unit == STRIDE_UNIT_TOKEN) {
        a.retained[r] = end - k0;
    } else {
        const int64_t T = a.L.n_turns;
        int64_t t0 = first + k0, t1 = first + end;
        t0 = t0 > T ? T : t0;
        t1 = t1 > T ? T : t1;
        a.retained[r] = a.L.turn_tok_off[t1] - a.L.turn_tok_off[t0];
    }
}

// Online form of the stop test (Algorithm 1's inner loop while a rollout is being
// generated): active rollout a = 0 .. n_active-1 (state slot rid[a]) receives new
// units [new_off[a], new_off[a+1]) with the given values; they are appended at
// local index state_units[slot] on.  One wavefront per active rollout scans them in
// 64-unit chunks (fixed shuffle tree in double) on top of the carried sum; the
// first crossing found (ballot, lowest lane) becomes stop_unit[slot].  A rollout
// that has already stopped ignores further units.
template <typename VT>
__global__ __launch_bounds__(256) void stop_step_kernel(int32_t n_active, const int32_t *rid,
                                                        const int64_t *new_off, const VT *values,
                                                        const int32_t *domain, DomainTable lambda,
                                                        int32_t n_dom, double *state_cum,
                                                        int32_t *state_units, int32_t *stop_unit,
                                                        uint32_t *flags) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t a = (int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave);
    if (a >= n_active) return;
    const int32_t slot = rid[a];
    if (slot < 0) {
        if (lane == 0) raise_flag(flags, STRIDE_FLAG_BAD_OFFSETS);
        return;
    }
    const int64_t b0 = new_off[a], b1 = new_off[a + 1];
    if (b1 < b0 || b0 < 0) {
        if (lane == 0) raise_flag(flags, STRIDE_FLAG_BAD_OFFSETS);
        return;
    }
    const int32_t d = domain ? domain[slot] : 0;
    if (d < 0 || d >= n_dom) {
        if (lane == 0) raise_flag(flags, STRIDE_FLAG_BAD_DOMAIN);
        return;
    }
    const double lam = lambda.v[d];
    int32_t stop = stop_unit[slot];
    double carry = state_cum[slot];
    const int32_t u0 = state_units[slot];
    if (stop < 0) {
        for (int64_t c = b0; c < b1; c += kWave) {
            const int64_t i = c + lane;
            double v = (i < b1) ? (double)values[i] : 0.0;
            // inclusive scan of the chunk, fixed association
#pragma unroll
            for (int off = 1; off < kWave; off <<= 1) {
                const double t = __shfl_up(v, off, kWave);
                if (lane >= off) v += t;
            }
            const double cum = carry + v;
            const bool cross = (i < b1) && (cum < lam);
            const uint64_t hit = __ballot(cross);
            if (hit) {
                const int first = __builtin_ctzll(hit);
                stop = u0 + (int32_t)(c - b0) + first;
                carry = __shfl(cum, first, kWave);
                break;
            }
            const int last = (int)((b1 - c) < kWave ? (b1 - c) : kWave) - 1;
            carry = __shfl(cum, last, kWave);
        }
    }
    if (lane == 0) {
        state_cum[slot] = carry;
        state_units[slot] = u0 + (int32_t)(b1 - b0);
        stop_unit[slot] = stop;
    }
}

}  // namespace

hipError_t launch_stop_step(int32_t n_active, const int32_t *rid, const int64_t *new_off,
                            int32_t unit, const void *values, const int32_t *domain,
                            const DomainTable &lambda, int32_t n_dom, double *state_cum,
                            int32_t *state_units, int32_t *stop_unit, uint32_t *flags,
                            hipStream_t stream) {
    if (n_active == 0) return hipSuccess;
    const unsigned blocks = (unsigned)((n_active + 3) / 4);
    if (unit == STRIDE_UNIT_TURN)
        hipLaunchKernelGGL(stop_step_kernel<double>, dim3(blocks), dim3(256), 0, stream, n_active,
                           rid, new_off, static_cast<const double *>(values), domain, lambda, n_dom,
                           state_cum, state_units, stop_unit, flags);
    else
        hipLaunchKernelGGL(stop_step_kernel<float>, dim3(blocks), dim3(256), 0, stream, n_active,
                           rid, new_off, static_cast<const float *>(values), domain, lambda, n_dom,
                           state_cum, state_units, stop_unit, flags);
    return hipGetLastError();
}

hipError_t launch_stop(const stride_layout &L, int32_t unit, const void *values,
                       const DomainTable &lambda, int32_t n_dom, const int32_t *start,
                       double *cum, int32_t *stop_unit, int64_t *retained, uint32_t *flags,
                       void *ws, hipStream_t stream) {
    const int64_t n_units = (unit == STRIDE_UNIT_TURN) ? L.n_turns : L.n_tokens;
    const WsLayout w = ws_layout(L.n_rollouts, 0, n_units, 0);
    char *base = static_cast<char *>(ws);
    StopArgs a;
    a.L = L;
    a.lambda = lambda;
    a.n_dom = n_dom;
    a.unit = unit;
    a.n_units = n_units;
    a.n_tiles = (n_units + kScanTile - 1) / kScanTile;
    a.values = values;
    a.start = start;
    a.unit_off = reinterpret_cast<const int64_t *>(base + w.unit_off);
    a.cum = cum;
    a.stop_unit = stop_unit;
    a.retained = retained;
    a.counter = reinterpret_cast<uint32_t *>(base + w.counter);
    a.desc = reinterpret_cast<TileDesc *>(base + w.desc);
    a.flags = flags;
#ifdef STRIDE_SCAN_DELAY_HOOK
    a.delay_seed = g_delay_seed.load();
    a.delay_one_in = g_delay_one_in.load();
    a.delay_sleeps = g_delay_sleeps.load();
    a.spin_limit = g_spin_limit.load();
#else
    a.delay_seed = 0;
    a.delay_one_in = 0;
    a.delay_sleeps = 0;
    a.spin_limit = 0;
#endif

    const int64_t prep_n = (L.n_rollouts + 1 > a.n_tiles) ? L.n_rollouts + 1 : a.n_tiles;
    hipLaunchKernelGGL(stop_prep_kernel, dim3((unsigned)((prep_n + 255) / 256)), dim3(256), 0,
                       stream, a, reinterpret_cast<int64_t *>(base + w.unit_off));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (a.n_tiles > 0) {
        if (unit == STRIDE_UNIT_TURN)
            hipLaunchKernelGGL(stop_scan_kernel<double>, dim3((unsigned)a.n_tiles),
                               dim3(kScanThreads), 0, stream, a);
        else
            hipLaunchKernelGGL(stop_scan_kernel<float>, dim3((unsigned)a.n_tiles),
                               dim3(kScanThreads), 0, stream, a);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (L.n_rollouts > 0) {
        hipLaunchKernelGGL(stop_finish_kernel, dim3((unsigned)((L.n_rollouts + 255) / 256)),
                           dim3(256), 0, stream, a);
        e = hipGetLastError();
    }
    return e;
}

// ---- scratch of the allocation-free stop test ----
// A fixed device array, one copy per GPU, held until the process ends.  In host code
// `scratch` names a host-side stand-in, not a device address: the device address of each
// GPU's copy comes from hipGetSymbolAddress, looked up once per device with that device
// current, and only that address is handed to kernels.
static __device__ __align__(256) char scratch[STRIDE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;

hipError_t noalloc_scratch(void **ptr) {
    static std::atomic<void *> addr[kMaxDevices];
    static std::mutex mu;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    void *p = addr[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> g(mu);
        p = addr[dev].load(std::memory_order_relaxed);
        if (!p) {
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return e;
            if (!p) return hipErrorInvalidSymbol;
            addr[dev].store(p, std::memory_order_release);
        }
    }
    *ptr = p;
    return hipSuccess;
}

}  // namespace stride

extern "C" stride_status stride_debug_scan_delay(uint64_t seed, uint32_t one_in, uint32_t sleeps) {
#ifdef STRIDE_SCAN_DELAY_HOOK
    if (one_in > 0 && (sleeps < 1 || sleeps > stride::kMaxDelaySleeps)) return STRIDE_ERR_INVALID_ARG;
    stride::g_delay_seed.store(seed);
    stride::g_delay_sleeps.store(sleeps);
    stride::g_delay_one_in.store(one_in);
    return STRIDE_OK;
#else
    (void)seed;
    (void)one_in;
    (void)sleeps;
    return STRIDE_ERR_UNSUPPORTED;
#endif
}

extern "C" stride_status stride_debug_scan_spin_limit(uint32_t limit) {
#ifdef STRIDE_SCAN_DELAY_HOOK
    stride::g_spin_limit.store(limit);
    return STRIDE_OK;
#else
    (void)limit;
    return STRIDE_ERR_UNSUPPORTED;
#endif
}
