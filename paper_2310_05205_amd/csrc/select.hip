// Trajectory selection on gfx950 (GEAR Sec. 1 strategies; Sec. 3.3).
//
// Prioritized (weighted) sampling is a prefix sum over the priorities
// followed by one search per uniform draw (Sec. 3.3, centralized selection).
// It runs as two kernels:
//
//   scan_kernel    one pass over the priorities with decoupled look-back.
//                  Each workgroup reduces a 4096-priority chunk (16 tiles of
//                  256), publishes its aggregate, looks back over its
//                  predecessors' published words 64 at a time for its
//                  exclusive prefix, and writes the global inclusive prefix
//                  at the end of each of its tiles (level 0 of the prefix
//                  tree) plus every 256^l-th of those (level l).  Nothing of
//                  size N is written.
//   search_kernel  one wave per draw: r = floor(u*S/2^64) for a splitmix64
//                  output u, then a 256-ary descent of the prefix tree (four
//                  entries per lane, ballot + popcount finds the first entry
//                  greater than r), then a wave scan of the chosen tile's 256
//                  priorities in registers and a final ballot.  The result is
//                  the smallest i with C_i > r, i.e. the binary-search answer
//                  over the full inclusive prefix C.
//
// FIFO, LIFO and uniform selection are one thread per draw.
#include "gear_internal.h"

namespace gear {
namespace {

constexpr uint64_t kValueMask = (1ull << 62) - 1;
constexpr uint64_t kAggregate = 1ull << 62;
constexpr uint64_t kInclusive = 2ull << 62;
constexpr uint32_t kMaxSpins = 1u << 22;

struct Levels {
    uint64_t* level[kMaxLevels];
    int64_t size[kMaxLevels];
    int nlevels;
};

// splitmix64 (Steele, Lea & Flood, OOPSLA 2014): output c of the stream
// seeded with `seed` is the finaliser applied to seed + (c+1)*gamma.
__device__ inline uint64_t splitmix64_out(uint64_t seed, uint64_t c) {
    uint64_t z = seed + (c + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// floor(u * n / 2^64): the high word of the 128-bit product.
__device__ inline uint64_t scale_draw(uint64_t u, uint64_t n) { return __umul64hi(u, n); }

__device__ inline uint64_t wave_sum(uint64_t v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
    return v;
}

__device__ inline uint64_t wave_inclusive_scan(uint64_t v, int lane) {
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        uint64_t o = __shfl_up(v, d);
        if (lane >= d) v += o;
    }
    return v;
}

__device__ inline uint64_t pick4(uint64_t a, uint64_t b, uint64_t c, uint64_t d, int q) {
    return q == 0 ? a : (q == 1 ? b : (q == 2 ? c : d));
}

__device__ inline uint64_t load_lookback(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ inline void store_lookback(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(256) void scan_kernel(const uint32_t* __restrict__ prio, int64_t N, int64_t ntiles,
                                                   Levels lv, uint64_t* __restrict__ look_cur,
                                                   uint64_t* __restrict__ look_next, uint32_t* ticket_cur,
                                                   uint32_t* ticket_next, int64_t nchunks, uint32_t* status) {
    __shared__ uint64_t tile_sum[kTilesPerChunk];
    __shared__ int64_t s_chunk;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;

    // Chunks are numbered in the order workgroups start, so a workgroup only
    // ever waits on chunks whose workgroups are already running.
    if (threadIdx.x == 0)
        s_chunk = (int64_t)__hip_atomic_fetch_add(ticket_cur, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    const int64_t chunk = s_chunk;
    if (chunk >= nchunks) return;  // only if a previous scan was interrupted
    if (threadIdx.x == 0) {
        // Prepare the other look-back buffer and ticket for the next scan.
        look_next[chunk] = 0;
        if (chunk == 0) *ticket_next = 0;
    }

    // Tile sums: wave w owns tiles 4w .. 4w+3 of the chunk, one 16-byte
    // load per lane per tile.
    uint32_t x[4][4];
#pragma unroll
    for (int q = 0; q < 4; q++) {
        const int64_t e = (chunk * kTilesPerChunk + wave * 4 + q) * kTile + lane * 4;
        if (e + 4 <= N) {
            uint4 v = *reinterpret_cast<const uint4*>(prio + e);
            x[q][0] = v.x; x[q][1] = v.y; x[q][2] = v.z; x[q][3] = v.w;
        } else {
#pragma unroll
            for (int k = 0; k < 4; k++) x[q][k] = (e + k < N) ? prio[e + k] : 0u;
        }
    }
#pragma unroll
    for (int q = 0; q < 4; q++) {
        uint64_t s = (uint64_t)x[q][0] + x[q][1] + x[q][2] + x[q][3];
        s = wave_sum(s);
        if (lane == 0) tile_sum[wave * 4 + q] = s;
    }
    __syncthreads();
    if (wave != 0) return;

    const uint64_t local = wave_inclusive_scan(lane < kTilesPerChunk ? tile_sum[lane] : 0, lane);
    const uint64_t aggregate = __shfl(local, kTilesPerChunk - 1);
    uint64_t prefix = 0;
    if (chunk == 0) {
        if (lane == 0) store_lookback(&look_cur[0], kInclusive | aggregate);
    } else {
        if (lane == 0) store_lookback(&look_cur[chunk], kAggregate | aggregate);
        int64_t base = chunk - 1;  // predecessor examined by lane 0
        uint32_t spins = 0;
        while (true) {
            const int64_t pos = base - lane;
            const uint64_t w = pos >= 0 ? load_lookback(&look_cur[pos]) : kInclusive;
            const uint64_t state = w >> 62;
            const unsigned long long not_ready = __ballot(state == 0);
            const unsigned long long inclusive = __ballot(state == 2);
            const int first_incl = inclusive ? __ffsll((long long)inclusive) - 1 : 64;
            const int first_wait = not_ready ? __ffsll((long long)not_ready) - 1 : 64;
            if (first_wait < first_incl) {
                // A chunk we need has not published yet.  Its workgroup is
                // running (tickets are taken in start order), so the wait
                // ends; the bound only guarantees every wave exits.
                if (++spins > kMaxSpins) {
                    if (lane == 0) atomicOr(status, GEAR_STATUS_INTERNAL);
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
                continue;
            }
            const int upto = first_incl < 64 ? first_incl : 63;
            prefix += wave_sum(lane <= upto ? (w & kValueMask) : 0);
            if (first_incl < 64) break;
            base -= 64;
        }
        if (lane == 0) store_lookback(&look_cur[chunk], kInclusive | (prefix + aggregate));
    }

    if (lane < kTilesPerChunk) {
        const int64_t gt = chunk * kTilesPerChunk + lane;
        if (gt < ntiles) {
            const uint64_t c = prefix + local;
            lv.level[0][gt] = c;
            int64_t span = kFanout;
            for (int l = 1; l < lv.nlevels; l++) {
                if (((gt + 1) % span) == 0 || gt == ntiles - 1) lv.level[l][gt / span] = c;
                span *= kFanout;
            }
        }
    }
}

// Number of entries <= r among a[s0 .. s0+256) (entries at or past n count as
// +inf), and the value of the last such entry (unchanged `lo` if none).
__device__ inline int64_t descend_level(const uint64_t* __restrict__ a, int64_t n, int64_t s0, uint64_t r,
                                        int lane, uint64_t& lo) {
    const int64_t e = s0 + lane * 4;
    uint64_t v0, v1, v2, v3;
    if (e + 4 <= n) {
        const ulonglong2 p0 = *reinterpret_cast<const ulonglong2*>(a + e);
        const ulonglong2 p1 = *reinterpret_cast<const ulonglong2*>(a + e + 2);
        v0 = p0.x; v1 = p0.y; v2 = p1.x; v3 = p1.y;
    } else {
        v0 = e + 0 < n ? a[e + 0] : ~0ull;
        v1 = e + 1 < n ? a[e + 1] : ~0ull;
        v2 = e + 2 < n ? a[e + 2] : ~0ull;
        v3 = e + 3 < n ? a[e + 3] : ~0ull;
    }
    const int cnt = __popcll(__ballot(v0 <= r)) + __popcll(__ballot(v1 <= r)) + __popcll(__ballot(v2 <= r)) +
                    __popcll(__ballot(v3 <= r));
    if (cnt > 0) {
        const int k = cnt - 1;
        lo = __shfl(pick4(v0, v1, v2, v3, k & 3), k >> 2);
    }
    return s0 + cnt;
}

__global__ __launch_bounds__(256) void search_kernel(const uint32_t* __restrict__ prio, int64_t N, Levels lv,
                                                     int32_t B, uint64_t span, uint64_t seed, int want_min,
                                                     uint32_t* __restrict__ wg_min, uint32_t* status,
                                                     int64_t* __restrict__ idx, int32_t* __restrict__ start) {
    __shared__ uint32_t s_min[4];
    const int lane = threadIdx.x & 63;
    const int64_t wave_id = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
    const int top = lv.nlevels - 1;
    const uint64_t S = lv.level[top][lv.size[top] - 1];
    uint32_t my_min = 0xFFFFFFFFu;  // smallest priority this wave selected

    for (int64_t b = wave_id; b < B; b += nwaves) {
        if (S == 0) {
            if (lane == 0) {
                idx[b] = -1;
                start[b] = 0;
                atomicOr(status, GEAR_STATUS_NO_WEIGHT);
            }
            continue;
        }
        const uint64_t r = scale_draw(splitmix64_out(seed, 2 * (uint64_t)b), S);
        uint64_t lo = 0;
        int64_t j = 0;
        for (int l = top; l >= 0; l--) j = descend_level(lv.level[l], lv.size[l], j * kFanout, r, lane, lo);

        // j is the tile holding r; scan its 256 priorities in registers.
        const uint64_t rr = r - lo;
        const int64_t e = j * kTile + lane * 4;
        uint32_t p0, p1, p2, p3;
        if (e + 4 <= N) {
            const uint4 v = *reinterpret_cast<const uint4*>(prio + e);
            p0 = v.x; p1 = v.y; p2 = v.z; p3 = v.w;
        } else {
            p0 = e + 0 < N ? prio[e + 0] : 0u;
            p1 = e + 1 < N ? prio[e + 1] : 0u;
            p2 = e + 2 < N ? prio[e + 2] : 0u;
            p3 = e + 3 < N ? prio[e + 3] : 0u;
        }
        const uint64_t lsum = (uint64_t)p0 + p1 + p2 + p3;
        const uint64_t excl = wave_inclusive_scan(lsum, lane) - lsum;
        const uint64_t c0 = excl + p0, c1 = c0 + p1, c2 = c1 + p2, c3 = c2 + p3;
        const int cnt = __popcll(__ballot(c0 <= rr)) + __popcll(__ballot(c1 <= rr)) +
                        __popcll(__ballot(c2 <= rr)) + __popcll(__ballot(c3 <= rr));
        if (lane == 0) {
            idx[b] = j * kTile + cnt;
            start[b] = (int32_t)scale_draw(splitmix64_out(seed, 2 * (uint64_t)b + 1), span);
        }
        if (want_min) {
            const uint32_t pv = (uint32_t)__shfl((uint64_t)pick4(p0, p1, p2, p3, cnt & 3), cnt >> 2);
            my_min = pv < my_min ? pv : my_min;
        }
    }
    if (want_min) {
        // One slot per workgroup, no atomics: the weight kernel reduces them.
        if (lane == 0) s_min[threadIdx.x >> 6] = my_min;
        __syncthreads();
        if (threadIdx.x == 0) {
            uint32_t m = s_min[0];
            for (int k = 1; k < (int)(blockDim.x >> 6); k++) m = s_min[k] < m ? s_min[k] : m;
            wg_min[blockIdx.x] = m;
        }
    }
}

// w_b = (n*P(i_b))^-beta / max_b' (n*P(i_b'))^-beta = (p_min / p_b)^beta,
// p_min the smallest selected priority; fp64, rounded once to fp32.  Every
// workgroup first reduces the search's per-workgroup minima.
__global__ __launch_bounds__(256) void is_weights_kernel(const uint32_t* __restrict__ prio, int64_t N,
                                                         const int64_t* __restrict__ idx, int32_t B, double beta,
                                                         const uint32_t* __restrict__ wg_min, int search_grid,
                                                         float* __restrict__ w) {
    __shared__ uint32_t s_min[4];
    uint32_t m = 0xFFFFFFFFu;
    for (int k = threadIdx.x; k < search_grid; k += blockDim.x) m = wg_min[k] < m ? wg_min[k] : m;
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const uint32_t o = __shfl_xor(m, d);
        m = o < m ? o : m;
    }
    if ((threadIdx.x & 63) == 0) s_min[threadIdx.x >> 6] = m;
    __syncthreads();
    m = s_min[0];
    for (int k = 1; k < (int)(blockDim.x >> 6); k++) m = s_min[k] < m ? s_min[k] : m;

    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    const int64_t i = idx[b];
    if (i < 0 || i >= N || m == 0u) {
        w[b] = 0.0f;
        return;
    }
    w[b] = (float)pow((double)m / (double)prio[i], beta);
}

// FIFO / LIFO: ring arithmetic from the oldest / newest live slot.
// Uniform: floor(u * n / 2^64) over the n live slots.
__global__ void simple_select_kernel(int strategy, int32_t B, int64_t N, int64_t live, int64_t oldest_slot,
                                     int64_t newest_slot, uint64_t span, uint64_t seed, int64_t* __restrict__ idx,
                                     int32_t* __restrict__ start, float* __restrict__ w) {
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    int64_t i;
    if (strategy == GEAR_FIFO) {
        i = oldest_slot + b;
        if (i >= N) i -= N;
    } else if (strategy == GEAR_LIFO) {
        i = newest_slot - b;
        if (i < 0) i += N;
    } else {
        i = (int64_t)scale_draw(splitmix64_out(seed, 2 * (uint64_t)b), (uint64_t)live);
    }
    idx[b] = i;
    start[b] = (int32_t)scale_draw(splitmix64_out(seed, 2 * (uint64_t)b + 1), span);
    if (w) w[b] = 1.0f;
}

Levels make_levels(const Table& t) {
    Levels lv{};
    for (int l = 0; l < t.nlevels; l++) {
        lv.level[l] = t.level[l];
        lv.size[l] = t.level_size[l];
    }
    lv.nlevels = t.nlevels;
    return lv;
}

}  // namespace

hipError_t launch_scan(Table& t, hipStream_t s) {
    const int par = t.scan_parity;
    hipLaunchKernelGGL(scan_kernel, dim3((unsigned)t.nchunks), dim3(256), 0, s, t.priority, t.N, t.ntiles,
                       make_levels(t), t.lookback + (size_t)par * t.nchunks,
                       t.lookback + (size_t)(1 - par) * t.nchunks, t.ticket + par, t.ticket + (1 - par),
                       t.nchunks, t.status);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) t.scan_parity = 1 - par;
    return e;
}

hipError_t launch_search(Table& t, int32_t B, int32_t L, uint64_t seed, bool want_min, int64_t* idx,
                         int32_t* start, int* grid_out, hipStream_t s) {
    int64_t g = ((int64_t)B + 3) / 4;  // one wave per draw while the grid allows
    const int grid = (int)(g < kSearchMaxGrid ? g : kSearchMaxGrid);
    hipLaunchKernelGGL(search_kernel, dim3(grid), dim3(256), 0, s, t.priority, t.N, make_levels(t), B,
                       (uint64_t)(t.T - L + 1), seed, want_min ? 1 : 0, t.wg_min, t.status, idx, start);
    *grid_out = grid;
    return hipGetLastError();
}

hipError_t launch_is_weights(Table& t, int32_t B, float beta, int search_grid, const int64_t* idx, float* w,
                             hipStream_t s) {
    hipLaunchKernelGGL(is_weights_kernel, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, s, t.priority, t.N, idx,
                       B, (double)beta, t.wg_min, search_grid, w);
    return hipGetLastError();
}

hipError_t launch_simple_select(Table& t, int32_t strategy, int32_t B, int32_t L, uint64_t seed, int64_t* idx,
                                int32_t* start, float* w, hipStream_t s) {
    const int64_t live = t.next_seq < (uint64_t)t.N ? (int64_t)t.next_seq : t.N;
    const int64_t oldest = (int64_t)((t.next_seq - (uint64_t)live) % (uint64_t)t.N);
    const int64_t newest = (int64_t)((t.next_seq - 1) % (uint64_t)t.N);
    hipLaunchKernelGGL(simple_select_kernel, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, s, strategy, B, t.N,
                       live, oldest, newest, (uint64_t)(t.T - L + 1), seed, idx, start, w);
    return hipGetLastError();
}

}  // namespace gear

using gear::fail;
using gear::hip_fail;

extern "C" int gear_select(gear_table* h, int32_t strategy, int32_t B, int32_t L, uint64_t seed, float beta,
                           int64_t* d_idx, int32_t* d_start, float* d_weights, void* stream) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_select: table is NULL");
    gear::Table* t = reinterpret_cast<gear::Table*>(h);
    if (strategy < GEAR_FIFO || strategy > GEAR_PRIORITIZED) return fail(GEAR_E_INVAL, "gear_select: unknown strategy");
    if (B < 1 || B > GEAR_MAX_BATCH) return fail(GEAR_E_INVAL, "gear_select: B out of range");
    if (L < 1 || L > t->T) return fail(GEAR_E_INVAL, "gear_select: L must lie in [1, T]");
    if (d_idx == nullptr || d_start == nullptr) return fail(GEAR_E_INVAL, "gear_select: output pointer is NULL");
    if (!(beta == beta)) return fail(GEAR_E_INVAL, "gear_select: beta is NaN");
    const int64_t live = t->next_seq < (uint64_t)t->N ? (int64_t)t->next_seq : t->N;
    if (live == 0) return fail(GEAR_E_EMPTY, "gear_select: nothing inserted");
    if ((strategy == GEAR_FIFO || strategy == GEAR_LIFO) && (int64_t)B > live)
        return fail(GEAR_E_INSUFFICIENT, "gear_select: FIFO/LIFO batch larger than the live count");
    gear::DeviceGuard guard(t->device);
    if (guard.error() != hipSuccess) return hip_fail(guard.error(), "gear_select: hipSetDevice");
    hipStream_t s = static_cast<hipStream_t>(stream);

    if (strategy != GEAR_PRIORITIZED) {
        hipError_t e = gear::launch_simple_select(*t, strategy, B, L, seed, d_idx, d_start, d_weights, s);
        return e == hipSuccess ? GEAR_OK : hip_fail(e, "gear_select: launch");
    }
    if (t->cdf_dirty) {
        hipError_t e = gear::launch_scan(*t, s);
        if (e != hipSuccess) return hip_fail(e, "gear_select: scan launch");
        t->cdf_dirty = false;
    }
    const bool weights = d_weights != nullptr;
    int grid = 0;
    hipError_t e = gear::launch_search(*t, B, L, seed, weights, d_idx, d_start, &grid, s);
    if (e != hipSuccess) return hip_fail(e, "gear_select: search launch");
    if (weights) {
        e = gear::launch_is_weights(*t, B, beta, grid, d_idx, d_weights, s);
        if (e != hipSuccess) return hip_fail(e, "gear_select: weight launch");
    }
    return GEAR_OK;
}
