// Trajectory selection on gfx950 (GEAR Sec. 1 strategies; Sec. 3.3).
//
// Prioritized (weighted) sampling is a prefix sum over the priorities
// followed by one search per uniform draw (Sec. 3.3, centralized selection).
// Here the prefix sum is split between two kernels so that no workgroup ever
// waits on another:
//
//   scan_kernel    one pass over the priorities.  A workgroup reduces a
//                  chunk of 32 tiles of 256 priorities, writes each tile's
//                  sum (level 0 of a 256-ary sum tree) and adds the chunk's
//                  sum into the one node of every higher level that covers
//                  it (at most 8 chunks share a level-1 node).  The top
//                  level has at most 256 nodes.
//   search_kernel  one wave per draw: the wave loads the top level (four
//                  nodes per lane), forms its inclusive prefix with a wave
//                  scan in registers (the total is S), draws r =
//                  floor(u*S/2^64), then descends: at each level it scans
//                  the 256 children of the chosen node in registers, counts
//                  the children whose inclusive prefix is <= r (ballot +
//                  popcount), takes the next one and subtracts the prefix
//                  before it from r; at the leaves it does the same over the
//                  chosen tile's 256 priorities.  The index found is the
//                  smallest i with C_i > r for the inclusive prefix C over
//                  all priorities: the binary-search answer.
//
// Small tables (N <= kSmallN, B <= kSmallMaxB, sum tree not kept across
// updates) take one launch instead: small_select_kernel, one workgroup,
// forms the inclusive prefix C of all N priorities in LDS with a block scan,
// finds each draw's slot as the smallest i with C_i > r by bisection over
// C, and computes the IS weights, all in one launch.
//
// FIFO, LIFO and uniform selection are one thread per draw.
#include <mutex>

#include "gear_internal.h"
#include "wave.h"

namespace gear {
namespace {

struct Levels {
    uint64_t* level[kMaxLevels];   // level 0: tile sums; level l: sums of 256^l tiles
    int64_t size[kMaxLevels];
    int nlevels;
    // The top level again (level[nlevels - 1]), so that a search reads it
    // without first waiting for nlevels.
    const uint64_t* top;
    int64_t top_size;
};

// Sets the top-level copy of a search's levels.
inline Levels with_top(Levels lv) {
    lv.top = lv.level[lv.nlevels - 1];
    lv.top_size = lv.size[lv.nlevels - 1];
    return lv;
}

// Inclusive prefix of 256 values held four per lane (lane l holds values
// 4l..4l+3): c0..c3 receive the prefix at this lane's four positions.
__device__ inline void wave_prefix4(uint64_t v0, uint64_t v1, uint64_t v2, uint64_t v3, uint64_t& c0,
                                    uint64_t& c1, uint64_t& c2, uint64_t& c3) {
    const uint64_t part = v0 + v1 + v2 + v3;
    const uint64_t excl = wave_inclusive_scan(part) - part;
    c0 = excl + v0;
    c1 = c0 + v1;
    c2 = c1 + v2;
    c3 = c2 + v3;
}

// Among 256 positions whose inclusive prefixes are c0..c3 (four per lane),
// the number whose prefix is <= r, i.e. the position of the first prefix
// greater than r; r is reduced by the prefix before that position.
__device__ inline int pick_child(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3, uint64_t& r) {
    const int cnt = __popcll(__ballot(c0 <= r)) + __popcll(__ballot(c1 <= r)) + __popcll(__ballot(c2 <= r)) +
                    __popcll(__ballot(c3 <= r));
    if (cnt > 0) {
        const int k = cnt - 1;
        r -= read_lane(pick4(c0, c1, c2, c3, k & 3), k >> 2);
    }
    return cnt;
}

__device__ inline void load4_u64(const uint64_t* __restrict__ a, int64_t n, int64_t e, uint64_t& v0, uint64_t& v1,
                                 uint64_t& v2, uint64_t& v3) {
    if (e + 4 <= n) {
        const ulonglong2 p0 = *reinterpret_cast<const ulonglong2*>(a + e);
        const ulonglong2 p1 = *reinterpret_cast<const ulonglong2*>(a + e + 2);
        v0 = p0.x; v1 = p0.y; v2 = p1.x; v3 = p1.y;
    } else {
        v0 = e + 0 < n ? a[e + 0] : 0;
        v1 = e + 1 < n ? a[e + 1] : 0;
        v2 = e + 2 < n ? a[e + 2] : 0;
        v3 = e + 3 < n ? a[e + 3] : 0;
    }
}

__device__ inline void load4_u32(const uint32_t* __restrict__ a, int64_t n, int64_t e, uint32_t& p0, uint32_t& p1,
                                 uint32_t& p2, uint32_t& p3) {
    if (e + 4 <= n) {
        const uint4 v = *reinterpret_cast<const uint4*>(a + e);
        p0 = v.x; p1 = v.y; p2 = v.z; p3 = v.w;
    } else {
        p0 = e + 0 < n ? a[e + 0] : 0u;
        p1 = e + 1 < n ? a[e + 1] : 0u;
        p2 = e + 2 < n ? a[e + 2] : 0u;
        p3 = e + 3 < n ? a[e + 3] : 0u;
    }
}

// `upper` holds the levels >= 1 this scan adds into; `clear` the other copy
// of those levels, which this scan zeroes for the next one (each node is
// zeroed by the chunk that starts it).
// kMin: also write the chunk's smallest non-zero priority (only the
// global IS normalisation needs it; the plain scan stays minimal).
template <bool kMin>
__global__ __launch_bounds__(256) void scan_kernel(const uint32_t* __restrict__ prio, int64_t N, Levels upper,
                                                   Levels clear, uint64_t* __restrict__ tile_sums, int64_t ntiles,
                                                   uint32_t* __restrict__ chunk_min) {
    __shared__ uint64_t tile_sum[kTilesPerChunk];
    __shared__ uint32_t wave_min[4];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t chunk = blockIdx.x;
    constexpr int kTilesPerWave = kTilesPerChunk / 4;

    // Wave w owns tiles 8w .. 8w+7 of the chunk: eight 16-byte loads per
    // lane, all issued before any is used.
    uint32_t x[kTilesPerWave][4];
#pragma unroll
    for (int q = 0; q < kTilesPerWave; q++)
        load4_u32(prio, N, (chunk * kTilesPerChunk + wave * kTilesPerWave + q) * kTile + lane * 4, x[q][0], x[q][1],
                  x[q][2], x[q][3]);
#pragma unroll
    for (int q = 0; q < kTilesPerWave; q++) {
        const uint64_t s = wave_sum((uint64_t)x[q][0] + x[q][1] + x[q][2] + x[q][3]);
        const int64_t gt = chunk * kTilesPerChunk + wave * kTilesPerWave + q;
        if (lane == 0) {
            tile_sum[wave * kTilesPerWave + q] = s;
            if (gt < ntiles) tile_sums[gt] = s;
        }
    }
    if (kMin) {
        // Smallest non-zero priority of the chunk.
        uint32_t m = 0xFFFFFFFFu;
#pragma unroll
        for (int q = 0; q < kTilesPerWave; q++)
#pragma unroll
            for (int e = 0; e < 4; e++) m = (x[q][e] != 0u && x[q][e] < m) ? x[q][e] : m;
#pragma unroll
        for (int d = 32; d >= 1; d >>= 1) {
            const uint32_t o = __shfl_xor(m, d);
            m = o < m ? o : m;
        }
        if (lane == 0) wave_min[wave] = m;
    }
    __syncthreads();
    if (wave != 0) return;
    if (kMin && lane == 0) {
        uint32_t cm = wave_min[0];
        for (int k = 1; k < 4; k++) cm = wave_min[k] < cm ? wave_min[k] : cm;
        chunk_min[chunk] = cm;
    }
    const uint64_t chunk_sum = wave_sum(lane < kTilesPerChunk ? tile_sum[lane] : 0);
    // Lane l - 1 handles level l (>= 1).
    const int l = lane + 1;
    if (l < upper.nlevels) {
        int64_t tiles_per_node = kFanout;
        for (int k = 1; k < l; k++) tiles_per_node *= kFanout;
        const int64_t first_tile = chunk * kTilesPerChunk;
        const int64_t node = first_tile / tiles_per_node;
        if (chunk_sum != 0) atomicAdd(reinterpret_cast<unsigned long long*>(upper.level[l] + node), chunk_sum);
        if (first_tile % tiles_per_node == 0) clear.level[l][node] = 0;
    }
}

// One GPU's share of a selection over G shards (the table is shard g).
// With totals == NULL the table is the whole population.
struct Shard {
    const uint64_t* totals;  // the G shard totals, identical on every shard
    int G, g;
    int64_t base;            // added to the local slot of an owned draw
};

template <bool kShard>
__global__ __launch_bounds__(256) void search_kernel(const uint32_t* __restrict__ prio, int64_t N, Levels lv,
                                                     int32_t B, uint64_t span, uint64_t seed, int want_min,
                                                     Shard sh, uint32_t* __restrict__ wg_min, uint32_t* status,
                                                     int64_t* __restrict__ idx, int32_t* __restrict__ start,
                                                     uint32_t* __restrict__ sel_prio) {
    __shared__ uint32_t s_min[4];
    const int lane = threadIdx.x & 63;
    const int64_t wave_id = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
    const int top = lv.nlevels - 1;

    // The top level is the same for every draw: its prefix and total once.
    uint64_t t0, t1, t2, t3, tc0, tc1, tc2, tc3;
    load4_u64(lv.top, lv.top_size, lane * 4, t0, t1, t2, t3);
    wave_prefix4(t0, t1, t2, t3, tc0, tc1, tc2, tc3);
    const uint64_t S = read_lane(tc3, 63);
    // Draws are numbers in [0, S_all); this table owns [P, P + S).
    uint64_t S_all = S, P = 0;
    if (kShard) {
        uint64_t all = 0, before = 0;
        for (int h = lane; h < sh.G; h += 64) {
            const uint64_t x = sh.totals[h];
            all += x;
            before += h < sh.g ? x : 0;
        }
        S_all = wave_sum(all);
        P = wave_sum(before);
    }
    uint32_t my_min = 0xFFFFFFFFu;  // smallest priority this wave selected

    for (int64_t b = wave_id; b < B; b += nwaves) {
        if (S_all == 0) {
            if (lane == 0) {
                idx[b] = -1;
                start[b] = 0;
                if (want_min) sel_prio[b] = 0u;
                atomicOr(status, GEAR_STATUS_NO_WEIGHT);
            }
            continue;
        }
        uint64_t r = scale_draw(splitmix64_out(seed, 2 * (uint64_t)b), S_all);
        if (kShard) {
            if (r < P || r - P >= S) {  // another shard's draw: same window start, no slot
                if (lane == 0) {
                    idx[b] = -1;
                    start[b] = (int32_t)scale_draw(splitmix64_out(seed, 2 * (uint64_t)b + 1), span);
                    if (want_min) sel_prio[b] = 0u;
                }
                continue;
            }
            r -= P;
        }
        int64_t j = pick_child(tc0, tc1, tc2, tc3, r);
        for (int l = top - 1; l >= 0; l--) {
            uint64_t v0, v1, v2, v3, c0, c1, c2, c3;
            load4_u64(lv.level[l], lv.size[l], j * kFanout + lane * 4, v0, v1, v2, v3);
            wave_prefix4(v0, v1, v2, v3, c0, c1, c2, c3);
            j = j * kFanout + pick_child(c0, c1, c2, c3, r);
        }
        // j is the tile holding r: the same over its 256 priorities.
        uint32_t p0, p1, p2, p3;
        uint64_t c0, c1, c2, c3;
        load4_u32(prio, N, j * kTile + lane * 4, p0, p1, p2, p3);
        wave_prefix4(p0, p1, p2, p3, c0, c1, c2, c3);
        const int cnt = pick_child(c0, c1, c2, c3, r);
        if (lane == 0) {
            idx[b] = (kShard ? sh.base : 0) + j * kTile + cnt;
            start[b] = (int32_t)scale_draw(splitmix64_out(seed, 2 * (uint64_t)b + 1), span);
        }
        if (want_min) {
            // The selected priority is kept for the weight kernel in the
            // caller's weight buffer, which that kernel then overwrites.
            const uint32_t pv = (uint32_t)read_lane(pick4(p0, p1, p2, p3, cnt & 3), cnt >> 2);
            my_min = pv < my_min ? pv : my_min;
            if (lane == 0) sel_prio[b] = pv;
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
// workgroup first reduces the search's per-workgroup minima.  The selected
// priority p_b arrives in w[b] itself (as uint32 bits; 0 marks a draw with
// no selectable slot) and is replaced by the weight.
__global__ __launch_bounds__(256) void is_weights_kernel(int32_t B, double beta, const uint32_t* __restrict__ wg_min,
                                                         int search_grid, float* __restrict__ w) {
    __shared__ uint32_t s_min[4];
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    // This draw's priority and the first eight minima per thread are loaded
    // together, from indices clamped into their buffers, before any is used:
    // one memory round trip covers the search's largest grid.
    constexpr int kMinPerThread = 8;
    const uint32_t pb_raw = reinterpret_cast<const uint32_t*>(w)[b < B ? b : B - 1];
    uint32_t v0[kMinPerThread];
#pragma unroll
    for (int u = 0; u < kMinPerThread; u++) {
        const int k = (int)threadIdx.x + u * (int)blockDim.x;
        v0[u] = wg_min[k < search_grid ? k : 0];
    }
    const uint32_t pb = b < B ? pb_raw : 0u;
    uint32_t m = 0xFFFFFFFFu;
#pragma unroll
    for (int u = 0; u < kMinPerThread; u++) {
        const int k = (int)threadIdx.x + u * (int)blockDim.x;
        m = (k < search_grid && v0[u] < m) ? v0[u] : m;
    }
    // Grids larger than blockDim * kMinPerThread (the table's chunk minima).
    for (int k0 = threadIdx.x + blockDim.x * kMinPerThread; k0 < search_grid; k0 += blockDim.x * kMinPerThread) {
        uint32_t v[kMinPerThread];
#pragma unroll
        for (int u = 0; u < kMinPerThread; u++) {
            const int k = k0 + u * (int)blockDim.x;
            v[u] = k < search_grid ? wg_min[k] : 0xFFFFFFFFu;
        }
#pragma unroll
        for (int u = 0; u < kMinPerThread; u++) m = v[u] < m ? v[u] : m;
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const uint32_t o = __shfl_xor(m, d);
        m = o < m ? o : m;
    }
    if ((threadIdx.x & 63) == 0) s_min[threadIdx.x >> 6] = m;
    __syncthreads();
    m = s_min[0];
    for (int k = 1; k < (int)(blockDim.x >> 6); k++) m = s_min[k] < m ? s_min[k] : m;
    if (b >= B) return;
    w[b] = (pb == 0u || m == 0u) ? 0.0f : (float)pow((double)m / (double)pb, beta);
}

constexpr int kSmallThreads = 1024;
constexpr int kSmallPerThread = (int)(kSmallN / kSmallThreads);  // consecutive priorities per thread
static_assert(kSmallN % (4 * kSmallThreads) == 0, "whole 16-byte loads per thread");

// LDS position of prefix entry e: one pad word after every run of
// kSmallPerThread entries, so that the lanes of a wave, each writing its own
// consecutive run, fall in different banks.
__device__ __forceinline__ int64_t small_pos(int64_t e) { return e + e / kSmallPerThread; }

// want_w: also compute weights (the selected priority waits in w[b] as
// uint32 bits, as in the multi-launch path).  global_min: normalise by the
// smallest non-zero priority of the table instead of the batch's.
__global__ __launch_bounds__(kSmallThreads) void small_select_kernel(const uint32_t* __restrict__ prio, int64_t N,
                                                                     int32_t B, uint64_t span, uint64_t seed,
                                                                     int want_w, int global_min, double beta,
                                                                     uint32_t* status, int64_t* __restrict__ idx,
                                                                     int32_t* __restrict__ start,
                                                                     float* __restrict__ w) {
    __shared__ uint64_t C[kSmallN + kSmallN / kSmallPerThread];
    __shared__ uint64_t s_wave[kSmallThreads / 64];
    __shared__ uint32_t s_min[kSmallThreads / 64];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int64_t e0 = (int64_t)t * kSmallPerThread;
    uint32_t v[kSmallPerThread];
#pragma unroll
    for (int k = 0; k < kSmallPerThread; k += 4) {
        if (e0 + k + 4 <= N) {
            const uint4 x = *reinterpret_cast<const uint4*>(prio + e0 + k);
            v[k] = x.x; v[k + 1] = x.y; v[k + 2] = x.z; v[k + 3] = x.w;
        } else {
#pragma unroll
            for (int q = 0; q < 4; q++) v[k + q] = e0 + k + q < N ? prio[e0 + k + q] : 0u;
        }
    }
    // Block-wide inclusive scan: this thread's run, then the waves in order.
    uint64_t run = 0;
    uint32_t pmin = 0xFFFFFFFFu;  // smallest non-zero priority of this thread's run
#pragma unroll
    for (int k = 0; k < kSmallPerThread; k++) {
        run += v[k];
        pmin = (v[k] != 0u && v[k] < pmin) ? v[k] : pmin;
    }
    const uint64_t incl = wave_inclusive_scan(run);
    if (lane == 63) s_wave[wave] = incl;
    __syncthreads();
    uint64_t acc = incl - run;
    for (int q = 0; q < wave; q++) acc += s_wave[q];
#pragma unroll
    for (int k = 0; k < kSmallPerThread; k++) {
        acc += v[k];
        if (e0 + k < N) C[small_pos(e0 + k)] = acc;
    }
    __syncthreads();
    const uint64_t S = C[small_pos(N - 1)];
    uint32_t m = 0xFFFFFFFFu;  // smallest selected priority (or of the table)
    for (int64_t b = t; b < B; b += kSmallThreads) {
        if (S == 0) {
            idx[b] = -1;
            start[b] = 0;
            if (want_w) reinterpret_cast<uint32_t*>(w)[b] = 0u;
            if (b == 0) atomicOr(status, GEAR_STATUS_NO_WEIGHT);
            continue;
        }
        const uint64_t r = scale_draw(splitmix64_out(seed, 2 * (uint64_t)b), S);
        int64_t lo = 0, hi = N;  // the smallest i with C_i > r lies in [lo, hi]
        while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            if (C[small_pos(mid)] > r) hi = mid;
            else lo = mid + 1;
        }
        const uint32_t pv = (uint32_t)(C[small_pos(lo)] - (lo > 0 ? C[small_pos(lo - 1)] : 0));
        idx[b] = lo;
        start[b] = (int32_t)scale_draw(splitmix64_out(seed, 2 * (uint64_t)b + 1), span);
        if (want_w) reinterpret_cast<uint32_t*>(w)[b] = pv;
        m = pv < m ? pv : m;
    }
    if (!want_w) return;
    if (global_min) m = pmin;
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const uint32_t o = __shfl_xor(m, d);
        m = o < m ? o : m;
    }
    if (lane == 0) s_min[wave] = m;
    __syncthreads();
    m = s_min[0];
    for (int q = 1; q < kSmallThreads / 64; q++) m = s_min[q] < m ? s_min[q] : m;
    for (int64_t b = t; b < B; b += kSmallThreads) {
        const uint32_t pb = reinterpret_cast<const uint32_t*>(w)[b];
        w[b] = (pb == 0u || m == 0u) ? 0.0f : (float)pow((double)m / (double)pb, beta);
    }
}

// FIFO / LIFO: ring arithmetic from the oldest / newest live position.
// Uniform: r = floor(u * n / 2^64) over the n live trajectories.
// A ring table's positions are its slots, and its live slots are [0, n).
// A managed table (index manager) reads the slot at each position of its
// commit-order ring `order`, oldest commit at `oldest`.
__global__ void simple_select_kernel(SimpleDraws d, int32_t B, int64_t* __restrict__ idx,
                                     int32_t* __restrict__ start, float* __restrict__ w) {
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    idx[b] = simple_slot(d, b);
    start[b] = simple_start(d, b);
    if (w) w[b] = 1.0f;
}

// The tree as the search sees it: level 0 and the copy of the upper levels
// that the last scan filled.
Levels tree(const Table& t) {
    Levels lv{};
    lv.nlevels = t.nlevels;
    for (int l = 0; l < t.nlevels; l++) {
        lv.level[l] = l == 0 ? t.tile_sums : t.upper[t.tree_parity][l];
        lv.size[l] = t.level_size[l];
    }
    return with_top(lv);
}

Levels upper_copy(const Table& t, int parity) {
    Levels lv{};
    lv.nlevels = t.nlevels;
    for (int l = 1; l < t.nlevels; l++) {
        lv.level[l] = t.upper[parity][l];
        lv.size[l] = t.level_size[l];
    }
    return lv;
}

}  // namespace

hipError_t launch_scan(Table& t, hipStream_t s) {
    // The copy this scan fills was zeroed by the previous scan (or at
    // creation); this scan zeroes the other copy for the next one.
    const int par = 1 - t.tree_parity;
    if (t.options & GEAR_OPT_IS_GLOBAL_MIN)
        hipLaunchKernelGGL(scan_kernel<true>, dim3((unsigned)t.nchunks), dim3(256), 0, s, t.priority, t.N,
                           upper_copy(t, par), upper_copy(t, 1 - par), t.tile_sums, t.ntiles, t.chunk_min);
    else
        hipLaunchKernelGGL(scan_kernel<false>, dim3((unsigned)t.nchunks), dim3(256), 0, s, t.priority, t.N,
                           upper_copy(t, par), upper_copy(t, 1 - par), t.tile_sums, t.ntiles, t.chunk_min);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) t.tree_parity = par;
    return e;
}

hipError_t launch_search(Table& t, int32_t B, int32_t L, uint64_t seed, bool want_min, int64_t* idx,
                         int32_t* start, uint32_t* sel_prio, int* grid_out, hipStream_t s,
                         const uint64_t* shard_totals, int G, int g, int64_t base) {
    int64_t gw = ((int64_t)B + 3) / 4;  // one wave per draw while the grid allows
    const int grid = (int)(gw < kSearchMaxGrid ? gw : kSearchMaxGrid);
    Shard sh;
    sh.totals = shard_totals;
    sh.G = G;
    sh.g = g;
    sh.base = base;
    if (shard_totals)
        hipLaunchKernelGGL(search_kernel<true>, dim3(grid), dim3(256), 0, s, t.priority, t.N, tree(t), B,
                           (uint64_t)(t.T - L + 1), seed, want_min ? 1 : 0, sh, t.wg_min, t.status, idx, start,
                           sel_prio);
    else
        hipLaunchKernelGGL(search_kernel<false>, dim3(grid), dim3(256), 0, s, t.priority, t.N, tree(t), B,
                           (uint64_t)(t.T - L + 1), seed, want_min ? 1 : 0, sh, t.wg_min, t.status, idx, start,
                           sel_prio);
    *grid_out = grid;
    return hipGetLastError();
}

hipError_t launch_is_weights(Table& t, int32_t B, float beta, int search_grid, float* w, hipStream_t s,
                             bool global_min) {
    // The minimum comes from the search's per-workgroup minima of the batch,
    // or from the scan's per-chunk minima of the whole table.
    hipLaunchKernelGGL(is_weights_kernel, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, s, B, (double)beta,
                       global_min ? t.chunk_min : t.wg_min, global_min ? (int)t.nchunks : search_grid, w);
    return hipGetLastError();
}

bool small_select_applies(const Table& t, int32_t B) {
    return t.N <= kSmallN && B <= kSmallMaxB && !(t.options & GEAR_OPT_INCREMENTAL_TREE);
}

hipError_t launch_small_select(Table& t, int32_t B, int32_t L, uint64_t seed, float beta, int64_t* idx,
                               int32_t* start, float* w, hipStream_t s) {
    hipLaunchKernelGGL(small_select_kernel, dim3(1), dim3(kSmallThreads), 0, s, t.priority, t.N, B,
                       (uint64_t)(t.T - L + 1), seed, w ? 1 : 0, (t.options & GEAR_OPT_IS_GLOBAL_MIN) ? 1 : 0,
                       (double)beta, t.status, idx, start, w);
    return hipGetLastError();
}

SimpleDraws simple_draws(const Table& t, int32_t strategy, int32_t L, uint64_t seed) {
    SimpleDraws d{};
    d.strategy = strategy;
    d.N = t.N;
    d.live = live_count(t);
    if (t.managed) {
        d.oldest = t.ord_head;
        d.newest = (t.ord_head + d.live - 1) % t.N;
    } else {
        d.oldest = (int64_t)((t.next_seq - (uint64_t)d.live) % (uint64_t)t.N);
        d.newest = (int64_t)((t.next_seq - 1) % (uint64_t)t.N);
    }
    d.order = t.managed ? t.order : nullptr;
    d.span = (uint64_t)(t.T - L + 1);
    d.seed = seed;
    return d;
}

hipError_t launch_simple_select(Table& t, int32_t strategy, int32_t B, int32_t L, uint64_t seed, int64_t* idx,
                                int32_t* start, float* w, hipStream_t s) {
    hipLaunchKernelGGL(simple_select_kernel, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, s,
                       simple_draws(t, strategy, L, seed), B, idx, start, w);
    return hipGetLastError();
}

}  // namespace gear

using gear::fail;
using gear::hip_fail;

extern "C" int gear_select(gear_table* h, int32_t strategy, int32_t B, int32_t L, uint64_t seed, float beta,
                           int64_t* d_idx, int32_t* d_start, float* d_weights, void* stream) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_select: table is NULL");
    gear::Table* t = reinterpret_cast<gear::Table*>(h);
    if (strategy < GEAR_FIFO || strategy > GEAR_TOPK) return fail(GEAR_E_INVAL, "gear_select: unknown strategy");
    if (strategy == GEAR_TOPK && B > GEAR_MAX_TOPK) return fail(GEAR_E_INVAL, "gear_select: TopK batch above GEAR_MAX_TOPK");
    if (B < 1 || B > GEAR_MAX_BATCH) return fail(GEAR_E_INVAL, "gear_select: B out of range");
    if (L < 1 || L > t->T) return fail(GEAR_E_INVAL, "gear_select: L must lie in [1, T]");
    if (d_idx == nullptr || d_start == nullptr) return fail(GEAR_E_INVAL, "gear_select: output pointer is NULL");
    if (!(beta == beta)) return fail(GEAR_E_INVAL, "gear_select: beta is NaN");
    const int64_t live = gear::live_count(*t);
    if (live == 0) return fail(GEAR_E_EMPTY, "gear_select: nothing inserted");
    if ((strategy == GEAR_FIFO || strategy == GEAR_LIFO) && (int64_t)B > live)
        return fail(GEAR_E_INSUFFICIENT, "gear_select: FIFO/LIFO batch larger than the live count");
    gear::DeviceGuard guard(t->device);
    if (guard.error() != hipSuccess) return hip_fail(guard.error(), "gear_select: hipSetDevice");
    hipStream_t s = static_cast<hipStream_t>(stream);

    if (strategy == GEAR_TOPK) {
        hipError_t e = gear::launch_topk(*t, B, L, seed, d_idx, d_start, d_weights, s);
        return e == hipSuccess ? GEAR_OK : hip_fail(e, "gear_select: TopK launch");
    }
    if (strategy != GEAR_PRIORITIZED) {
        hipError_t e = gear::launch_simple_select(*t, strategy, B, L, seed, d_idx, d_start, d_weights, s);
        return e == hipSuccess ? GEAR_OK : hip_fail(e, "gear_select: launch");
    }
    if (gear::small_select_applies(*t, B)) {
        // One launch; the sum tree is left as it is (still marked for a rescan if stale).
        hipError_t e = gear::launch_small_select(*t, B, L, seed, beta, d_idx, d_start, d_weights, s);
        return e == hipSuccess ? GEAR_OK : hip_fail(e, "gear_select: small-table launch");
    }
    if (t->cdf_dirty) {
        hipError_t e = gear::launch_scan(*t, s);
        if (e != hipSuccess) return hip_fail(e, "gear_select: scan launch");
        t->cdf_dirty = false;
    }
    const bool weights = d_weights != nullptr;
    int grid = 0;
    hipError_t e = gear::launch_search(*t, B, L, seed, weights, d_idx, d_start,
                                       reinterpret_cast<uint32_t*>(d_weights), &grid, s);
    if (e != hipSuccess) return hip_fail(e, "gear_select: search launch");
    if (weights) {
        e = gear::launch_is_weights(*t, B, beta, grid, d_weights, s, (t->options & GEAR_OPT_IS_GLOBAL_MIN) != 0);
        if (e != hipSuccess) return hip_fail(e, "gear_select: weight launch");
    }
    return GEAR_OK;
}

// ---------------------------------------------------------------------------
// Prioritized selection without allocation: the kernels above, run over a
// caller's priority array with the sum tree, the per-workgroup minima and
// the status word in a fixed file-scope device array instead of table
// memory.  For callers that cannot allocate (graph capture, serving loops).
// ---------------------------------------------------------------------------
namespace gear {
namespace {

constexpr int64_t kNaTiles = GEAR_NOALLOC_MAX_N / kTile;            // level 0 entries
constexpr int64_t kNaLevel1 = (kNaTiles + kFanout - 1) / kFanout;     // level 1 entries (the top)
static_assert(kNaLevel1 <= kFanout, "two levels cover every allowed table");
static_assert(GEAR_NOALLOC_MAX_N % (kTile * kTilesPerChunk) == 0, "whole scan chunks");
// Layout in 64-bit words: tile sums | level 1 (the scan adds into it) |
// level 1 spare (the scan's zeroing target, never read) | wg_min (uint32) |
// status (uint32).
constexpr int64_t kNaOffTiles = 0;
constexpr int64_t kNaOffLevel1 = kNaOffTiles + kNaTiles;
constexpr int64_t kNaOffSpare = kNaOffLevel1 + kFanout;
constexpr int64_t kNaOffMin = kNaOffSpare + kFanout;
constexpr int64_t kNaOffStatus = kNaOffMin + kSearchMaxGrid / 2;
constexpr int64_t kNaWords = (kNaOffStatus + 1 + 31) / 32 * 32;
static_assert(kNaWords * 8 == GEAR_NOALLOC_SCRATCH_BYTES, "header states the scratch size");

// Holds every call's scratch on each device, until the process ends.
static __device__ __align__(256) uint64_t scratch[kNaWords];

// Device address of `scratch` on each device, looked up once per device
// with that device current (host code must not pass the symbol itself).
constexpr int kNaMaxDevices = 64;
std::mutex g_na_mutex;
uint64_t* g_na_ptr[kNaMaxDevices] = {};

// Zeroes the level-1 nodes the scan accumulates into and the status word:
// a kernel, not a memset, so that a captured graph replays it faithfully.
__global__ void noalloc_clear_kernel(uint64_t* __restrict__ level1, uint32_t* __restrict__ status) {
    const int k = threadIdx.x;
    if (k < kFanout) level1[k] = 0;
    if (k == 0) *status = 0u;
}

hipError_t noalloc_scratch(int dev, uint64_t** out) {
    std::lock_guard<std::mutex> lock(g_na_mutex);
    if (g_na_ptr[dev] == nullptr) {
        void* p = nullptr;
        hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_na_ptr[dev] = static_cast<uint64_t*>(p);
    }
    *out = g_na_ptr[dev];
    return hipSuccess;
}

}  // namespace
}  // namespace gear

extern "C" int gear_select_prioritized_noalloc(const uint32_t* d_priority, int64_t N, int32_t T, int32_t B,
                                               int32_t L, uint64_t seed, float beta, int64_t* d_idx,
                                               int32_t* d_start, float* d_weights, void* stream) {
    using namespace gear;
    if (d_priority == nullptr || d_idx == nullptr || d_start == nullptr)
        return fail(GEAR_E_INVAL, "gear_select_prioritized_noalloc: NULL pointer argument");
    if (N < 1 || N > GEAR_NOALLOC_MAX_N)
        return fail(GEAR_E_INVAL, "gear_select_prioritized_noalloc: N must lie in [1, GEAR_NOALLOC_MAX_N]");
    if (B < 1 || B > GEAR_MAX_BATCH) return fail(GEAR_E_INVAL, "gear_select_prioritized_noalloc: B out of range");
    if (T < 1 || L < 1 || L > T) return fail(GEAR_E_INVAL, "gear_select_prioritized_noalloc: L must lie in [1, T]");
    if (!(beta == beta)) return fail(GEAR_E_INVAL, "gear_select_prioritized_noalloc: beta is NaN");
    (void)hipGetLastError();  // an error pending from an earlier HIP call is not this call's
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "gear_select_prioritized_noalloc: hipGetDevice");
    if (dev < 0 || dev >= kNaMaxDevices) return fail(GEAR_E_INVAL, "gear_select_prioritized_noalloc: device ordinal above 63");
    uint64_t* base = nullptr;
    e = noalloc_scratch(dev, &base);
    if (e != hipSuccess) return hip_fail(e, "gear_select_prioritized_noalloc: hipGetSymbolAddress");
    uint32_t* status = reinterpret_cast<uint32_t*>(base + kNaOffStatus);
    uint32_t* wg_min = reinterpret_cast<uint32_t*>(base + kNaOffMin);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const uint64_t span = (uint64_t)(T - L + 1);

    if (N <= kSmallN && B <= kSmallMaxB) {
        // One launch, as gear_select takes for a table this small.
        hipLaunchKernelGGL(small_select_kernel, dim3(1), dim3(kSmallThreads), 0, s, d_priority, N, B, span, seed,
                           d_weights ? 1 : 0, 0, (double)beta, status, d_idx, d_start, d_weights);
        e = hipGetLastError();
        return e == hipSuccess ? GEAR_OK : hip_fail(e, "gear_select_prioritized_noalloc: small-table launch");
    }
    const int64_t ntiles = (N + kTile - 1) / kTile;
    const int64_t nchunks = (ntiles + kTilesPerChunk - 1) / kTilesPerChunk;
    Levels lv{}, upper{}, spare{};
    lv.nlevels = ntiles > kFanout ? 2 : 1;
    lv.level[0] = base + kNaOffTiles;
    lv.size[0] = ntiles;
    upper.nlevels = spare.nlevels = lv.nlevels;
    if (lv.nlevels == 2) {
        lv.level[1] = upper.level[1] = base + kNaOffLevel1;
        spare.level[1] = base + kNaOffSpare;
        lv.size[1] = upper.size[1] = spare.size[1] = (ntiles + kFanout - 1) / kFanout;
    }
    const char* what = "gear_select_prioritized_noalloc: clear launch";
    hipLaunchKernelGGL(noalloc_clear_kernel, dim3(1), dim3(kFanout), 0, s, base + kNaOffLevel1, status);
    if ((e = hipGetLastError()) == hipSuccess) {
        what = "gear_select_prioritized_noalloc: scan launch";
        hipLaunchKernelGGL(scan_kernel<false>, dim3((unsigned)nchunks), dim3(256), 0, s, d_priority, N, upper, spare,
                           lv.level[0], ntiles, static_cast<uint32_t*>(nullptr));
        e = hipGetLastError();
    }
    const int64_t gw = ((int64_t)B + 3) / 4;
    const int grid = (int)(gw < kSearchMaxGrid ? gw : kSearchMaxGrid);
    if (e == hipSuccess) {
        what = "gear_select_prioritized_noalloc: search launch";
        Shard sh{};
        sh.G = 1;
        hipLaunchKernelGGL(search_kernel<false>, dim3(grid), dim3(256), 0, s, d_priority, N, with_top(lv), B, span,
                           seed, d_weights ? 1 : 0, sh, wg_min, status, d_idx, d_start,
                           reinterpret_cast<uint32_t*>(d_weights));
        e = hipGetLastError();
    }
    if (e == hipSuccess && d_weights) {
        what = "gear_select_prioritized_noalloc: weight launch";
        hipLaunchKernelGGL(is_weights_kernel, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, s, B, (double)beta,
                           static_cast<const uint32_t*>(wg_min), grid, d_weights);
        e = hipGetLastError();
    }
    return e == hipSuccess ? GEAR_OK : hip_fail(e, what);
}
