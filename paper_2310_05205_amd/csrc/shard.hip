// One GPU's share of selection over G shards (GEAR Sec. 3.3, centralized
// and decentralized trajectory selection; Sec. 3.4, global index =
// shard * capacity + local index).
//
// Prioritized (weighted) selection needs one exchange of G numbers instead
// of gathering all weights on one GPU: every shard publishes the total of
// its priorities (gear_shard_total), the totals are all-gathered, and every
// shard draws the same r_b over the sum of the totals and resolves the draws
// that fall into its own prefix range (gear_select_shard).  The union of the
// shards' answers equals selection over the concatenated table.  After an
// all-reduce of the selected priorities (each draw is owned by one shard),
// every shard computes the same importance-sampling weights
// (gear_is_weights).
//
// TopK (decentralized): every shard computes its local top-K, sorted; one
// GPU merges the G sorted lists (gear_topk_merge).  A candidate's place in
// the merged order is its place in its own list plus, for every other
// list, the number of entries that come before it there: no sort.
#include "gear_internal.h"
#include "wave.h"

namespace gear {
namespace {

constexpr int kMaxShards = 4096;

// Sum of the top level of the tree (at most 256 nodes), by one wave.
__global__ void tree_total_kernel(const uint64_t* __restrict__ top, int64_t n, uint64_t* __restrict__ out) {
    uint64_t v = 0;
    for (int64_t k = threadIdx.x; k < n; k += 64) v += top[k];
    v = wave_sum(v);
    if (threadIdx.x == 0) *out = v;
}

// The selected priorities go to the weight buffer as uint32 bits (read by
// the weight kernel) and each workgroup's smallest non-zero one to wg_min.
__global__ __launch_bounds__(256) void batch_min_kernel(const uint32_t* __restrict__ p, int32_t B,
                                                        uint32_t* __restrict__ w_bits, uint32_t* __restrict__ wg_min) {
    __shared__ uint32_t s_min[4];
    uint32_t m = 0xFFFFFFFFu;
    for (int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; b < B; b += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t v = p[b];
        w_bits[b] = v;
        if (v != 0u && v < m) m = v;
    }
    for (int off = 32; off > 0; off >>= 1) {
        const uint32_t o = (uint32_t)__shfl_xor((int)m, off);
        m = o < m ? o : m;
    }
    if ((threadIdx.x & 63) == 0) s_min[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = s_min[0];
        for (int k = 1; k < (int)(blockDim.x >> 6); k++) r = s_min[k] < r ? s_min[k] : r;
        wg_min[blockIdx.x] = r;
    }
}

// Candidate order of TopK: higher priority first, then lower global index.
__device__ __forceinline__ bool before(uint32_t pa, int64_t ia, uint32_t pb, int64_t ib) {
    return pa > pb || (pa == pb && ia < ib);
}

__global__ void merge_fill_kernel(int32_t K, int64_t* __restrict__ idx, int32_t* __restrict__ start,
                                  float* __restrict__ w, uint32_t* __restrict__ out_prio) {
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= K) return;
    idx[k] = -1;
    start[k] = 0;
    if (w) w[k] = 0.0f;
    if (out_prio) out_prio[k] = 0u;
}

// Merge of G sorted lists by ranks.  A workgroup takes a tile of
// kMergeTile consecutive entries of list g, kMergeParts threads per entry.
// The entries of another list h that come before a tile entry are all of h
// up to a point that moves forward along the tile, so for the whole tile
// they lie between two positions of h: the ranks in h of the tile's first
// and last valid entries.  Those two ranks, for every other list of a round
// of kMergeRound lists, are found by cooperative searches of kProbeLanes
// lanes each; the entries between them (the bracket) go to LDS; and each
// thread finishes the ranks of its entry in its share of the round's lists
// by binary searches in LDS.  A bracket that does not fit in LDS is
// searched in global memory instead.  Binary searches by every thread
// straight over global memory cost about eight times more load
// instructions; one thread per entry leaves one wave per SIMD.
constexpr int kMergeThreads = 256;
constexpr int kMergeParts = 4;                          // threads per tile entry
constexpr int kMergeTile = kMergeThreads / kMergeParts;  // 64 entries
constexpr int kMergeRound = 8;                           // lists per round: 2 * 8 searches, 4 per wave
constexpr int kListsPerPart = kMergeRound / kMergeParts;
constexpr int kProbeLanes = 16;                          // lanes per cooperative search
constexpr int kBracketCap = 1024;                        // bracket entries in LDS per round (12 KiB)
constexpr int kFillPerThread = kBracketCap / kMergeThreads;

// Entries of list (ph, ih) of length K that come before (p, i), by the 16
// lanes of group `grp` of the wave (lane `sub` within it).  Valid entries
// form a sorted prefix, so "comes before" is true on a prefix of positions.
// Each round probes 15 evenly spaced positions of the remaining range and
// keeps the piece between the last probe that comes before and the first
// that does not; a range of at most 16 positions is probed whole.  Every
// lane of the wave must call this (the rounds use wave ballots).
__device__ int group_count_before(const uint32_t* __restrict__ ph, const int64_t* __restrict__ ih, int K, uint32_t p,
                                  int64_t i, bool active, int grp, int sub) {
    int lo = 0, hi = K;  // the count lies in [lo, hi]
    bool done = !active;
    int count = 0;
    while (__ballot(!done) != 0) {
        const int n = hi - lo;
        const bool whole = n <= kProbeLanes;
        const int q = whole ? lo + sub : lo + ((sub + 1) * n) / kProbeLanes - 1;
        bool pred = false;
        if (!done && sub < (whole ? n : kProbeLanes - 1)) {
            const int64_t iq = ih[q];  // both loads issued before either is used
            const uint32_t pq = ph[q];
            pred = (iq >= 0) & before(pq, iq, p, i);
        }
        const int c = __popcll((__ballot(pred) >> (grp * kProbeLanes)) & 0xFFFFull);
        if (!done) {
            if (whole) {
                count = lo + c;
                done = true;
            } else {
                const int nlo = c > 0 ? lo + (c * n) / kProbeLanes : lo;
                const int nhi = c < kProbeLanes - 1 ? lo + ((c + 1) * n) / kProbeLanes - 1 : hi;
                lo = nlo;
                hi = nhi;
            }
        }
    }
    return count;
}

__global__ __launch_bounds__(kMergeThreads) void merge_kernel(const uint32_t* __restrict__ prio,
                                                              const int64_t* __restrict__ gidx, int32_t G, int32_t K,
                                                              uint64_t span, uint64_t seed, int64_t* __restrict__ idx,
                                                              int32_t* __restrict__ start, float* __restrict__ w,
                                                              uint32_t* __restrict__ out_prio) {
    __shared__ uint32_t s_p[kBracketCap];
    __shared__ int64_t s_i[kBracketCap];
    __shared__ int s_lo[kMergeRound], s_hi[kMergeRound], s_off[kMergeRound];
    __shared__ int s_steps;
    __shared__ uint32_t s_kp[2];
    __shared__ int64_t s_ki[2];
    const int tiles = (K + kMergeTile - 1) / kMergeTile;
    const int g = (int)(blockIdx.x / tiles);
    const int entry = (int)threadIdx.x / kMergeParts, part = (int)threadIdx.x % kMergeParts;
    const int j = (int)(blockIdx.x % tiles) * kMergeTile + entry;
    const int64_t at = (int64_t)g * K + j;
    const int64_t i = j < K ? gidx[at] : -1;
    const uint32_t p = j < K ? prio[at] : 0u;
    // Valid entries are a prefix of the list, hence of the tile.
    const int nvalid = __syncthreads_count(i >= 0 && part == 0);
    if (nvalid == 0) return;
    if (threadIdx.x == 0) {
        s_kp[0] = p;
        s_ki[0] = i;
    }
    if ((int)threadIdx.x == (nvalid - 1) * kMergeParts) {
        s_kp[1] = p;
        s_ki[1] = i;
    }
    __syncthreads();
    const int wave = (int)threadIdx.x >> 6, lane = (int)threadIdx.x & 63;
    const int grp = lane / kProbeLanes, sub = lane % kProbeLanes;
    const int search = wave * (64 / kProbeLanes) + grp;  // 0 .. 2 * kMergeRound - 1
    const int su = search >> 1, end = search & 1;         // list in the round; 0: first entry, 1: last entry
    int count = 0;
    for (int h0 = 0; h0 < G; h0 += kMergeRound) {
        {
            const int h = h0 + su;
            const bool act = h < G && h != g;
            const int r = group_count_before(prio + (int64_t)(act ? h : 0) * K, gidx + (int64_t)(act ? h : 0) * K, K,
                                             s_kp[end], s_ki[end], act, grp, sub);
            if (act && sub == 0) (end ? s_hi : s_lo)[su] = r;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            int used = 0, widest = 0;
            for (int u = 0; u < kMergeRound; u++) {
                const int h = h0 + u;
                if (h >= G || h == g) {
                    s_lo[u] = s_hi[u] = 0;
                    s_off[u] = 0;
                    continue;
                }
                const int wdt = s_hi[u] - s_lo[u];
                widest = wdt > widest ? wdt : widest;
                if (used + wdt <= kBracketCap) {
                    s_off[u] = used;
                    used += wdt;
                } else {
                    s_off[u] = -1;
                }
            }
            s_steps = 32 - __clz((unsigned)widest);  // halvings that empty the widest bracket
        }
        __syncthreads();
        int r_off[kMergeRound], r_lo[kMergeRound], r_w[kMergeRound];
#pragma unroll
        for (int u = 0; u < kMergeRound; u++) {
            r_off[u] = s_off[u];
            r_lo[u] = s_lo[u];
            r_w[u] = s_hi[u] - s_lo[u];
        }
        {
            // Every bracket entry of the round, kFillPerThread per thread at
            // most: all loads are issued before the first LDS store.
            uint32_t vp[kFillPerThread];
            int64_t vi[kFillPerThread];
            int dst[kFillPerThread];
#pragma unroll
            for (int k = 0; k < kFillPerThread; k++) {
                const int e = (int)threadIdx.x + k * kMergeThreads;
                dst[k] = -1;
                int64_t a = 0;
#pragma unroll
                for (int u = 0; u < kMergeRound; u++) {
                    if (r_off[u] >= 0 && e >= r_off[u] && e < r_off[u] + r_w[u]) {
                        a = (int64_t)(h0 + u) * K + r_lo[u] + (e - r_off[u]);
                        dst[k] = e;
                    }
                }
                if (dst[k] >= 0) {
                    vp[k] = prio[a];
                    vi[k] = gidx[a];
                }
            }
#pragma unroll
            for (int k = 0; k < kFillPerThread; k++) {
                if (dst[k] >= 0) {
                    s_p[dst[k]] = vp[k];
                    s_i[dst[k]] = vi[k];
                }
            }
        }
        __syncthreads();
        if (i >= 0) {
            // This thread's lists of the round: part, part + kMergeParts, ...
            int lo[kListsPerPart], hi[kListsPerPart];
#pragma unroll
            for (int v = 0; v < kListsPerPart; v++) {
                lo[v] = 0;
                hi[v] = r_w[part + v * kMergeParts];
            }
            const int steps = s_steps;
            for (int step = 0; step < steps; step++) {
#pragma unroll
                for (int v = 0; v < kListsPerPart; v++) {
                    if (lo[v] < hi[v]) {
                        const int u = part + v * kMergeParts;
                        const int mid = (lo[v] + hi[v]) >> 1;
                        uint32_t pm;
                        int64_t im;
                        if (r_off[u] >= 0) {
                            pm = s_p[r_off[u] + mid];
                            im = s_i[r_off[u] + mid];
                        } else {
                            const int64_t a = (int64_t)(h0 + u) * K + r_lo[u] + mid;
                            pm = prio[a];
                            im = gidx[a];
                        }
                        if (before(pm, im, p, i))
                            lo[v] = mid + 1;
                        else
                            hi[v] = mid;
                    }
                }
            }
#pragma unroll
            for (int v = 0; v < kListsPerPart; v++) count += r_lo[part + v * kMergeParts] + lo[v];
        }
        __syncthreads();  // the next round overwrites the brackets
    }
    // The parts of one entry are adjacent lanes of one wave.
    for (int off = kMergeParts >> 1; off > 0; off >>= 1) count += __shfl_xor(count, off);
    const int64_t place = (int64_t)j + count;
    if (i < 0 || part != 0 || place >= K) return;
    idx[place] = i;
    start[place] = (int32_t)scale_draw(splitmix64_out(seed, 2 * (uint64_t)place + 1), span);
    if (w) w[place] = 1.0f;
    if (out_prio) out_prio[place] = p;
}

unsigned blocks_for(int64_t n) { return (unsigned)((n + 255) / 256); }

}  // namespace
}  // namespace gear

using gear::fail;
using gear::hip_fail;
using gear::Table;

extern "C" int gear_shard_total(gear_table* h, uint64_t* d_total, void* stream) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_shard_total: table is NULL");
    if (d_total == nullptr) return fail(GEAR_E_INVAL, "gear_shard_total: d_total is NULL");
    Table* t = reinterpret_cast<Table*>(h);
    gear::DeviceGuard guard(t->device);
    if (guard.error() != hipSuccess) return hip_fail(guard.error(), "gear_shard_total: hipSetDevice");
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (t->cdf_dirty) {
        if ((e = gear::launch_scan(*t, s)) != hipSuccess) return hip_fail(e, "gear_shard_total: scan launch");
        t->cdf_dirty = false;
    }
    const int top = t->nlevels - 1;
    const uint64_t* lv = top == 0 ? t->tile_sums : t->upper[t->tree_parity][top];
    hipLaunchKernelGGL(gear::tree_total_kernel, dim3(1), dim3(64), 0, s, lv, t->level_size[top], d_total);
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "gear_shard_total: launch");
    return GEAR_OK;
}

extern "C" int gear_select_shard(gear_table* h, int32_t G, int32_t g, const uint64_t* d_totals, int64_t base,
                                 int32_t B, int32_t L, uint64_t seed, int64_t* d_idx, int32_t* d_start,
                                 uint32_t* d_sel_prio, void* stream) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_select_shard: table is NULL");
    Table* t = reinterpret_cast<Table*>(h);
    if (G < 1 || G > gear::kMaxShards || g < 0 || g >= G) return fail(GEAR_E_INVAL, "gear_select_shard: need 0 <= g < G <= 4096");
    if (d_totals == nullptr || d_idx == nullptr || d_start == nullptr)
        return fail(GEAR_E_INVAL, "gear_select_shard: NULL pointer argument");
    if (base < 0) return fail(GEAR_E_INVAL, "gear_select_shard: base < 0");
    if (B < 1 || B > GEAR_MAX_BATCH) return fail(GEAR_E_INVAL, "gear_select_shard: B out of range");
    if (L < 1 || L > t->T) return fail(GEAR_E_INVAL, "gear_select_shard: L must lie in [1, T]");
    gear::DeviceGuard guard(t->device);
    if (guard.error() != hipSuccess) return hip_fail(guard.error(), "gear_select_shard: hipSetDevice");
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (t->cdf_dirty) {
        if ((e = gear::launch_scan(*t, s)) != hipSuccess) return hip_fail(e, "gear_select_shard: scan launch");
        t->cdf_dirty = false;
    }
    int grid = 0;
    e = gear::launch_search(*t, B, L, seed, d_sel_prio != nullptr, d_idx, d_start, d_sel_prio, &grid, s, d_totals, G,
                            g, base);
    if (e != hipSuccess) return hip_fail(e, "gear_select_shard: search launch");
    return GEAR_OK;
}

extern "C" int gear_is_weights(gear_table* h, const uint32_t* d_sel_prio, int32_t B, float beta, float* d_weights,
                               void* stream) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_is_weights: table is NULL");
    Table* t = reinterpret_cast<Table*>(h);
    if (d_sel_prio == nullptr || d_weights == nullptr) return fail(GEAR_E_INVAL, "gear_is_weights: NULL pointer argument");
    if (B < 1 || B > GEAR_MAX_BATCH) return fail(GEAR_E_INVAL, "gear_is_weights: B out of range");
    if (!(beta == beta)) return fail(GEAR_E_INVAL, "gear_is_weights: beta is NaN");
    gear::DeviceGuard guard(t->device);
    if (guard.error() != hipSuccess) return hip_fail(guard.error(), "gear_is_weights: hipSetDevice");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int64_t bl = ((int64_t)B + 255) / 256;
    const int grid = (int)(bl < gear::kSearchMaxGrid ? bl : gear::kSearchMaxGrid);
    hipLaunchKernelGGL(gear::batch_min_kernel, dim3(grid), dim3(256), 0, s, d_sel_prio, B,
                       reinterpret_cast<uint32_t*>(d_weights), t->wg_min);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) e = gear::launch_is_weights(*t, B, beta, grid, d_weights, s);
    if (e != hipSuccess) return hip_fail(e, "gear_is_weights: launch");
    return GEAR_OK;
}

extern "C" int gear_topk_merge(const uint32_t* d_prio, const int64_t* d_gidx, int32_t G, int32_t K, int32_t T,
                               int32_t L, uint64_t seed, int64_t* d_idx, int32_t* d_start, float* d_weights,
                               uint32_t* d_out_prio, void* stream) {
    if (G < 1 || G > gear::kMaxShards) return fail(GEAR_E_INVAL, "gear_topk_merge: G out of range");
    if (K < 1 || K > GEAR_MAX_TOPK) return fail(GEAR_E_INVAL, "gear_topk_merge: K out of range");
    if (T < 1 || L < 1 || L > T) return fail(GEAR_E_INVAL, "gear_topk_merge: L must lie in [1, T]");
    if (d_prio == nullptr || d_gidx == nullptr || d_idx == nullptr || d_start == nullptr)
        return fail(GEAR_E_INVAL, "gear_topk_merge: NULL pointer argument");
    (void)hipGetLastError();  // an error pending from an earlier HIP call is not this call's
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipLaunchKernelGGL(gear::merge_fill_kernel, dim3(gear::blocks_for(K)), dim3(256), 0, s, K, d_idx, d_start,
                       d_weights, d_out_prio);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) {
        const int64_t tiles = ((int64_t)K + gear::kMergeTile - 1) / gear::kMergeTile;
        hipLaunchKernelGGL(gear::merge_kernel, dim3((unsigned)(G * tiles)), dim3(gear::kMergeThreads), 0, s, d_prio, d_gidx,
                           G, K, (uint64_t)(T - L + 1), seed, d_idx, d_start, d_weights, d_out_prio);
        e = hipGetLastError();
    }
    if (e != hipSuccess) return hip_fail(e, "gear_topk_merge: launch");
    return GEAR_OK;
}
