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
// list, the number of entries that come before it there (a binary search):
// O(G*K*G*log K) work, no sort.
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

// Thread t: entry j = t mod K of list g = t / K.  Lists are sorted in
// candidate order with their -1 entries last.
__global__ void merge_kernel(const uint32_t* __restrict__ prio, const int64_t* __restrict__ gidx, int32_t G,
                             int32_t K, uint64_t span, uint64_t seed, int64_t* __restrict__ idx,
                             int32_t* __restrict__ start, float* __restrict__ w, uint32_t* __restrict__ out_prio) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)G * K) return;
    const int g = (int)(t / K);
    const int64_t i = gidx[t];
    if (i < 0) return;
    const uint32_t p = prio[t];
    int64_t place = t - (int64_t)g * K;
    for (int h = 0; h < G && place < K; h++) {
        if (h == g) continue;
        const uint32_t* ph = prio + (int64_t)h * K;
        const int64_t* ih = gidx + (int64_t)h * K;
        int lo = 0, hi = K;  // first entry of list h that does not come before (p, i)
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            const int64_t im = ih[mid];
            if (im >= 0 && before(ph[mid], im, p, i))
                lo = mid + 1;
            else
                hi = mid;
        }
        place += lo;
    }
    if (place >= K) return;
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
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipLaunchKernelGGL(gear::merge_fill_kernel, dim3(gear::blocks_for(K)), dim3(256), 0, s, K, d_idx, d_start,
                       d_weights, d_out_prio);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) {
        hipLaunchKernelGGL(gear::merge_kernel, dim3(gear::blocks_for((int64_t)G * K)), dim3(256), 0, s, d_prio, d_gidx,
                           G, K, (uint64_t)(T - L + 1), seed, d_idx, d_start, d_weights, d_out_prio);
        e = hipGetLastError();
    }
    if (e != hipSuccess) return hip_fail(e, "gear_topk_merge: launch");
    return GEAR_OK;
}
