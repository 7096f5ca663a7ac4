// TopK selection on gfx950 (GEAR Sec. 3.3, decentralized selection: TopK
// is deterministic; each GPU computes its top-K priority trajectories).
//
// The K highest priorities among slots with non-zero priority, higher
// priority first, the lower slot first among equal priorities.  The K-th
// largest priority P* is found by a radix select over the 32-bit priority in
// three digit passes (bits 31..21, 20..10, 9..0):
//
//   topk_hist_kernel  (x3) a workgroup histograms one digit of the
//                     priorities whose higher digits match the ones already
//                     chosen; a wave whose lanes all fall into one bin adds
//                     with a single LDS atomic (skewed priorities pile into
//                     few bins).  The last workgroup to finish (one ticket
//                     per workgroup) picks the bin that holds the K-th
//                     largest, records how many of that bin are still to be
//                     taken, and clears the histogram for the next call.
//   topk_count_kernel per workgroup: how many priorities are > P* and == P*.
//   topk_compact      every workgroup derives its output offsets from those
//                     counts and writes keys (p << 32 | ~slot) of all slots
//                     above P* and of the lowest-slot ties at P*.
//   topk_sort_kernel  one workgroup sorts the K keys (bitonic, in LDS),
//                     descending, and writes slots, window starts, weights.
#include "gear_internal.h"
#include "wave.h"

namespace gear {
namespace {

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / 64;

struct TopkState {
    uint32_t prefix;  // chosen high digits of the K-th largest priority
    uint32_t k_rem;   // of the priorities matching `prefix`, how many are still to be taken
    uint32_t all;     // 1: fewer than K slots have non-zero priority, take all of them
    uint32_t total;   // number of slots with non-zero priority
};

__device__ __forceinline__ int pass_shift(int pass) { return pass == 0 ? 21 : (pass == 1 ? 10 : 0); }
__device__ __forceinline__ int pass_bits(int pass) { return pass == 2 ? 10 : 11; }

// Slots [blockIdx.x * chunk, ...) of this workgroup; chunk is a multiple of
// 4 so every 16-byte load is aligned.
__device__ __forceinline__ void wg_range(int64_t N, int64_t chunk, int64_t& lo, int64_t& hi) {
    lo = (int64_t)blockIdx.x * chunk;
    hi = lo + chunk < N ? lo + chunk : N;
}

// One batch: kVec 16-byte loads per thread, all issued before any is used;
// thread t, load k covers slots base + (k * kTopkThreads + t) * 4 .. +3,
// and slots at or past `hi` read as priority 0 (never a candidate).
constexpr int kVec = 8;
constexpr int64_t kBatch = (int64_t)kVec * kTopkThreads * 4;

__device__ __forceinline__ void load_batch(const uint32_t* __restrict__ prio, int64_t base, int64_t hi,
                                           uint32_t v[kVec][4]) {
#pragma unroll
    for (int k = 0; k < kVec; k++) {
        const int64_t e = base + ((int64_t)k * kTopkThreads + threadIdx.x) * 4;
        if (e + 4 <= hi) {
            const uint4 x = *reinterpret_cast<const uint4*>(prio + e);
            v[k][0] = x.x; v[k][1] = x.y; v[k][2] = x.z; v[k][3] = x.w;
        } else {
#pragma unroll
            for (int q = 0; q < 4; q++) v[k][q] = e + q < hi ? prio[e + q] : 0u;
        }
    }
}

__global__ __launch_bounds__(kTopkThreads) void topk_hist_kernel(const uint32_t* __restrict__ prio, int64_t N,
                                                                 int64_t chunk, int pass, uint32_t K,
                                                                 uint32_t* __restrict__ hist, TopkState* state,
                                                                 uint32_t* ticket) {
    __shared__ uint32_t sh[2048];
    __shared__ int s_last;
    const int nb = 1 << pass_bits(pass);
    const int shift = pass_shift(pass);
    TopkState prev;
    if (pass == 0) {
        prev.prefix = 0;
        prev.k_rem = K;
        prev.all = 0;
        prev.total = 0;
    } else {
        prev = state[pass - 1];
    }
    if (prev.all) {  // nothing left to decide
        if (blockIdx.x == 0 && threadIdx.x == 0) state[pass] = prev;
        return;
    }
    const int prev_shift = pass == 0 ? 0 : pass_shift(pass - 1);
    for (int b = threadIdx.x; b < nb; b += kTopkThreads) sh[b] = 0;
    __syncthreads();
    int64_t lo, hi;
    wg_range(N, chunk, lo, hi);
    const int lane = threadIdx.x & 63;
    for (int64_t base = lo; base < hi; base += kBatch) {
        uint32_t v[kVec][4];
        load_batch(prio, base, hi, v);
#pragma unroll
        for (int k = 0; k < kVec; k++) {
#pragma unroll
            for (int q = 0; q < 4; q++) {
                const uint32_t p = v[k][q];
                const bool valid = p != 0u && (pass == 0 || (p >> prev_shift) == prev.prefix);
                const uint32_t bin = (p >> shift) & (uint32_t)(nb - 1);
                const unsigned long long vm = __ballot(valid);
                if (vm == 0) continue;
                const int first = __ffsll((long long)vm) - 1;
                const uint32_t b0 = (uint32_t)__builtin_amdgcn_readlane((int)bin, first);
                if (__ballot(valid && bin == b0) == vm) {
                    if (lane == first) atomicAdd(&sh[b0], (uint32_t)__popcll(vm));
                } else if (valid) {
                    atomicAdd(&sh[bin], 1u);
                }
            }
        }
    }
    __syncthreads();
    for (int b = threadIdx.x; b < nb; b += kTopkThreads)
        if (sh[b] != 0u) atomicAdd(&hist[b], sh[b]);
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) s_last = atomicAdd(ticket, 1u) == gridDim.x - 1;
    __syncthreads();
    if (!s_last) return;

    // The last workgroup: every other workgroup's histogram is in.
    __threadfence();
    for (int b = threadIdx.x; b < nb; b += kTopkThreads)
        sh[b] = __hip_atomic_load(&hist[b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (threadIdx.x < 64) {
        // Lane l covers bins top, top-1, .., top-per+1 (the highest bins in lane 0).
        const int per = nb / 64;
        const int top = nb - 1 - lane * per;
        uint64_t part = 0;
        for (int k = 0; k < per; k++) part += sh[top - k];
        const uint64_t incl = wave_inclusive_scan(part);
        const uint64_t total = read_lane(incl, 63);
        TopkState st = prev;
        if (pass == 0) st.total = (uint32_t)total;
        if (pass == 0 && total < K) {
            st.all = 1;
            if (lane == 0) state[pass] = st;
        } else {
            // The sub-histogram holds at least k_rem entries (the chosen bin of
            // the previous pass did), so some lane reaches k_rem.
            const int L = __ffsll((long long)__ballot(incl >= prev.k_rem)) - 1;
            if (lane == L) {
                uint64_t cum = incl - part;
                int sel = top - per + 1;
                for (int k = 0; k < per; k++) {
                    const int b = top - k;
                    if (cum + sh[b] >= prev.k_rem) {
                        sel = b;
                        break;
                    }
                    cum += sh[b];
                }
                st.prefix = (prev.prefix << pass_bits(pass)) | (uint32_t)sel;
                st.k_rem = prev.k_rem - (uint32_t)cum;
                state[pass] = st;
            }
        }
    }
    __syncthreads();
    for (int b = threadIdx.x; b < nb; b += kTopkThreads) hist[b] = 0u;  // ready for the next call
    if (threadIdx.x == 0) *ticket = 0u;
}

__device__ __forceinline__ void classify(uint32_t p, const TopkState& st, bool& gt, bool& eq) {
    if (st.all) {
        gt = p != 0u;
        eq = false;
    } else {
        gt = p > st.prefix;
        eq = p == st.prefix;
    }
}

__global__ __launch_bounds__(kTopkThreads) void topk_count_kernel(const uint32_t* __restrict__ prio, int64_t N,
                                                                  int64_t chunk, const TopkState* state,
                                                                  uint32_t* __restrict__ counts, int grid) {
    __shared__ uint64_t s_gt[kTopkWaves], s_eq[kTopkWaves];
    const TopkState st = state[2];
    int64_t lo, hi;
    wg_range(N, chunk, lo, hi);
    uint32_t ngt = 0, neq = 0;
    for (int64_t base = lo; base < hi; base += kBatch) {
        uint32_t v[kVec][4];
        load_batch(prio, base, hi, v);
#pragma unroll
        for (int k = 0; k < kVec; k++)
#pragma unroll
            for (int q = 0; q < 4; q++) {
                bool gt, eq;
                classify(v[k][q], st, gt, eq);
                ngt += gt;
                neq += eq;
            }
    }
    const uint64_t wgt = wave_sum(ngt), weq = wave_sum(neq);
    if ((threadIdx.x & 63) == 0) {
        s_gt[threadIdx.x >> 6] = wgt;
        s_eq[threadIdx.x >> 6] = weq;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t a = 0, b = 0;
        for (int k = 0; k < kTopkWaves; k++) {
            a += s_gt[k];
            b += s_eq[k];
        }
        counts[blockIdx.x] = (uint32_t)a;
        counts[grid + blockIdx.x] = (uint32_t)b;
    }
}

// Thread t of a workgroup owns the contiguous run of `run` slots starting
// at lo + t * run (run = chunk / kTopkThreads, a multiple of 4), so slot
// order is thread order and one block-wide scan of per-thread counts gives
// every output position.
__device__ __forceinline__ void count_run(const uint32_t* __restrict__ prio, int64_t r0, int64_t r1,
                                          const TopkState& st, uint32_t& ngt, uint32_t& neq) {
    ngt = 0;
    neq = 0;
    for (int64_t e = r0; e < r1; e += 4) {
        uint32_t v[4];
        if (e + 4 <= r1) {
            const uint4 x = *reinterpret_cast<const uint4*>(prio + e);
            v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
        } else {
#pragma unroll
            for (int q = 0; q < 4; q++) v[q] = e + q < r1 ? prio[e + q] : 0u;
        }
#pragma unroll
        for (int q = 0; q < 4; q++) {
            bool gt, eq;
            classify(v[q], st, gt, eq);
            ngt += gt;
            neq += eq;
        }
    }
}

__global__ __launch_bounds__(kTopkThreads) void topk_compact_kernel(const uint32_t* __restrict__ prio, int64_t N,
                                                                    int64_t chunk, const TopkState* state,
                                                                    const uint32_t* __restrict__ counts, int grid,
                                                                    uint64_t* __restrict__ keys) {
    __shared__ uint64_t s_wgt[kTopkWaves], s_weq[kTopkWaves];
    __shared__ uint64_t s_base[3];  // gt base, eq base, total above P*
    const TopkState st = state[2];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    if (wave == 0) {
        uint64_t gb = 0, eb = 0, tot = 0;
        for (int w = lane; w < grid; w += 64) {
            const uint64_t g = counts[w], e = counts[grid + w];
            tot += g;
            if (w < (int)blockIdx.x) {
                gb += g;
                eb += e;
            }
        }
        gb = wave_sum(gb);
        eb = wave_sum(eb);
        tot = wave_sum(tot);
        if (lane == 0) {
            s_base[0] = gb;
            s_base[1] = eb;
            s_base[2] = tot;
        }
    }
    int64_t lo, hi;
    wg_range(N, chunk, lo, hi);
    const int64_t run = chunk / kTopkThreads;
    int64_t r0 = lo + (int64_t)threadIdx.x * run;
    int64_t r1 = r0 + run;
    if (r0 > hi) r0 = hi;
    if (r1 > hi) r1 = hi;
    uint32_t ngt, neq;
    count_run(prio, r0, r1, st, ngt, neq);
    // Exclusive prefix of the per-thread counts across the workgroup.
    const uint64_t ig = wave_inclusive_scan(ngt), ie = wave_inclusive_scan(neq);
    if (lane == 63) {
        s_wgt[wave] = ig;
        s_weq[wave] = ie;
    }
    __syncthreads();
    uint64_t pg = 0, pe = 0;
    for (int k = 0; k < wave; k++) {
        pg += s_wgt[k];
        pe += s_weq[k];
    }
    uint64_t og = s_base[0] + pg + ig - ngt;  // output position of this thread's first slot above P*
    uint64_t oe = s_base[1] + pe + ie - neq;  // rank of its first tie among all ties, in slot order
    const uint64_t total_gt = s_base[2];
    const uint64_t e_need = st.all ? 0 : st.k_rem;
    if (ngt == 0 && (neq == 0 || oe >= e_need)) return;
    for (int64_t e0 = r0; e0 < r1; e0 += 4 * kVec) {
        // Reload the run kVec x 4 slots at a time, all loads in flight together.
        uint32_t v[kVec][4];
#pragma unroll
        for (int k = 0; k < kVec; k++) {
            const int64_t e = e0 + 4 * k;
            if (e + 4 <= r1) {
                const uint4 x = *reinterpret_cast<const uint4*>(prio + e);
                v[k][0] = x.x; v[k][1] = x.y; v[k][2] = x.z; v[k][3] = x.w;
            } else {
#pragma unroll
                for (int q = 0; q < 4; q++) v[k][q] = e + q < r1 ? prio[e + q] : 0u;
            }
        }
#pragma unroll
        for (int k = 0; k < kVec; k++)
#pragma unroll
            for (int q = 0; q < 4; q++) {
                const int64_t e = e0 + 4 * k + q;
                if (e >= r1) continue;
                const uint32_t p = v[k][q];
                bool gt, eq;
                classify(p, st, gt, eq);
                const uint64_t key = ((uint64_t)p << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)e);
                if (gt) keys[og++] = key;
                if (eq) {
                    if (oe < e_need) keys[total_gt + oe] = key;
                    oe++;
                }
            }
    }
}

__global__ __launch_bounds__(kTopkThreads) void topk_sort_kernel(const uint64_t* __restrict__ keys,
                                                                 const TopkState* state, int32_t K, uint64_t span,
                                                                 uint64_t seed, int64_t* __restrict__ idx,
                                                                 int32_t* __restrict__ start, float* __restrict__ w,
                                                                 uint32_t* status) {
    __shared__ uint64_t sk[kTopkMaxK];
    const TopkState st = state[2];
    const int n = st.all ? (int)st.total : K;  // keys written by the compaction
    int npow = 1;
    while (npow < n) npow <<= 1;
    for (int k = threadIdx.x; k < npow; k += kTopkThreads) sk[k] = k < n ? keys[k] : 0ull;
    __syncthreads();
    // Bitonic sort, descending: a key is (priority << 32) | ~slot, so larger
    // keys are higher priorities and, among equal priorities, lower slots.
    constexpr int kPairs = kTopkMaxK / 2 / kTopkThreads;  // pairs per thread at the largest size
    for (int k = 2; k <= npow; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            // The pairs of one step are disjoint: load them all, then compare,
            // then store, so each step costs one LDS round trip.
            uint64_t x[kPairs], y[kPairs];
            int a[kPairs];
#pragma unroll
            for (int r = 0; r < kPairs; r++) {
                const int t = threadIdx.x + r * kTopkThreads;
                a[r] = -1;
                if (t < (npow >> 1)) {
                    a[r] = ((t & ~(j - 1)) << 1) | (t & (j - 1));
                    x[r] = sk[a[r]];
                    y[r] = sk[a[r] | j];
                }
            }
#pragma unroll
            for (int r = 0; r < kPairs; r++) {
                if (a[r] < 0) continue;
                const bool down = (a[r] & k) == 0;
                if (down ? (x[r] < y[r]) : (x[r] > y[r])) {
                    sk[a[r]] = y[r];
                    sk[a[r] | j] = x[r];
                }
            }
            __syncthreads();
        }
    }
    for (int b = threadIdx.x; b < K; b += kTopkThreads) {
        if (b < n) {
            idx[b] = (int64_t)(0xFFFFFFFFu - (uint32_t)sk[b]);
            start[b] = (int32_t)scale_draw(splitmix64_out(seed, 2 * (uint64_t)b + 1), span);
            if (w) w[b] = 1.0f;
        } else {
            idx[b] = -1;
            start[b] = 0;
            if (w) w[b] = 0.0f;
        }
    }
    if (threadIdx.x == 0 && n < K) atomicOr(status, GEAR_STATUS_NO_WEIGHT);
}

}  // namespace

hipError_t launch_topk(Table& t, int32_t K, int32_t L, uint64_t seed, int64_t* idx, int32_t* start, float* w,
                       hipStream_t s) {
    // chunk: a multiple of 4 * kTopkThreads (aligned loads, whole per-thread runs).
    const int64_t unit = 4 * 1024;
    int64_t g = (t.N + unit - 1) / unit;
    g = g < kTopkMaxGrid ? g : kTopkMaxGrid;
    const int64_t chunk = ((t.N + g - 1) / g + unit - 1) / unit * unit;
    const int grid = (int)((t.N + chunk - 1) / chunk);
    TopkState* state = reinterpret_cast<TopkState*>(t.topk_state);
    for (int pass = 0; pass < 3; pass++) {
        hipLaunchKernelGGL(topk_hist_kernel, dim3(grid), dim3(kTopkThreads), 0, s, t.priority, t.N, chunk, pass,
                           (uint32_t)K, t.topk_hist + pass * 2048, state, t.topk_ticket + pass);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(topk_count_kernel, dim3(grid), dim3(kTopkThreads), 0, s, t.priority, t.N, chunk, state,
                       t.topk_counts, grid);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(topk_compact_kernel, dim3(grid), dim3(kTopkThreads), 0, s, t.priority, t.N, chunk, state,
                       t.topk_counts, grid, t.topk_keys);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(topk_sort_kernel, dim3(1), dim3(kTopkThreads), 0, s, t.topk_keys, state, K,
                       (uint64_t)(t.T - L + 1), seed, idx, start, w, t.status);
    return hipGetLastError();
}

}  // namespace gear
