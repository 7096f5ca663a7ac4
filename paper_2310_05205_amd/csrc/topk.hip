// TopK selection on gfx950 (GEAR Sec. 3.3, decentralized selection: TopK
// is deterministic; each GPU computes its top-K priority trajectories).
//
// The K highest priorities among slots with non-zero priority, higher
// priority first, the lower slot first among equal priorities.
//
// The K-th largest priority is found by a radix select over a 36-bit key
// that orders priorities like the priorities themselves: the position e of
// the leading one (5 bits) above the e bits below it, left-aligned in 31
// bits.  Its three 12-bit digits give small priorities their own pass-0
// bins (every value below 256 is one bin) and spread skewed distributions
// over many bins.  Selection stops early once the chosen bin is a single
// value or is taken whole.  No workgroup waits for another and no kernel
// fences memory: workgroup 0 of each kernel stores the selection state it
// derived, and the next kernel (after the kernel boundary that makes it and
// the previous pass's complete histogram visible) derives at most one more
// digit from that histogram.
//
//   topk_hist_kernel    (x3) a workgroup histograms one digit of the keys
//                       whose higher digits match the ones chosen so far,
//                       in eight LDS copies of the histogram (a thread adds
//                       into copy thread mod 8), sums the copies, adds its
//                       bins into the pass's global histogram and stores the
//                       suffix sums of its own histogram.
//   topk_compact_kernel finishes the threshold and turns it into a range of
//                       priorities, so a key is classified with two integer
//                       compares; the stored suffix sums give every
//                       workgroup's count above and at it, hence this
//                       workgroup's output offsets; one scan per batch of
//                       loads orders its keys by slot.  It writes
//                       (p << 32 | ~slot) of every slot above the threshold
//                       and of the lowest-slot ones at it.
//   topk_rank_emit_kernel  a key's place in descending order is the number
//                       of larger keys (keys hold the slot, so they are
//                       unique); every workgroup stages all K keys in LDS
//                       and ranks 32 of them, 32 lanes per key, then writes
//                       slot, window start and weight at each key's place
//                       and clears the histograms for the next call.
//
// Loads that a derivation waits for are issued before the bulk priority
// loads: vector loads complete in issue order, so the reverse would make the
// derivation wait for the whole batch.
#include "gear_internal.h"
#include "wave.h"

namespace gear {
namespace {

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / 64;
constexpr int kBins = kTopkBins;
constexpr int kDigit = 12;
constexpr int kKeyBits = 36;
constexpr int kPasses = kKeyBits / kDigit;
// LDS copies of a digit histogram.  With skewed priorities most lanes of a
// wave add into the same few bins, and LDS serialises atomics of one
// instruction that hit one address; spreading the lanes over eight copies
// (rows 4 words longer than a histogram, so a bin's copies sit in
// different banks) cuts those conflicts eightfold: 131 KB of LDS.
constexpr int kLdsCopies = 8;
constexpr int kLdsStride = kBins + 4;

constexpr uint32_t kAll = 1u;           // fewer than K candidates: take every one
constexpr uint32_t kDone = 2u;          // the threshold is fully determined
constexpr uint32_t kInconsistent = 4u;  // histograms disagree (priorities changed mid-selection)

struct TopkState {
    uint64_t prefix;  // key digits chosen so far
    uint32_t k_rem;   // of the keys whose digits match `prefix`, how many are taken (lowest slots first)
    uint32_t total;   // number of slots with non-zero priority
    int32_t passes;   // digits chosen; keys are compared after >> (36 - 12 * passes)
    uint32_t flags;
};
static_assert(sizeof(TopkState) * (kPasses + 1) <= kTopkStateWords * sizeof(uint32_t), "state buffer");

// Order-preserving 36-bit key of a non-zero priority (0 maps to 0 like 1;
// validity is tested separately).
__device__ __forceinline__ uint64_t order_key(uint32_t p) {
    const int e = 31 - __clz(p | 1u);
    const uint32_t mant = (p << (31 - e)) & 0x7FFFFFFFu;
    return ((uint64_t)e << 31) | mant;
}

__device__ __forceinline__ int state_shift(const TopkState& st) { return kKeyBits - kDigit * st.passes; }
__device__ __forceinline__ bool decided(const TopkState& st) { return (st.flags & (kAll | kDone)) != 0; }

// Slots [blockIdx.x * chunk, ...) of this workgroup; chunk is a multiple of
// 4 * kTopkThreads, so every 16-byte load is aligned.
__device__ __forceinline__ void wg_range(int64_t N, int64_t chunk, int64_t& lo, int64_t& hi) {
    lo = (int64_t)blockIdx.x * chunk;
    hi = lo + chunk < N ? lo + chunk : N;
}

// One batch: kVec 16-byte loads per thread, all issued before any is used;
// thread t, load k covers slots base + (k * kTopkThreads + t) * 4 .. +3,
// so (k, t, element) order is slot order.  Slots at or past `hi` read as
// priority 0 (never a candidate).
constexpr int kVec = 4;
constexpr int64_t kBatch = (int64_t)kVec * kTopkThreads * 4;

__device__ __forceinline__ void load_batch(const uint32_t* __restrict__ prio, int64_t base, int64_t hi,
                                           uint32_t v[kVec][4]) {
    if (base + kBatch <= hi) {
        // The whole batch is in range (every batch but a ragged last one):
        // a branch the workgroup takes as one, so the loads are issued
        // back to back, none waiting for another.
#pragma unroll
        for (int k = 0; k < kVec; k++) {
            const uint4 x = *reinterpret_cast<const uint4*>(prio + base + ((int64_t)k * kTopkThreads + threadIdx.x) * 4);
            v[k][0] = x.x; v[k][1] = x.y; v[k][2] = x.z; v[k][3] = x.w;
        }
        return;
    }
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

// Thread t's four bins of a histogram row, kBins-4-4t .. kBins-1-4t (so
// thread order is descending bin order; .w is the highest).
__device__ __forceinline__ int first_bin() { return kBins - 4 - 4 * (int)threadIdx.x; }

// This thread's four bins of digit pass q's global histogram.
__device__ __forceinline__ uint4 load_row(const uint32_t* __restrict__ hist, int q) {
    return *reinterpret_cast<const uint4*>(hist + q * kBins + first_bin());
}

struct DeriveShared {
    TopkState state[kPasses];
    uint64_t wave_total[kPasses][kTopkWaves];
};

// Block-wide choice of digit pass q from its global histogram.
__device__ TopkState derive_pass(uint4 h, int q, const TopkState& prev, uint32_t K, DeriveShared& sh) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint64_t part = (uint64_t)h.x + h.y + h.z + h.w;
    const uint64_t incl = wave_inclusive_scan(part);
    if (lane == 63) sh.wave_total[q][wave] = incl;
    if (threadIdx.x == 0) {
        TopkState f = prev;  // kept only if no bin holds the k_rem-th key
        f.flags |= kDone | kInconsistent;
        sh.state[q] = f;
    }
    __syncthreads();
    uint64_t before = 0, total = 0;
    for (int w = 0; w < kTopkWaves; w++) {
        const uint64_t x = sh.wave_total[q][w];
        before += w < wave ? x : 0;
        total += x;
    }
    before += incl - part;
    if (q == 0 && total < K) {
        if (threadIdx.x == 0) {
            TopkState st = prev;
            st.total = (uint32_t)total;
            st.flags = kAll;
            sh.state[q] = st;
        }
    } else if (before < prev.k_rem && prev.k_rem <= before + part) {
        const uint32_t bins[4] = {h.w, h.z, h.y, h.x};
        const int top = first_bin() + 3;
        uint64_t cum = before;
        int j = 0;
        while (j < 3 && cum + bins[j] < prev.k_rem) cum += bins[j++];
        TopkState st = prev;
        if (q == 0) st.total = (uint32_t)total;
        st.prefix = (prev.prefix << kDigit) | (uint64_t)(top - j);
        st.k_rem = prev.k_rem - (uint32_t)cum;
        st.passes = q + 1;
        const int mant_bits = kDigit * (q + 1) - 5;  // mantissa bits the prefix fixes
        const int e = (int)(st.prefix >> mant_bits);
        if (q + 1 == kPasses || bins[j] == st.k_rem || e <= mant_bits) st.flags |= kDone;
        sh.state[q] = st;
    }
    __syncthreads();
    return sh.state[q];
}

__device__ __forceinline__ TopkState initial_state(uint32_t K) {
    TopkState st;
    st.prefix = 0;
    st.k_rem = K;
    st.total = 0;
    st.passes = 0;
    st.flags = 0;
    return st;
}

// The state after digit passes 0 .. q-1 (q >= 1): the state after passes
// 0 .. q-2 that the previous kernel stored in states[q - 1] (the initial
// state when q = 1), advanced by pass q - 1 unless it was already decided.
// `row` is this thread's part of pass q - 1's histogram, loaded together with
// the stored state.  Every thread of the block must call this.
__device__ TopkState state_after(int q, const TopkState& stored, uint4 row, uint32_t K, DeriveShared& sh) {
    const TopkState s = q >= 2 ? stored : initial_state(K);
    return decided(s) ? s : derive_pass(row, q - 1, s, K, sh);
}

__global__ __launch_bounds__(kTopkThreads) void topk_hist_kernel(const uint32_t* __restrict__ prio, int64_t N,
                                                                 int64_t chunk, int pass, uint32_t K,
                                                                 uint32_t* __restrict__ hist,
                                                                 uint32_t* __restrict__ local,
                                                                 TopkState* __restrict__ states) {
    __shared__ __align__(16) uint32_t sh[kLdsCopies * kLdsStride];
    __shared__ DeriveShared dsh;
    __shared__ uint64_t s_wt[kTopkWaves];
    TopkState prev = initial_state(K);
    if (pass > 0) {
        const uint4 row = load_row(hist, pass - 1);
        const TopkState stored = states[pass - 1];
        prev = state_after(pass, stored, row, K, dsh);
        if (blockIdx.x == 0 && threadIdx.x == 0) states[pass] = prev;  // for the next kernel
    }
    if (decided(prev)) return;  // nothing left to histogram
    const int prev_shift = kKeyBits - kDigit * pass;
    const int shift = prev_shift - kDigit;
    int64_t lo, hi;
    wg_range(N, chunk, lo, hi);
    uint32_t v[kVec][4];
    load_batch(prio, lo, hi, v);
    for (int b = threadIdx.x * 4; b < kLdsCopies * kLdsStride; b += kTopkThreads * 4)
        *reinterpret_cast<uint4*>(&sh[b]) = make_uint4(0u, 0u, 0u, 0u);
    uint32_t* const copy = sh + (threadIdx.x % kLdsCopies) * kLdsStride;
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    // Pass 0 counts every non-zero priority; its digit is the leading-one
    // position and the 7 bits below it, computed in 32 bits.  A zero
    // priority adds into one of the row's unused padding words instead, so
    // the loop has no branch.
    const uint32_t pad = (uint32_t)kBins + ((threadIdx.x >> 3) & 3u);
    for (int64_t base = lo; base < hi; base += kBatch) {
        if (base != lo) load_batch(prio, base, hi, v);
        if (pass == 0) {
#pragma unroll
            for (int k = 0; k < kVec; k++) {
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    const uint32_t p = v[k][q];
                    const uint32_t z = __clz(p | 1u);                    // 31 - leading-one position
                    const uint32_t d = ((31u - z) << 7) | ((p << z) >> 24 & 0x7Fu);
                    atomicAdd(&copy[p != 0u ? d : pad], 1u);
                }
            }
        } else {
#pragma unroll
            for (int k = 0; k < kVec; k++) {
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    const uint32_t p = v[k][q];
                    const uint64_t key = order_key(p);
                    const bool counted = p != 0u && (key >> prev_shift) == prev.prefix;
                    const uint32_t bin = (uint32_t)(key >> shift) & (uint32_t)(kBins - 1);
                    if (counted) atomicAdd(&copy[bin], 1u);
                }
            }
        }
    }
    __syncthreads();
    // Add into the global histogram; store this workgroup's suffix sums
    // (S[b] = its keys in bins >= b) for the offsets of the compaction.
    const int b0 = first_bin();
    uint4 h = make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
    for (int c = 0; c < kLdsCopies; c++) {
        const uint4 x = *reinterpret_cast<const uint4*>(&sh[c * kLdsStride + b0]);
        h.x += x.x;
        h.y += x.y;
        h.z += x.z;
        h.w += x.w;
    }
    uint32_t* out = hist + pass * kBins + b0;
    if (h.x) atomicAdd(out + 0, h.x);
    if (h.y) atomicAdd(out + 1, h.y);
    if (h.z) atomicAdd(out + 2, h.z);
    if (h.w) atomicAdd(out + 3, h.w);
    const uint64_t part = (uint64_t)h.x + h.y + h.z + h.w;
    const uint64_t incl = wave_inclusive_scan(part);
    if (lane == 63) s_wt[wave] = incl;
    __syncthreads();
    uint64_t above = incl - part;
    for (int w = 0; w < wave; w++) above += s_wt[w];
    uint4 S;
    S.w = (uint32_t)(above + h.w);
    S.z = S.w + h.z;
    S.y = S.z + h.y;
    S.x = S.y + h.x;
    *reinterpret_cast<uint4*>(local + ((size_t)pass * kTopkMaxGrid + blockIdx.x) * kBins + b0) = S;
}

// The smallest priority p >= 1 whose order key is at least X, or 2^32 if
// there is none.  Keys of the priorities with leading one at bit e are
// (e << 31) | (r << (31 - e)) for p = 2^e + r, increasing in r.
__device__ __forceinline__ uint64_t first_priority_with_key(uint64_t X) {
    const uint64_t e = X >> 31;
    if (e > 31) return 1ull << 32;
    const uint64_t m = X & 0x7FFFFFFFull;
    const int sh = 31 - (int)e;
    const uint64_t r = (m + (1ull << sh) - 1) >> sh;
    if (r < (1ull << e)) return (1ull << e) + r;
    return 2ull << e;  // the first priority of the next leading-one position (2^32: none)
}

// A decided state as a priority range: keys at the threshold are the
// priorities in [lo, hi), keys above it those from hi on (the order key is
// increasing in the priority).  Taking every candidate is lo = hi = 1.
__device__ __forceinline__ void threshold_range(const TopkState& st, uint64_t& lo, uint64_t& hi) {
    if (st.flags & kAll) {
        lo = hi = 1;
        return;
    }
    const int shift = state_shift(st);
    lo = first_priority_with_key(st.prefix << shift);
    hi = first_priority_with_key((st.prefix + 1) << shift);
}

// Keys above and at the threshold of workgroups g = lane + 64 r (r < kCountRounds),
// from their suffix sums of every pass that ran.  Every count is loaded
// before any is used (one memory round trip): rows of passes that did not
// run, and of workgroups past the grid, are read from valid addresses and
// then ignored.
constexpr int kCountRounds = kTopkMaxGrid / 64;
static_assert(kPasses == 3, "the loads below are listed per pass");

__device__ __forceinline__ void wg_counts(const uint32_t* __restrict__ local, const TopkState& st, int lane, int grid,
                                          uint32_t gt[kCountRounds], uint32_t eq[kCountRounds]) {
    int sel[kPasses];
#pragma unroll
    for (int q = 0; q < kPasses; q++)
        sel[q] = q < st.passes ? (int)(st.prefix >> (kDigit * (st.passes - 1 - q))) & (kBins - 1) : 0;
    uint32_t above[kCountRounds][kPasses], at[kCountRounds][kPasses], all[kCountRounds];
#pragma unroll
    for (int r = 0; r < kCountRounds; r++) {
        const int g = lane + 64 * r < grid ? lane + 64 * r : grid - 1;
        all[r] = local[(size_t)g * kBins];  // pass 0, bin 0: every non-zero priority of the workgroup
#pragma unroll
        for (int q = 0; q < kPasses; q++) {
            const uint32_t* row = local + ((size_t)q * kTopkMaxGrid + g) * kBins;
            above[r][q] = row[sel[q] + 1 < kBins ? sel[q] + 1 : sel[q]];
            at[r][q] = row[sel[q]];
        }
    }
    // Keeps the compiler from moving loads into the branches below.
#pragma unroll
    for (int r = 0; r < kCountRounds; r++)
        asm volatile("" ::"v"(all[r]), "v"(above[r][0]), "v"(above[r][1]), "v"(above[r][2]), "v"(at[r][0]),
                     "v"(at[r][1]), "v"(at[r][2]));
#pragma unroll
    for (int r = 0; r < kCountRounds; r++) {
        gt[r] = 0;
        eq[r] = 0;
        if (lane + 64 * r >= grid) continue;
        if (st.flags & kAll) {
            gt[r] = all[r];
            continue;
        }
#pragma unroll
        for (int q = 0; q < kPasses; q++) {
            if (q >= st.passes) break;
            const uint32_t a = sel[q] + 1 < kBins ? above[r][q] : 0u;
            gt[r] += a;
            if (q == st.passes - 1) eq[r] = at[r][q] - a;
        }
    }
}

__global__ __launch_bounds__(kTopkThreads) void topk_compact_kernel(const uint32_t* __restrict__ prio, int64_t N,
                                                                    int64_t chunk, uint32_t K,
                                                                    const uint32_t* __restrict__ hist,
                                                                    const uint32_t* __restrict__ local, int grid,
                                                                    TopkState* __restrict__ states,
                                                                    uint64_t* __restrict__ keys) {
    __shared__ DeriveShared dsh;
    __shared__ uint32_t s_pre[kVec * kTopkWaves];  // per (load, wave): packed counts, then their prefix
    __shared__ uint64_t s_base[5];                 // above base, at base, total above, own above, own at
    __shared__ uint32_t s_batch;                   // packed counts of the whole batch
    const uint4 row = load_row(hist, kPasses - 1);
    const TopkState stored = states[kPasses - 1];
    int64_t lo, hi;
    wg_range(N, chunk, lo, hi);
    uint32_t v[kVec][4];
    load_batch(prio, lo, hi, v);
    const TopkState st = state_after(kPasses, stored, row, K, dsh);
    if (blockIdx.x == 0 && threadIdx.x == 0) states[kPasses] = st;  // the final state, for the ranking
    uint64_t p_lo, p_hi;
    threshold_range(st, p_lo, p_hi);
    const uint64_t p_width = p_hi - p_lo;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    if (wave == 0) {
        uint64_t gb = 0, eb = 0, tot = 0;
        uint32_t gt[kCountRounds], eq[kCountRounds];
        wg_counts(local, st, lane, grid, gt, eq);
#pragma unroll
        for (int r = 0; r < kCountRounds; r++) {
            const int g = lane + 64 * r;
            tot += gt[r];
            if (g < (int)blockIdx.x) {
                gb += gt[r];
                eb += eq[r];
            }
            if (g == (int)blockIdx.x) {
                s_base[3] = gt[r];
                s_base[4] = eq[r];
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
    __syncthreads();
    const uint64_t e_need = (st.flags & kAll) ? 0 : st.k_rem;
    const uint64_t total_gt = s_base[2];
    uint64_t run_gt = s_base[0], run_eq = s_base[1];
    if (s_base[3] == 0 && (s_base[4] == 0 || run_eq >= e_need)) return;
    for (int64_t base = lo; base < hi; base += kBatch) {
        if (base != lo) load_batch(prio, base, hi, v);
        // Counts packed as above | at << 16: a batch holds at most kBatch keys.
        uint32_t c[kVec], incl[kVec];
        uint32_t cls[kVec];  // per element: bit q above, bit 4 + q at
#pragma unroll
        for (int k = 0; k < kVec; k++) {
            c[k] = 0;
            cls[k] = 0;
#pragma unroll
            for (int q = 0; q < 4; q++) {
                const uint64_t p = v[k][q];
                const bool gt = p >= p_hi;
                const bool eq = p - p_lo < p_width;
                c[k] += (uint32_t)gt | ((uint32_t)eq << 16);
                cls[k] |= (gt ? 1u << q : 0u) | (eq ? 16u << q : 0u);
            }
            incl[k] = wave_inclusive_scan32(c[k]);
            if (lane == 63) s_pre[k * kTopkWaves + wave] = incl[k];
        }
        __syncthreads();
        if (wave == 0) {
            // Exclusive scan of the kVec x kTopkWaves wave counts in (load, wave) order.
            const uint32_t a = s_pre[lane];
            const uint32_t s = wave_inclusive_scan32(a);
            s_pre[lane] = s - a;
            if (lane == 63) s_batch = s;
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < kVec; k++) {
            if (cls[k] == 0) continue;
            const uint32_t off = s_pre[k * kTopkWaves + wave] + incl[k] - c[k];
            uint64_t og = run_gt + (off & 0xFFFFu);  // output position of this lane's first key above
            uint64_t oe = run_eq + (off >> 16);      // slot-order rank of its first key at the threshold
            const int64_t e0 = base + ((int64_t)k * kTopkThreads + threadIdx.x) * 4;
#pragma unroll
            for (int q = 0; q < 4; q++) {
                const uint64_t key = ((uint64_t)v[k][q] << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)(e0 + q));
                // The counts bound both positions by K; the checks keep a
                // priority changed under a running selection from writing
                // past the key buffer.
                if (cls[k] & (1u << q)) {
                    if (og < (uint64_t)K) keys[og] = key;
                    og++;
                }
                if (cls[k] & (16u << q)) {
                    if (oe < e_need && total_gt + oe < (uint64_t)K) keys[total_gt + oe] = key;
                    oe++;
                }
            }
        }
        const uint32_t tb = s_batch;
        run_gt += tb & 0xFFFFu;
        run_eq += tb >> 16;
        __syncthreads();  // s_pre and s_batch are rewritten by the next batch
    }
}
static_assert(kVec * kTopkWaves == 64, "one lane of wave 0 per (load, wave) count");
static_assert(kBatch < 65536, "a batch's counts fit the 16-bit fields");

// Number of selected keys: K, or every candidate when there are fewer.
__device__ __forceinline__ int selected(const TopkState& st, int32_t K) {
    return (st.flags & kAll) ? (int)st.total : K;
}

// Rank and emit in one launch.  Keys are unique (they hold the slot), so a
// key's place in descending order is the number of larger keys.  The
// compaction wrote the n_gt keys above the threshold first, then those at
// it, each group in slot order.  When every key at the threshold has the
// same priority (the usual case: a threshold fixed to one value), a key at
// it is preceded by all keys above and by the keys at it with lower slots,
// so its place is its position in the list, and a key above the threshold
// only needs comparing with the n_gt keys above it.  Otherwise every key is
// compared with all n selected keys.
//
// Every workgroup stages the keys to compare with in LDS (positions past
// them read as 0, below every key, since p >= 1) and ranks kEmitKeys keys,
// kEmitLanes lanes per key each counting the larger keys among every
// kEmitLanes-th pair of the staged list.  The lanes of one key read
// consecutive pairs and the two keys of a wave read the same pairs, so every
// LDS read is a conflict-free broadcast.  The counts are summed within each
// 32-lane half of a wave, and the half's last lane writes slot, window start
// and weight at its key's place.  Workgroups also clear the digit histograms
// for the next call.
constexpr int kEmitThreads = 1024;
constexpr int kEmitLanes = 32;
constexpr int kEmitKeys = kEmitThreads / kEmitLanes;
constexpr int kEmitPad = 2 * kEmitLanes;  // staged keys per compare round (one pair per lane)
static_assert(kTopkMaxK % kEmitPad == 0, "a padded key count never passes the key buffer");
constexpr int kEmitLoads = kTopkMaxK / 2 / kEmitThreads;  // 16-byte loads per thread for the largest K

__device__ __forceinline__ ulonglong2 keep_below(ulonglong2 v, int e, int lim) {
    return make_ulonglong2(2 * e < lim ? v.x : 0ull, 2 * e + 1 < lim ? v.y : 0ull);
}

__global__ __launch_bounds__(kEmitThreads) void topk_rank_emit_kernel(const uint64_t* __restrict__ keys,
                                                                      const TopkState* __restrict__ state, int32_t K,
                                                                      uint64_t span, uint64_t seed,
                                                                      int64_t* __restrict__ idx,
                                                                      int32_t* __restrict__ start,
                                                                      float* __restrict__ w, uint32_t* status,
                                                                      uint32_t* __restrict__ hist) {
    __shared__ ulonglong2 staged[kTopkMaxK / 2];
    const int tid = (int)threadIdx.x;
    const int pairs = (K + kEmitPad - 1) / kEmitPad * (kEmitPad / 2);  // within the kTopkMaxK-entry buffer
    // The state, this thread's key and the first kEmitThreads pairs of the
    // list are loaded together (one memory round trip), from indices
    // clamped into the padded list.
    const ulonglong2* kp = reinterpret_cast<const ulonglong2*>(keys);
    const ulonglong2 v0 = kp[tid < pairs ? tid : pairs - 1];
    const int i = blockIdx.x * kEmitKeys + tid / kEmitLanes;
    const uint64_t km = keys[i < K ? i : K - 1];
    const TopkState st = *state;
    const int n = selected(st, K);
    uint64_t p_lo, p_hi;
    threshold_range(st, p_lo, p_hi);
    const bool all = (st.flags & kAll) != 0;
    int n_gt = all ? n : K - (int)st.k_rem;  // keys above the threshold, at the front of the list
    n_gt = n_gt < 0 ? 0 : (n_gt < n ? n_gt : n);
    const bool one = !all && p_hi - p_lo == 1;  // every key at the threshold has priority p_lo
    const int lim = one ? n_gt : n;             // keys that some ranked key is compared with
    const int pl = (lim + kEmitPad - 1) / kEmitPad * (kEmitPad / 2);  // staged pairs, <= pairs
    if (tid < pl) staged[tid] = keep_below(v0, tid, lim);
    if (pl > kEmitThreads) {  // the same branch for the whole workgroup
        ulonglong2 v[kEmitLoads - 1];
#pragma unroll
        for (int k = 1; k < kEmitLoads; k++) {
            const int e = k * kEmitThreads + tid;
            v[k - 1] = kp[e < pl ? e : pl - 1];
        }
#pragma unroll
        for (int k = 1; k < kEmitLoads; k++) {
            const int e = k * kEmitThreads + tid;
            if (e < pl) staged[e] = keep_below(v[k - 1], e, lim);
        }
    }
    for (int h = blockIdx.x * kEmitThreads + tid; h < kPasses * kBins; h += gridDim.x * kEmitThreads)
        hist[h] = 0u;  // every digit pass of this call is done
    if (blockIdx.x == 0 && tid == 0 && (st.flags & kInconsistent)) atomicOr(status, GEAR_STATUS_INTERNAL);
    __syncthreads();
    const int lane = tid & (kEmitLanes - 1);
    const bool by_position = one && i >= n_gt;        // a key at a one-value threshold
    const uint64_t mine = i < lim ? km : ~0ull;       // ~0: larger than every key, counts nothing
    uint32_t c = 0;
#pragma unroll 8
    for (int q = lane; q < pl; q += kEmitLanes) {
        const ulonglong2 y = staged[q];
        c += (uint32_t)(y.x > mine) + (uint32_t)(y.y > mine);
    }
    // Sum over the 32 lanes of this key: row scans, then row 0's total into
    // row 1 and row 2's into row 3, so lanes 31 and 63 hold the two keys' sums.
    c += dpp32<0x111, 0xf>(c);
    c += dpp32<0x112, 0xf>(c);
    c += dpp32<0x114, 0xf>(c);
    c += dpp32<0x118, 0xf>(c);
    c += dpp32<0x142, 0xa>(c);
    if (lane != kEmitLanes - 1 || i >= K) return;
    if (i < n) {
        const uint32_t b = by_position ? (uint32_t)i : c;
        if (b >= (uint32_t)n) {  // a key list changed under a running selection
            atomicOr(status, GEAR_STATUS_INTERNAL);
            return;
        }
        idx[b] = (int64_t)(0xFFFFFFFFu - (uint32_t)km);
        start[b] = (int32_t)scale_draw(splitmix64_out(seed, 2 * (uint64_t)b + 1), span);
        if (w) w[b] = 1.0f;
    } else {
        idx[i] = -1;
        start[i] = 0;
        if (w) w[i] = 0.0f;
        if (i == n) atomicOr(status, GEAR_STATUS_NO_WEIGHT);
    }
}
static_assert(kEmitLanes == 32 && kEmitThreads % 64 == 0, "the count sum covers the two halves of a wave");

}  // namespace

hipError_t launch_topk(Table& t, int32_t K, int32_t L, uint64_t seed, int64_t* idx, int32_t* start, float* w,
                       hipStream_t s) {
    // chunk: a multiple of 4 * kTopkThreads (aligned 16-byte loads).
    const int64_t unit = 4 * kTopkThreads;
    int64_t g = (t.N + unit - 1) / unit;
    g = g < kTopkMaxGrid ? g : kTopkMaxGrid;
    const int64_t chunk = ((t.N + g - 1) / g + unit - 1) / unit * unit;
    const int grid = (int)((t.N + chunk - 1) / chunk);
    // states[q]: the state after digit passes 0 .. q-1, stored by kernel q
    // (digit pass q, or the compaction for q = kPasses) for the kernels after it.
    TopkState* states = reinterpret_cast<TopkState*>(t.topk_state);
    TopkState* state = states + kPasses;
    hipError_t e;
    for (int pass = 0; pass < kPasses; pass++) {
        hipLaunchKernelGGL(topk_hist_kernel, dim3(grid), dim3(kTopkThreads), 0, s, t.priority, t.N, chunk, pass,
                           (uint32_t)K, t.topk_hist, t.topk_local, states);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    hipLaunchKernelGGL(topk_compact_kernel, dim3(grid), dim3(kTopkThreads), 0, s, t.priority, t.N, chunk,
                       (uint32_t)K, t.topk_hist, t.topk_local, grid, states, t.topk_keys);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(topk_rank_emit_kernel, dim3((K + kEmitKeys - 1) / kEmitKeys), dim3(kEmitThreads), 0, s,
                       t.topk_keys, state, K, (uint64_t)(t.T - L + 1), seed, idx, start, w, t.status, t.topk_hist);
    return hipGetLastError();
}

}  // namespace gear
