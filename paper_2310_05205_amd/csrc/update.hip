// Priority update on gfx950 (GEAR Sec. 3.2: the status table holds the
// priorities, and changes to it are gathered and then applied).
//
// The batch is applied as if in order, so for a slot that appears several
// times the last occurrence's value wins.
//
// Batches of up to 8192 run in one launch of 32 workgroups.  Workgroup g
// owns the slots whose hash falls in partition g: it reads the whole batch,
// inserts each of its draws' slots into an open-addressing hash table in LDS
// and raises that entry's tag to b+1 (LDS atomic max); after a barrier the
// draw whose b+1 equals its entry's tag is the last occurrence of its slot
// and writes the new priority.  Every occurrence of a slot lands in the
// same workgroup, so no other synchronisation is needed.
//
// Larger batches use two kernels over a table-owned tag array:
//   tag    every draw b raises tag[slot] to b+1 (atomic max), so after the
//          kernel tag[slot] names the last occurrence of that slot;
//   apply  the draw whose b+1 equals tag[slot] writes the new priority and
//          puts the tag back to zero.  Other draws of the same slot see
//          either the winner's tag or zero, never their own, so they never
//          write.  Tags are zero again when the kernel ends.
//
// When the table keeps its selection sum tree up to date across updates,
// each writing draw also adds new - old (mod 2^64) into its tile's sum and
// into the covering node of every upper level.  Exactly one draw writes each
// changed slot, so the tree stays equal to the sums of the priorities.  In
// the one-launch path the upper-level additions of a workgroup are first
// combined per node in LDS (levels of at most 1024 nodes), so each node sees
// at most one global atomic per workgroup.
#include "gear_internal.h"

namespace gear {
namespace {

constexpr int kHashThreads = 1024;
constexpr int kHashMaxBatch = 8192;                 // load factor <= 1/2
constexpr int kHashBits = 14;
constexpr int kHashSize = 1 << kHashBits;           // 2 x 64 KiB of LDS
constexpr int kPerThread = kHashMaxBatch / kHashThreads;
constexpr uint32_t kEmpty = 0xFFFFFFFFu;            // never a slot: slots are < 2^30
constexpr int kPartBits = 5;
constexpr int kParts = 1 << kPartBits;              // workgroups of the one-launch path
constexpr int kAggLevels = 2;                       // upper levels combined in LDS
constexpr int kAggNodes = 1024;                     // ... when they have at most this many nodes

struct Tree {
    uint64_t* tile_sums;             // level 0
    uint64_t* upper[kMaxLevels];     // levels 1 .. nlevels-1 (the copy the last scan filled)
    int64_t size[kMaxLevels];
    int nlevels;
    int maintain;                    // 0: leave the tree alone
};

// Level l >= 1 node covering `slot`: a level-l node covers 256^l tiles of 256.
__device__ inline int64_t node_of(int64_t slot, int l) { return slot >> (8 * (l + 1)); }

__device__ inline void add_u64(uint64_t* p, uint64_t d) {
    atomicAdd(reinterpret_cast<unsigned long long*>(p), (unsigned long long)d);
}

// `live`: indices at or past it are invalid.  `committed` (managed tables
// only, else NULL): an index whose flag is 0 is released or still being
// written; its update is dropped, so it never becomes selectable.
__global__ __launch_bounds__(kHashThreads) void scatter_lds_kernel(const int64_t* __restrict__ idx,
                                                                   const uint32_t* __restrict__ newp, int32_t B,
                                                                   int64_t live, const uint8_t* __restrict__ committed,
                                                                   uint32_t* __restrict__ prio,
                                                                   uint32_t* status, Tree tree) {
    __shared__ uint32_t key[kHashSize];
    __shared__ uint32_t tag[kHashSize];
    __shared__ uint64_t agg[kAggLevels][kAggNodes];
    for (int h = threadIdx.x; h < kHashSize; h += kHashThreads) {
        key[h] = kEmpty;
        tag[h] = 0u;
    }
    for (int h = threadIdx.x; h < kAggLevels * kAggNodes; h += kHashThreads) agg[h / kAggNodes][h % kAggNodes] = 0;
    int64_t slot[kPerThread];
    uint32_t val[kPerThread];
#pragma unroll
    for (int k = 0; k < kPerThread; k++) {
        const int b = threadIdx.x + k * kHashThreads;
        slot[k] = b < B ? idx[b] : -1;
        val[k] = b < B ? newp[b] : 0u;
    }
    // Draws of this workgroup's partition.  Their committed flags and old
    // priorities are read now, overlapping the hash phase, all issued
    // before any is used.  Draws of other partitions and invalid ones read
    // slot 0 instead, the same word for every such lane, and ignore it:
    // each workgroup then fetches only its own ~B/32 scattered words, not
    // all B (reading every draw's old priority in all 32 workgroups made an
    // update that keeps the tree 15.7 instead of 9.7 us).  Only the winning
    // draw of a slot writes it, and only after the barrier below.
    bool mine[kPerThread];
    bool part[kPerThread];
    uint32_t old[kPerThread];
    uint32_t flag[kPerThread];
    bool bad = false;
#pragma unroll
    for (int k = 0; k < kPerThread; k++) {
        const int b = threadIdx.x + k * kHashThreads;
        const bool valid = b < B && slot[k] >= 0 && slot[k] < live;
        part[k] = valid && (((uint32_t)slot[k] * 0x85EBCA6Bu) >> (32 - kPartBits)) == blockIdx.x;
        const int64_t s = part[k] ? slot[k] : 0;
        flag[k] = committed != nullptr ? committed[s] : 1u;
        old[k] = tree.maintain ? prio[s] : 0u;
    }
    static_assert(kPerThread == 8, "the values below are listed per draw");
    // Keeps the compiler from waiting on each load before issuing the next.
    asm volatile("" ::"v"(flag[0]), "v"(flag[1]), "v"(flag[2]), "v"(flag[3]), "v"(flag[4]), "v"(flag[5]),
                 "v"(flag[6]), "v"(flag[7]), "v"(old[0]), "v"(old[1]), "v"(old[2]), "v"(old[3]), "v"(old[4]),
                 "v"(old[5]), "v"(old[6]), "v"(old[7]));
#pragma unroll
    for (int k = 0; k < kPerThread; k++) {
        const int b = threadIdx.x + k * kHashThreads;
        const bool valid = b < B && slot[k] >= 0 && slot[k] < live;
        if (b < B && !valid && blockIdx.x == 0) bad = true;
        mine[k] = part[k] && flag[k] != 0;
        if (!mine[k]) old[k] = 0u;
    }
    __syncthreads();
    int pos[kPerThread];
#pragma unroll
    for (int k = 0; k < kPerThread; k++) {
        const int b = threadIdx.x + k * kHashThreads;
        pos[k] = -1;
        if (!mine[k]) continue;
        const uint32_t kk = (uint32_t)slot[k];
        uint32_t h = (kk * 2654435761u) >> (32 - kHashBits);
        while (true) {  // at most B < kHashSize occupied entries, so a free or equal key is found
            const uint32_t prev = atomicCAS(&key[h], kEmpty, kk);
            if (prev == kEmpty || prev == kk) break;
            h = (h + 1) & (kHashSize - 1);
        }
        atomicMax(&tag[h], (uint32_t)(b + 1));
        pos[k] = (int)h;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kPerThread; k++) {
        const int b = threadIdx.x + k * kHashThreads;
        if (pos[k] < 0 || tag[pos[k]] != (uint32_t)(b + 1)) continue;
        const int64_t s = slot[k];
        prio[s] = val[k];
        if (!tree.maintain) continue;
        const uint64_t d = (uint64_t)val[k] - (uint64_t)old[k];  // mod 2^64
        if (d == 0) continue;
        add_u64(tree.tile_sums + (s >> 8), d);
        for (int l = 1; l < tree.nlevels; l++) {
            const int64_t n = node_of(s, l);
            if (l <= kAggLevels && tree.size[l] <= kAggNodes)
                atomicAdd(reinterpret_cast<unsigned long long*>(&agg[l - 1][n]), (unsigned long long)d);
            else
                add_u64(tree.upper[l] + n, d);
        }
    }
    if (bad) atomicOr(status, GEAR_STATUS_BAD_INDEX);
    if (!tree.maintain) return;
    __syncthreads();
    for (int l = 1; l < tree.nlevels && l <= kAggLevels; l++) {
        if (tree.size[l] > kAggNodes) continue;
        for (int n = threadIdx.x; n < tree.size[l]; n += kHashThreads)
            if (agg[l - 1][n] != 0) add_u64(tree.upper[l] + n, agg[l - 1][n]);
    }
}

__global__ void scatter_tag_kernel(const int64_t* __restrict__ idx, int32_t B, int64_t live,
                                   const uint8_t* __restrict__ committed, uint32_t* tag, uint32_t* status) {
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    const int64_t i = idx[b];
    if (i < 0 || i >= live) {
        atomicOr(status, GEAR_STATUS_BAD_INDEX);
        return;
    }
    if (committed != nullptr && committed[i] == 0) return;
    atomicMax(tag + i, (uint32_t)(b + 1));
}

__global__ void scatter_apply_kernel(const int64_t* __restrict__ idx, const uint32_t* __restrict__ newp, int32_t B,
                                     int64_t live, uint32_t* tag, uint32_t* __restrict__ prio, Tree tree) {
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    const int64_t i = idx[b];
    if (i < 0 || i >= live) return;
    // Dropped updates of uncommitted slots never raised the tag, so it is 0.
    if (tag[i] == (uint32_t)(b + 1)) {
        const uint32_t old = prio[i];
        prio[i] = newp[b];
        tag[i] = 0;
        if (tree.maintain) {
            const uint64_t d = (uint64_t)newp[b] - (uint64_t)old;  // mod 2^64
            if (d != 0) {
                add_u64(tree.tile_sums + (i >> 8), d);
                for (int l = 1; l < tree.nlevels; l++) add_u64(tree.upper[l] + node_of(i, l), d);
            }
        }
    }
}

Tree tree_of(const Table& t, bool maintain) {
    Tree tr{};
    tr.tile_sums = t.tile_sums;
    tr.nlevels = t.nlevels;
    for (int l = 0; l < t.nlevels; l++) {
        tr.upper[l] = l == 0 ? nullptr : t.upper[t.tree_parity][l];
        tr.size[l] = t.level_size[l];
    }
    tr.maintain = maintain ? 1 : 0;
    return tr;
}

}  // namespace

hipError_t launch_scatter(Table& t, const int64_t* idx, const uint32_t* newp, int32_t B, bool maintain_tree,
                          hipStream_t s) {
    // Ring tables: slots [0, live count); managed tables: any slot, updates
    // of uncommitted ones dropped.
    const int64_t live = t.managed ? t.N : live_count(t);
    const uint8_t* committed = t.managed ? t.committed : nullptr;
    const Tree tree = tree_of(t, maintain_tree);
    if (B <= kHashMaxBatch) {
        hipLaunchKernelGGL(scatter_lds_kernel, dim3(kParts), dim3(kHashThreads), 0, s, idx, newp, B, live,
                           committed, t.priority, t.status, tree);
        return hipGetLastError();
    }
    const unsigned grid = (unsigned)((B + 255) / 256);
    hipLaunchKernelGGL(scatter_tag_kernel, dim3(grid), dim3(256), 0, s, idx, B, live, committed, t.tag, t.status);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(scatter_apply_kernel, dim3(grid), dim3(256), 0, s, idx, newp, B, live, t.tag, t.priority,
                       tree);
    return hipGetLastError();
}

}  // namespace gear

using gear::fail;
using gear::hip_fail;

extern "C" int gear_update_priorities(gear_table* h, const int64_t* d_idx, const uint32_t* d_new_priorities,
                                      int32_t B, void* stream) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_update_priorities: table is NULL");
    gear::Table* t = reinterpret_cast<gear::Table*>(h);
    if (B < 0 || B > GEAR_MAX_BATCH) return fail(GEAR_E_INVAL, "gear_update_priorities: B out of range");
    if (B == 0) return GEAR_OK;
    if (d_idx == nullptr || d_new_priorities == nullptr)
        return fail(GEAR_E_INVAL, "gear_update_priorities: NULL pointer argument");
    gear::DeviceGuard guard(t->device);
    if (guard.error() != hipSuccess) return hip_fail(guard.error(), "gear_update_priorities: hipSetDevice");
    // Keep the tree current only if it is current now; otherwise the next
    // prioritized select rescans anyway.
    // Under global IS normalisation the next select rescans anyway, for the
    // chunk minima, so the tree is not maintained.
    const bool maintain = (t->options & GEAR_OPT_INCREMENTAL_TREE) && !(t->options & GEAR_OPT_IS_GLOBAL_MIN) &&
                          !t->cdf_dirty;
    hipError_t e = gear::launch_scatter(*t, d_idx, d_new_priorities, B, maintain, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "gear_update_priorities: launch");
    if (!maintain) t->cdf_dirty = true;
    return GEAR_OK;
}
