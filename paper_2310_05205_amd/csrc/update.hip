// Priority update on gfx950 (GEAR Sec. 3.2: the status table holds the
// priorities; updates are consolidated and committed).
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

__global__ __launch_bounds__(kHashThreads) void scatter_lds_kernel(const int64_t* __restrict__ idx,
                                                                   const uint32_t* __restrict__ newp, int32_t B,
                                                                   int64_t live, uint32_t* __restrict__ prio,
                                                                   uint32_t* status) {
    __shared__ uint32_t key[kHashSize];
    __shared__ uint32_t tag[kHashSize];
    for (int h = threadIdx.x; h < kHashSize; h += kHashThreads) {
        key[h] = kEmpty;
        tag[h] = 0u;
    }
    int64_t slot[kPerThread];
    uint32_t val[kPerThread];
#pragma unroll
    for (int k = 0; k < kPerThread; k++) {
        const int b = threadIdx.x + k * kHashThreads;
        slot[k] = b < B ? idx[b] : -1;
        val[k] = b < B ? newp[b] : 0u;
    }
    __syncthreads();
    int pos[kPerThread];
    bool bad = false;
#pragma unroll
    for (int k = 0; k < kPerThread; k++) {
        const int b = threadIdx.x + k * kHashThreads;
        pos[k] = -1;
        if (b >= B) continue;
        if (slot[k] < 0 || slot[k] >= live) {
            if (blockIdx.x == 0) bad = true;
            continue;
        }
        const uint32_t kk = (uint32_t)slot[k];
        if (((kk * 0x85EBCA6Bu) >> (32 - kPartBits)) != blockIdx.x) continue;  // another partition's slot
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
        if (pos[k] >= 0 && tag[pos[k]] == (uint32_t)(b + 1)) prio[slot[k]] = val[k];
    }
    if (bad) atomicOr(status, GEAR_STATUS_BAD_INDEX);
}

__global__ void scatter_tag_kernel(const int64_t* __restrict__ idx, int32_t B, int64_t live, uint32_t* tag,
                                   uint32_t* status) {
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    const int64_t i = idx[b];
    if (i < 0 || i >= live) {
        atomicOr(status, GEAR_STATUS_BAD_INDEX);
        return;
    }
    atomicMax(tag + i, (uint32_t)(b + 1));
}

__global__ void scatter_apply_kernel(const int64_t* __restrict__ idx, const uint32_t* __restrict__ newp, int32_t B,
                                     int64_t live, uint32_t* tag, uint32_t* __restrict__ prio) {
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    const int64_t i = idx[b];
    if (i < 0 || i >= live) return;
    if (tag[i] == (uint32_t)(b + 1)) {
        prio[i] = newp[b];
        tag[i] = 0;
    }
}

}  // namespace

hipError_t launch_scatter(Table& t, const int64_t* idx, const uint32_t* newp, int32_t B, hipStream_t s) {
    const int64_t live = t.next_seq < (uint64_t)t.N ? (int64_t)t.next_seq : t.N;
    if (B <= kHashMaxBatch) {
        hipLaunchKernelGGL(scatter_lds_kernel, dim3(kParts), dim3(kHashThreads), 0, s, idx, newp, B, live,
                           t.priority, t.status);
        return hipGetLastError();
    }
    const unsigned grid = (unsigned)((B + 255) / 256);
    hipLaunchKernelGGL(scatter_tag_kernel, dim3(grid), dim3(256), 0, s, idx, B, live, t.tag, t.status);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(scatter_apply_kernel, dim3(grid), dim3(256), 0, s, idx, newp, B, live, t.tag, t.priority);
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
    hipError_t e = gear::launch_scatter(*t, d_idx, d_new_priorities, B, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "gear_update_priorities: launch");
    t->cdf_dirty = true;
    return GEAR_OK;
}
