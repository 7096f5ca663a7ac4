// Priority update on gfx950 (GEAR Sec. 3.2: the status table holds the
// priorities; updates are consolidated and committed).
//
// The batch is applied as if in order, so for a slot that appears several
// times the last occurrence's value wins.  Two kernels:
//   tag    every draw b raises tag[slot] to b+1 (atomic max), so after the
//          kernel tag[slot] names the last occurrence of that slot;
//   apply  the draw whose b+1 equals tag[slot] writes the new priority and
//          puts the tag back to zero.  Other draws of the same slot see
//          either the winner's tag or zero, never their own, so they never
//          write.  Tags are zero again when the kernel ends.
#include "gear_internal.h"

namespace gear {
namespace {

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
