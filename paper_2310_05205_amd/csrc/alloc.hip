// Index manager of a table (GEAR Sec. 3.2): a block allocator with one queue
// of free indices and a status table whose priority is zero for indices that
// are free or still being written.
//
// Insertion (Sec. 3.2, trajectory insertion and deletion):
//   gear_allocate  dequeues free indices.  When none is free, or the
//                  committed and pending indices have reached the preset
//                  maximum, it first releases a victim by the removal
//                  strategy (FIFO: the oldest commit, LIFO: the newest): the
//                  victim's priority is zeroed on the device and its index
//                  joins the back of the free queue.
//   (the client writes the blocks of its indices in place, through the
//    column base addresses)
//   gear_commit    writes the priorities, marks the indices committed and
//                  appends them to the commit-order ring on the device, so
//                  they become selectable.
//
// The queue, the per-slot state and the commit order are host data: each
// call's decisions are a few integer operations per index.  The device keeps
// a copy of the commit-order ring (FIFO, LIFO and uniform selection read it)
// and a committed flag per slot (priority updates of other slots are
// dropped).  Index lists reach the device through the table's ring of
// pinned, mapped staging slots, which the kernels read in place; a slot is
// refilled only after its last reader has run, so the host waits only when
// every slot is still in use.
//
// Rows are written into their slots by one scatter kernel per column (any
// slot order), or, from pageable host memory that kernels cannot read, by
// one copy per run of consecutive slots.
#include <algorithm>
#include <cstring>
#include <new>

#include "gear_internal.h"

namespace gear {
namespace {

__global__ void evict_kernel(const int64_t* __restrict__ victims, int64_t n, uint32_t* __restrict__ prio,
                             uint8_t* __restrict__ committed) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= n) return;
    const int64_t i = victims[j];
    prio[i] = 0u;
    committed[i] = 0;
}

// Commit j of this chunk takes commit-order position pos0 + j (mod N).
__global__ void commit_kernel(const int64_t* __restrict__ idx, const uint32_t* __restrict__ p, int64_t n,
                              int64_t pos0, int64_t N, int32_t* __restrict__ order, uint32_t* __restrict__ prio,
                              uint8_t* __restrict__ committed) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= n) return;
    const int64_t i = idx[j];
    prio[i] = p[j];
    committed[i] = 1;
    int64_t pos = pos0 + j;
    if (pos >= N) pos -= N;
    order[pos] = (int32_t)i;
}

// Row scatter: row r of a contiguous [n][row] source goes to slot idx[r] of
// a column ([N][row]).  Rows of at least half a piece: a workgroup copies
// one piece of one row.  Smaller rows: a workgroup copies the whole rows that
// fit in one piece, the destination of each row staged in LDS.  Both the
// source (read once) and the table rows (not read soon) are accessed
// non-temporally: measured on gfx950, that beats plain loads and stores for
// this copy.  Pieces are small, 1 KiB for every element width (16 bytes per
// lane of a 64-lane workgroup): writing 200 KB rows into a full table, that
// reached 6.3 TB/s against 6.1 with 4 KiB and 5.6 with 16 KiB pieces.
constexpr int kRowThreads = 64;
template <typename V>
constexpr int row_unroll() { return 16 / (int)sizeof(V); }  // elements per lane
template <typename V>
constexpr int64_t row_piece() { return (int64_t)kRowThreads * row_unroll<V>(); }  // elements per piece

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

template <typename V>
__global__ __launch_bounds__(kRowThreads) void scatter_rows_kernel(const int64_t* __restrict__ idx,
                                                                   const V* __restrict__ src, V* __restrict__ dst,
                                                                   int64_t row_elems, int64_t pieces_per_row) {
    constexpr int U = row_unroll<V>();
    constexpr int64_t P = row_piece<V>();
    const int64_t q = blockIdx.x;
    const int64_t r = q / pieces_per_row;
    const int64_t off = (q - r * pieces_per_row) * P;
    const int64_t len = row_elems - off < P ? row_elems - off : P;
    const V* s = src + r * row_elems + off;
    V* d = dst + idx[r] * row_elems + off;
    if (len == P) {
        V v[U];
#pragma unroll
        for (int k = 0; k < U; k++) v[k] = __builtin_nontemporal_load(s + threadIdx.x + k * kRowThreads);
#pragma unroll
        for (int k = 0; k < U; k++) __builtin_nontemporal_store(v[k], d + threadIdx.x + k * kRowThreads);
    } else {
        for (int64_t e = threadIdx.x; e < len; e += kRowThreads)
            __builtin_nontemporal_store(__builtin_nontemporal_load(s + e), d + e);
    }
}

// Rows of fewer than half a piece: workgroup q copies rows
// q*rpw .. q*rpw + rpw - 1.  Element e of that range is row e / row_elems,
// computed as (e * magic) >> 32 with magic = ceil(2^32 / row_elems), exact
// for e below a piece (at most 1024 elements).
template <typename V>
__global__ __launch_bounds__(kRowThreads) void scatter_small_rows_kernel(const int64_t* __restrict__ idx, int64_t n,
                                                                         const V* __restrict__ src,
                                                                         V* __restrict__ dst, int64_t row_elems,
                                                                         int rpw, uint64_t magic) {
    __shared__ int64_t s_dst[row_piece<V>()];
    const int64_t r0 = (int64_t)blockIdx.x * rpw;
    const int nr = (int)(n - r0 < rpw ? n - r0 : rpw);
    for (int i = threadIdx.x; i < nr; i += kRowThreads) s_dst[i] = idx[r0 + i] * row_elems;
    __syncthreads();
    const V* s = src + r0 * row_elems;
    const uint32_t total = (uint32_t)(nr * row_elems);
    for (uint32_t e = threadIdx.x; e < total; e += kRowThreads) {
        const uint32_t r = (uint32_t)(((uint64_t)e * magic) >> 32);
        const uint32_t o = e - r * (uint32_t)row_elems;
        __builtin_nontemporal_store(__builtin_nontemporal_load(s + e), dst + s_dst[r] + o);
    }
}

template <typename V>
hipError_t launch_rows(const int64_t* d_idx, int64_t n, const uint8_t* src, uint8_t* dst, int64_t row_bytes,
                       hipStream_t s) {
    constexpr int64_t P = row_piece<V>();
    const int64_t row_elems = row_bytes / (int64_t)sizeof(V);
    if (row_elems * 2 < P) {
        const int rpw = (int)(P / row_elems);
        const uint64_t magic = ((1ull << 32) + (uint64_t)row_elems - 1) / (uint64_t)row_elems;
        hipLaunchKernelGGL(scatter_small_rows_kernel<V>, dim3((unsigned)((n + rpw - 1) / rpw)), dim3(kRowThreads), 0,
                           s, d_idx, n, reinterpret_cast<const V*>(src), reinterpret_cast<V*>(dst), row_elems, rpw,
                           magic);
        return hipGetLastError();
    }
    // One workgroup per piece; rows are split over launches so that no grid
    // exceeds 2^31 - 1 workgroups.
    const int64_t ppr = (row_elems + P - 1) / P;
    const int64_t rows_per_launch = ppr >= 0x7FFFFFFF ? 1 : 0x7FFFFFFF / ppr;
    for (int64_t r0 = 0; r0 < n; r0 += rows_per_launch) {
        const int64_t m = n - r0 < rows_per_launch ? n - r0 : rows_per_launch;
        hipLaunchKernelGGL(scatter_rows_kernel<V>, dim3((unsigned)(m * ppr)), dim3(kRowThreads), 0, s, d_idx + r0,
                           reinterpret_cast<const V*>(src + r0 * row_bytes), reinterpret_cast<V*>(dst), row_elems, ppr);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// Whether a kernel on the table's device can read `p` (device memory, or
// pinned / mapped host memory); pageable host memory cannot.
bool device_readable(const void* p) {
    hipPointerAttribute_t a;
    if (hipPointerGetAttributes(&a, p) != hipSuccess) {
        (void)hipGetLastError();  // clear the error a pageable pointer leaves
        return false;
    }
    return a.type == hipMemoryTypeDevice || a.type == hipMemoryTypeHost || a.type == hipMemoryTypeManaged;
}

// One slot of the table's pinned staging ring: a host list is copied into
// it by the CPU and read in place by the kernels of one chunk.  A slot is
// refilled only after the event recorded behind its last reader, so the
// host waits only when every slot is still being read.
struct PinSlot {
    int k;
    int64_t* h_idx;
    uint32_t* h_prio;
    const int64_t* d_idx;    // device addresses of the same memory
    const uint32_t* d_prio;
};

hipError_t acquire_slot(Table& t, PinSlot& ps) {
    ps.k = t.pin_next;
    t.pin_next = (ps.k + 1) % kStageSlots;
    const hipError_t e = hipEventSynchronize(t.pin_free[ps.k]);
    if (e != hipSuccess) return e;
    const int64_t off = (int64_t)ps.k * kStageSlotBytes;
    const int64_t prio_off = off + kStageRows * (int64_t)sizeof(int64_t);
    ps.h_idx = reinterpret_cast<int64_t*>(t.pin_host + off);
    ps.h_prio = reinterpret_cast<uint32_t*>(t.pin_host + prio_off);
    ps.d_idx = reinterpret_cast<const int64_t*>(t.pin_dev + off);
    ps.d_prio = reinterpret_cast<const uint32_t*>(t.pin_dev + prio_off);
    return hipSuccess;
}

// Call after enqueuing the last kernel that reads the slot.
hipError_t release_slot(Table& t, const PinSlot& ps, hipStream_t s) { return hipEventRecord(t.pin_free[ps.k], s); }

__global__ void copy_list_kernel(const int64_t* __restrict__ src, int64_t n, int64_t* __restrict__ dst) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j < n) dst[j] = src[j];
}

unsigned blocks_for(int64_t n) { return (unsigned)((n + 255) / 256); }

// Releases one victim by the removal strategy (host state only).
// Positions in the rings are below N and counts at most N, so a sum of the
// two wraps with one subtraction (no division in these per-index loops).
inline int64_t wrap(int64_t pos, int64_t N) { return pos >= N ? pos - N : pos; }

int64_t release_victim(Table& t) {
    int64_t pos;
    if (t.removal == GEAR_FIFO) {
        pos = t.ord_head;
        t.ord_head = wrap(t.ord_head + 1, t.N);
    } else {
        pos = wrap(t.ord_head + t.n_committed - 1, t.N);
    }
    const int32_t v = t.order_h[(size_t)pos];
    t.n_committed--;
    t.slot_state[(size_t)v] = kSlotFree;
    t.free_q[(size_t)wrap(t.fq_head + t.n_free, t.N)] = v;
    t.n_free++;
    return v;
}

}  // namespace

void free_index_manager(Table& t) {
    (void)hipFree(t.order);
    (void)hipFree(t.committed);
    t.order = nullptr;
    t.committed = nullptr;
    std::vector<int32_t>().swap(t.free_q);
    std::vector<int32_t>().swap(t.order_h);
    std::vector<uint8_t>().swap(t.slot_state);
    t.managed = false;
}

int write_rows(Table& t, int64_t n, const int64_t* idx, const void* const* col_src, hipStream_t s) {
    std::vector<bool> kernel_path((size_t)t.ncols);
    bool any_kernel = false;
    for (int c = 0; c < t.ncols; c++) {
        const int64_t rb = (int64_t)t.T * t.elem_bytes[c];
        const uint8_t* src = static_cast<const uint8_t*>(col_src[c]);
        kernel_path[(size_t)c] = device_readable(src);
        any_kernel = any_kernel || kernel_path[(size_t)c];
        if (kernel_path[(size_t)c]) continue;
        // Pageable host source: one copy per run of consecutive slots.
        uint8_t* hbase = t.residency == GEAR_HOST_PINNED ? t.col_host[c] : t.col_dev[c];
        int64_t r0 = 0;
        while (r0 < n) {
            int64_t r1 = r0 + 1;
            while (r1 < n && idx[r1] == idx[r1 - 1] + 1) r1++;
            hipError_t e = hipMemcpyAsync(hbase + (size_t)idx[r0] * rb, src + (size_t)r0 * rb,
                                          (size_t)(r1 - r0) * rb, hipMemcpyDefault, s);
            if (e != hipSuccess) return hip_fail(e, "row copy");
            r0 = r1;
        }
    }
    if (!any_kernel) return GEAR_OK;
    // The slot list moves to HBM once per chunk for all columns.
    for (int64_t off = 0; off < n; off += kStageRows) {
        const int64_t cnt = std::min(n - off, kStageRows);
        PinSlot ps;
        hipError_t e = acquire_slot(t, ps);
        if (e == hipSuccess) {
            std::memcpy(ps.h_idx, idx + off, sizeof(int64_t) * (size_t)cnt);
            hipLaunchKernelGGL(copy_list_kernel, dim3(blocks_for(cnt)), dim3(256), 0, s, ps.d_idx, cnt, t.stage_idx);
            e = hipGetLastError();
        }
        if (e == hipSuccess) e = release_slot(t, ps, s);
        if (e != hipSuccess) return hip_fail(e, "staging slots");
        for (int c = 0; c < t.ncols && e == hipSuccess; c++) {
            if (!kernel_path[(size_t)c]) continue;
            const int64_t rb = (int64_t)t.T * t.elem_bytes[c];
            uint8_t* base = t.col_dev[c];  // the mapped device address for pinned tables
            const uint8_t* sc = static_cast<const uint8_t*>(col_src[c]) + (size_t)off * rb;
            const uintptr_t align = reinterpret_cast<uintptr_t>(sc) | reinterpret_cast<uintptr_t>(base) | (uintptr_t)rb;
            if (align % 16 == 0)
                e = launch_rows<u32x4_t>(t.stage_idx, cnt, sc, base, rb, s);
            else if (align % 4 == 0)
                e = launch_rows<uint32_t>(t.stage_idx, cnt, sc, base, rb, s);
            else
                e = launch_rows<uint8_t>(t.stage_idx, cnt, sc, base, rb, s);
        }
        if (e != hipSuccess) return hip_fail(e, "row scatter");
    }
    return GEAR_OK;
}

int managed_insert(Table& t, int64_t n, const void* const* col_src, const uint32_t* priorities, hipStream_t s) {
    if (t.n_pending + n > t.max_selectable)
        return fail(GEAR_E_INSUFFICIENT, "gear_insert: more rows than the index manager can hold pending");
    std::vector<int64_t> idx;
    try {
        idx.resize((size_t)n);
    } catch (const std::bad_alloc&) {
        return fail(GEAR_E_NOMEM, "gear_insert: host index list");
    }
    gear_table* h = reinterpret_cast<gear_table*>(&t);
    int rc = gear_allocate(h, n, idx.data(), s);
    if (rc != GEAR_OK) return rc;
    rc = write_rows(t, n, idx.data(), col_src, s);
    if (rc != GEAR_OK) return rc;
    return gear_commit(h, n, idx.data(), priorities, s);
}

}  // namespace gear

using gear::fail;
using gear::hip_fail;
using gear::Table;

extern "C" int gear_table_use_allocator(gear_table* h, int32_t removal, int64_t max_selectable) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_table_use_allocator: table is NULL");
    Table* t = reinterpret_cast<Table*>(h);
    if (removal != GEAR_FIFO && removal != GEAR_LIFO)
        return fail(GEAR_E_INVAL, "gear_table_use_allocator: removal must be GEAR_FIFO or GEAR_LIFO");
    if (max_selectable < 1 || max_selectable > t->N)
        return fail(GEAR_E_INVAL, "gear_table_use_allocator: max_selectable must lie in [1, capacity]");
    if (t->managed) return fail(GEAR_E_INVAL, "gear_table_use_allocator: the table already has an index manager");
    if (t->next_seq != 0) return fail(GEAR_E_INVAL, "gear_table_use_allocator: the table already holds insertions");
    gear::DeviceGuard guard(t->device);
    if (guard.error() != hipSuccess) return hip_fail(guard.error(), "gear_table_use_allocator: hipSetDevice");
    try {
        t->free_q.resize((size_t)t->N);
        t->order_h.resize((size_t)t->N);
        t->slot_state.assign((size_t)t->N, gear::kSlotFree);
    } catch (const std::bad_alloc&) {
        gear::free_index_manager(*t);
        return fail(GEAR_E_NOMEM, "gear_table_use_allocator: host index arrays");
    }
    for (int64_t i = 0; i < t->N; i++) t->free_q[(size_t)i] = (int32_t)i;  // every index free, in index order
    hipError_t e = hipSuccess;
    gear::AllocHook hook;
    if ((e = hook.fail_next() ? hipErrorOutOfMemory
                              : hipMalloc(reinterpret_cast<void**>(&t->order), sizeof(int32_t) * (size_t)t->N)) !=
            hipSuccess ||
        (e = hook.fail_next() ? hipErrorOutOfMemory : hipMalloc(reinterpret_cast<void**>(&t->committed), (size_t)t->N)) !=
            hipSuccess) {
        gear::free_index_manager(*t);
        (void)hipGetLastError();  // reported here, not by a later launch
        return fail(GEAR_E_NOMEM, "gear_table_use_allocator: device arrays");
    }
    if ((e = hipMemset(t->committed, 0, (size_t)t->N)) != hipSuccess ||
        (e = hipDeviceSynchronize()) != hipSuccess) {
        gear::free_index_manager(*t);
        return hip_fail(e, "gear_table_use_allocator: initialising");
    }
    t->fq_head = 0;
    t->n_free = t->N;
    t->ord_head = 0;
    t->n_committed = 0;
    t->n_pending = 0;
    t->removal = removal;
    t->max_selectable = max_selectable;
    t->managed = true;
    return GEAR_OK;
}

extern "C" int gear_allocate(gear_table* h, int64_t n, int64_t* idx_out, void* stream) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_allocate: table is NULL");
    Table* t = reinterpret_cast<Table*>(h);
    if (!t->managed) return fail(GEAR_E_INVAL, "gear_allocate: the table has no index manager");
    if (n < 0) return fail(GEAR_E_INVAL, "gear_allocate: n < 0");
    if (n == 0) return GEAR_OK;
    if (idx_out == nullptr) return fail(GEAR_E_INVAL, "gear_allocate: idx_out is NULL");
    if (t->n_pending + n > t->max_selectable)
        return fail(GEAR_E_INSUFFICIENT, "gear_allocate: pending indices would exceed the maximum");
    gear::DeviceGuard guard(t->device);
    if (guard.error() != hipSuccess) return hip_fail(guard.error(), "gear_allocate: hipSetDevice");
    hipStream_t s = static_cast<hipStream_t>(stream);
    std::vector<int64_t> victims;
    try {
        victims.reserve((size_t)n);
    } catch (const std::bad_alloc&) {
        return fail(GEAR_E_NOMEM, "gear_allocate: host victim list");
    }
    for (int64_t r = 0; r < n; r++) {
        // Pending stays below the maximum here, so a victim exists whenever one is needed.
        while (t->n_free == 0 || t->n_committed + t->n_pending >= t->max_selectable)
            victims.push_back(gear::release_victim(*t));
        const int32_t i = t->free_q[(size_t)t->fq_head];
        t->fq_head = t->fq_head + 1 == t->N ? 0 : t->fq_head + 1;
        t->n_free--;
        t->slot_state[(size_t)i] = gear::kSlotPending;
        t->n_pending++;
        idx_out[r] = i;
    }
    // Victims become unselectable before the caller writes into any slot.
    for (size_t off = 0; off < victims.size(); off += (size_t)gear::kStageRows) {
        const int64_t cnt = (int64_t)std::min(victims.size() - off, (size_t)gear::kStageRows);
        gear::PinSlot ps;
        hipError_t e = gear::acquire_slot(*t, ps);
        if (e != hipSuccess) return hip_fail(e, "gear_allocate: staging victims");
        std::memcpy(ps.h_idx, victims.data() + off, sizeof(int64_t) * (size_t)cnt);
        hipLaunchKernelGGL(gear::evict_kernel, dim3(gear::blocks_for(cnt)), dim3(256), 0, s, ps.d_idx, cnt,
                           t->priority, t->committed);
        if ((e = hipGetLastError()) == hipSuccess) e = gear::release_slot(*t, ps, s);
        if (e != hipSuccess) return hip_fail(e, "gear_allocate: launch");
    }
    if (!victims.empty()) t->cdf_dirty = true;
    return GEAR_OK;
}

extern "C" int gear_commit(gear_table* h, int64_t n, const int64_t* idx, const uint32_t* priorities, void* stream) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_commit: table is NULL");
    Table* t = reinterpret_cast<Table*>(h);
    if (!t->managed) return fail(GEAR_E_INVAL, "gear_commit: the table has no index manager");
    if (n < 0) return fail(GEAR_E_INVAL, "gear_commit: n < 0");
    if (n == 0) return GEAR_OK;
    if (idx == nullptr || priorities == nullptr) return fail(GEAR_E_INVAL, "gear_commit: NULL pointer argument");
    // Every index pending and listed once; marks are undone on any failure.
    int64_t r = 0;
    for (; r < n; r++) {
        if (idx[r] < 0 || idx[r] >= t->N || t->slot_state[(size_t)idx[r]] != gear::kSlotPending) break;
        t->slot_state[(size_t)idx[r]] = gear::kSlotMark;
    }
    for (int64_t q = 0; q < r; q++) t->slot_state[(size_t)idx[q]] = gear::kSlotPending;
    if (r < n) return fail(GEAR_E_INVAL, "gear_commit: an index is not pending or is listed twice");
    gear::DeviceGuard guard(t->device);
    if (guard.error() != hipSuccess) return hip_fail(guard.error(), "gear_commit: hipSetDevice");
    hipStream_t s = static_cast<hipStream_t>(stream);
    // Priorities in device or pinned memory are read in place; pageable
    // ones go through the staging slot with the indices.
    const bool prio_in_place = gear::device_readable(priorities);
    for (int64_t off = 0; off < n; off += gear::kStageRows) {
        const int64_t cnt = std::min(n - off, gear::kStageRows);
        gear::PinSlot ps;
        hipError_t e = gear::acquire_slot(*t, ps);
        if (e != hipSuccess) return hip_fail(e, "gear_commit: staging");
        std::memcpy(ps.h_idx, idx + off, sizeof(int64_t) * (size_t)cnt);
        const uint32_t* p = priorities + off;
        if (!prio_in_place) {
            std::memcpy(ps.h_prio, p, sizeof(uint32_t) * (size_t)cnt);
            p = ps.d_prio;
        }
        const int64_t pos0 = gear::wrap(t->ord_head + t->n_committed, t->N);
        hipLaunchKernelGGL(gear::commit_kernel, dim3(gear::blocks_for(cnt)), dim3(256), 0, s, ps.d_idx, p, cnt, pos0,
                           t->N, t->order, t->priority, t->committed);
        if ((e = hipGetLastError()) == hipSuccess) e = gear::release_slot(*t, ps, s);
        if (e != hipSuccess) return hip_fail(e, "gear_commit: launch");
        int64_t pos = pos0;
        for (int64_t j = off; j < off + cnt; j++) {
            t->slot_state[(size_t)idx[j]] = gear::kSlotCommitted;
            t->order_h[(size_t)pos] = (int32_t)idx[j];
            pos = gear::wrap(pos + 1, t->N);
        }
        t->n_committed += cnt;
        t->n_pending -= cnt;
    }
    t->next_seq += (uint64_t)n;
    t->cdf_dirty = true;
    return GEAR_OK;
}

extern "C" int gear_write_rows(gear_table* h, int64_t n, const int64_t* idx, const void* const* col_src,
                               void* stream) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_write_rows: table is NULL");
    Table* t = reinterpret_cast<Table*>(h);
    if (n < 0) return fail(GEAR_E_INVAL, "gear_write_rows: n < 0");
    if (n == 0 || t->ncols == 0) return GEAR_OK;
    if (idx == nullptr || col_src == nullptr) return fail(GEAR_E_INVAL, "gear_write_rows: NULL pointer argument");
    for (int c = 0; c < t->ncols; c++)
        if (col_src[c] == nullptr) return fail(GEAR_E_INVAL, "gear_write_rows: a column source is NULL");
    for (int64_t r = 0; r < n; r++)
        if (idx[r] < 0 || idx[r] >= t->N) return fail(GEAR_E_INVAL, "gear_write_rows: a slot is out of range");
    gear::DeviceGuard guard(t->device);
    if (guard.error() != hipSuccess) return hip_fail(guard.error(), "gear_write_rows: hipSetDevice");
    return gear::write_rows(*t, n, idx, col_src, static_cast<hipStream_t>(stream));
}

extern "C" int gear_allocator_info(const gear_table* h, int64_t* committed, int64_t* pending, int64_t* free_count) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_allocator_info: table is NULL");
    const Table* t = reinterpret_cast<const Table*>(h);
    if (!t->managed) return fail(GEAR_E_INVAL, "gear_allocator_info: the table has no index manager");
    if (committed) *committed = t->n_committed;
    if (pending) *pending = t->n_pending;
    if (free_count) *free_count = t->n_free;
    return GEAR_OK;
}
