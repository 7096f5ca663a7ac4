// Host runtime of the replay store: creation, insertion with FIFO removal,
// status synchronisation and accessors (GEAR Sec. 3.2).
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <string>

#include "gear_internal.h"

namespace gear {

namespace {
thread_local std::string g_last_error;
}

int fail(int code, const std::string& msg) {
    g_last_error = msg;
    return code;
}

int hip_fail(hipError_t e, const char* what) {
    std::string m = what;
    m += ": ";
    m += hipGetErrorString(e);
    return fail(GEAR_E_HIP, m);
}

DeviceGuard::DeviceGuard(int dev) {
    // Kernel launches are checked with hipGetLastError, which also returns
    // an error left pending by any earlier HIP call of this thread (a failed
    // allocation elsewhere, say).  Clear it, so that the call's return code
    // describes only its own work.
    (void)hipGetLastError();
    int cur = -1;
    err_ = hipGetDevice(&cur);
    if (err_ == hipSuccess && cur != dev) {
        err_ = hipSetDevice(dev);
        if (err_ == hipSuccess) prev_ = cur;
    }
}

DeviceGuard::~DeviceGuard() {
    if (prev_ >= 0) (void)hipSetDevice(prev_);
}

AllocHook::AllocHook() {
    const char* v = getenv("GEAR_TEST_FAIL_ALLOC");
    if (v != nullptr) fail_at_ = strtol(v, nullptr, 10);
}

}  // namespace gear

using gear::fail;
using gear::hip_fail;
using gear::Table;

namespace {

void free_table(Table* t) {
    if (!t) return;
    gear::free_index_manager(*t);
    (void)hipFree(t->stage_idx);
    if (t->pin_host) (void)hipHostFree(t->pin_host);
    for (int k = 0; k < gear::kStageSlots; k++)
        if (t->pin_free[k]) (void)hipEventDestroy(t->pin_free[k]);
    for (int c = 0; c < t->ncols; c++) {
        if (t->residency == GEAR_HOST_PINNED) {
            if (t->col_host[c]) (void)hipHostFree(t->col_host[c]);
        } else if (t->col_dev[c]) {
            (void)hipFree(t->col_dev[c]);
        }
    }
    (void)hipFree(t->priority);
    (void)hipFree(t->tag);
    (void)hipFree(t->tile_sums);
    for (int c = 0; c < 2; c++)
        for (int l = 0; l < gear::kMaxLevels; l++) (void)hipFree(t->upper[c][l]);
    (void)hipFree(t->wg_min);
    (void)hipFree(t->chunk_min);
    (void)hipFree(t->topk_hist);
    (void)hipFree(t->topk_state);
    (void)hipFree(t->topk_local);
    (void)hipFree(t->topk_keys);
    (void)hipFree(t->status);
    delete t;
}

template <typename P>
hipError_t dmalloc(gear::AllocHook& hook, P** p, size_t bytes) {
    if (hook.fail_next()) return hipErrorOutOfMemory;
    return hipMalloc(reinterpret_cast<void**>(p), bytes);
}

hipError_t hmalloc(gear::AllocHook& hook, void** p, size_t bytes, unsigned flags) {
    if (hook.fail_next()) return hipErrorOutOfMemory;
    return hipHostMalloc(p, bytes, flags);
}

}  // namespace

namespace {

int dtype_bytes(int32_t dtype) {
    switch (dtype) {
        case GEAR_DTYPE_U8: case GEAR_DTYPE_I8: return 1;
        case GEAR_DTYPE_U16: case GEAR_DTYPE_I16: case GEAR_DTYPE_F16: case GEAR_DTYPE_BF16: return 2;
        case GEAR_DTYPE_U32: case GEAR_DTYPE_I32: case GEAR_DTYPE_F32: return 4;
        case GEAR_DTYPE_U64: case GEAR_DTYPE_I64: case GEAR_DTYPE_F64: return 8;
        default: return 0;
    }
}

// Column names, types and element counts of a new table; byte columns when
// `cols` is NULL.
struct ColumnMeta {
    std::vector<std::string> name;
    std::vector<int32_t> dtype, elems;
};

int create_table(const int64_t* elem_bytes, int32_t ncols, int64_t capacity, int32_t T, int32_t residency,
                 int32_t device, gear_table** out, ColumnMeta meta);

}  // namespace

extern "C" int gear_table_create(const int64_t* elem_bytes, int32_t ncols, int64_t capacity, int32_t T,
                                 int32_t residency, int32_t device, gear_table** out) {
    ColumnMeta meta;
    if (elem_bytes != nullptr && ncols > 0 && ncols <= GEAR_MAX_COLUMNS)
        for (int c = 0; c < ncols; c++) {
            meta.name.push_back("c" + std::to_string(c));
            meta.dtype.push_back(GEAR_DTYPE_U8);
            meta.elems.push_back((int32_t)(elem_bytes[c] > 0 && elem_bytes[c] <= (1ll << 30) ? elem_bytes[c] : 0));
        }
    return create_table(elem_bytes, ncols, capacity, T, residency, device, out, std::move(meta));
}

extern "C" int gear_table_create_columns(const gear_column* cols, int32_t ncols, int64_t capacity, int32_t T,
                                         int32_t residency, int32_t device, gear_table** out) {
    if (out == nullptr) return fail(GEAR_E_INVAL, "gear_table_create_columns: out is NULL");
    *out = nullptr;
    if (ncols < 0 || ncols > GEAR_MAX_COLUMNS)
        return fail(GEAR_E_INVAL, "gear_table_create_columns: ncols out of range");
    if (ncols > 0 && cols == nullptr) return fail(GEAR_E_INVAL, "gear_table_create_columns: cols is NULL");
    ColumnMeta meta;
    std::vector<int64_t> eb;
    for (int c = 0; c < ncols; c++) {
        if (cols[c].name == nullptr) return fail(GEAR_E_INVAL, "gear_table_create_columns: a column name is NULL");
        const size_t len = strnlen(cols[c].name, GEAR_MAX_NAME + 1);
        if (len == 0 || len > GEAR_MAX_NAME)
            return fail(GEAR_E_INVAL, "gear_table_create_columns: a column name is empty or longer than GEAR_MAX_NAME");
        std::string name(cols[c].name, len);
        for (const std::string& other : meta.name)
            if (other == name) return fail(GEAR_E_INVAL, "gear_table_create_columns: repeated column name " + name);
        const int size = dtype_bytes(cols[c].dtype);
        if (size == 0) return fail(GEAR_E_INVAL, "gear_table_create_columns: unknown dtype of column " + name);
        if (cols[c].elems_per_step < 1)
            return fail(GEAR_E_INVAL, "gear_table_create_columns: elems_per_step < 1 in column " + name);
        meta.name.push_back(name);
        meta.dtype.push_back(cols[c].dtype);
        meta.elems.push_back(cols[c].elems_per_step);
        eb.push_back((int64_t)size * cols[c].elems_per_step);
    }
    return create_table(eb.data(), ncols, capacity, T, residency, device, out, std::move(meta));
}

namespace {

int create_table(const int64_t* elem_bytes, int32_t ncols, int64_t capacity, int32_t T, int32_t residency,
                 int32_t device, gear_table** out, ColumnMeta meta) {
    if (out == nullptr) return fail(GEAR_E_INVAL, "gear_table_create: out is NULL");
    *out = nullptr;
    if (ncols < 0 || ncols > GEAR_MAX_COLUMNS) return fail(GEAR_E_INVAL, "gear_table_create: ncols out of range");
    if (ncols > 0 && elem_bytes == nullptr) return fail(GEAR_E_INVAL, "gear_table_create: elem_bytes is NULL");
    if (capacity < 1 || capacity > GEAR_MAX_CAPACITY) return fail(GEAR_E_INVAL, "gear_table_create: capacity out of range");
    if (T < 1) return fail(GEAR_E_INVAL, "gear_table_create: T must be >= 1");
    if (residency != GEAR_DEVICE && residency != GEAR_HOST_PINNED)
        return fail(GEAR_E_INVAL, "gear_table_create: unknown residency");
    for (int c = 0; c < ncols; c++) {
        if (elem_bytes[c] < 1 || elem_bytes[c] > (1ll << 30))
            return fail(GEAR_E_INVAL, "gear_table_create: elem_bytes out of range");
        // Column bytes must fit in int64 with room for offsets.
        if ((double)capacity * (double)T * (double)elem_bytes[c] > 9.0e18)
            return fail(GEAR_E_INVAL, "gear_table_create: column too large");
    }
    if (device < 0) return fail(GEAR_E_INVAL, "gear_table_create: negative device");
    int ndev = 0;
    hipError_t e = hipGetDeviceCount(&ndev);
    if (e != hipSuccess) return hip_fail(e, "gear_table_create: hipGetDeviceCount");
    if (device >= ndev) return fail(GEAR_E_INVAL, "gear_table_create: no such device");
    gear::DeviceGuard guard(device);
    if (guard.error() != hipSuccess) return hip_fail(guard.error(), "gear_table_create: hipSetDevice");
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, device);
    if (e != hipSuccess) return hip_fail(e, "gear_table_create: hipGetDeviceProperties");
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(GEAR_E_INVAL, std::string("gear_table_create: library is built for gfx950, device is ") + prop.gcnArchName);

    gear::AllocHook hook;
    Table* t = new Table();
    t->device = device;
    t->residency = residency;
    t->N = capacity;
    t->T = T;
    t->ncols = ncols;
    t->elem_bytes.assign(elem_bytes, elem_bytes + ncols);
    t->col_name = std::move(meta.name);
    t->col_dtype = std::move(meta.dtype);
    t->col_elems = std::move(meta.elems);
    t->col_dev.assign(ncols, nullptr);
    t->col_host.assign(ncols, nullptr);

    auto oom = [&](const char* what, hipError_t err) {
        free_table(t);
        (void)hipGetLastError();  // the failed allocation's error is reported here, not by a later launch
        std::string m = std::string("gear_table_create: allocation of ") + what + " failed: " + hipGetErrorString(err);
        return fail(GEAR_E_NOMEM, m);
    };

    for (int c = 0; c < ncols; c++) {
        size_t bytes = (size_t)capacity * (size_t)T * (size_t)elem_bytes[c];
        if (residency == GEAR_DEVICE) {
            e = dmalloc(hook, &t->col_dev[c], bytes);
            if (e != hipSuccess) return oom("a device column", e);
            // Slots never inserted read as zeros.
            e = hipMemsetAsync(t->col_dev[c], 0, bytes, nullptr);
            if (e != hipSuccess) {
                free_table(t);
                return hip_fail(e, "gear_table_create: clearing a device column");
            }
        } else {
            // Page-locked, mapped into the GPU's address space.  Coarse-grained
            // (non-coherent) so the GPU may cache lines it reads; the table is
            // only written by insertion, ordered on the stream.
            void* h = nullptr;
            e = hmalloc(hook, &h, bytes, hipHostMallocMapped | hipHostMallocNonCoherent);
            if (e != hipSuccess) return oom("a pinned host column", e);
            t->col_host[c] = static_cast<uint8_t*>(h);
            void* d = nullptr;
            e = hipHostGetDevicePointer(&d, h, 0);
            if (e != hipSuccess) return oom("a device view of a pinned column", e);
            t->col_dev[c] = static_cast<uint8_t*>(d);
            // Slots never inserted read as zeros: pinned memory the runtime
            // hands out again after a free keeps its old contents.
            e = hipMemsetAsync(t->col_dev[c], 0, bytes, nullptr);
            if (e != hipSuccess) {
                free_table(t);
                return hip_fail(e, "gear_table_create: clearing a pinned column");
            }
        }
    }

    // Sum tree geometry.
    t->ntiles = (capacity + gear::kTile - 1) / gear::kTile;
    t->nchunks = (t->ntiles + gear::kTilesPerChunk - 1) / gear::kTilesPerChunk;
    int64_t sz = t->ntiles;
    t->nlevels = 0;
    while (true) {
        t->level_size[t->nlevels] = sz;
        t->nlevels++;
        if (sz <= gear::kFanout) break;
        sz = (sz + gear::kFanout - 1) / gear::kFanout;
    }
    if ((e = dmalloc(hook, &t->priority, sizeof(uint32_t) * capacity)) != hipSuccess) return oom("priorities", e);
    if ((e = dmalloc(hook, &t->tag, sizeof(uint32_t) * capacity)) != hipSuccess) return oom("scatter tags", e);
    if ((e = dmalloc(hook, &t->tile_sums, sizeof(uint64_t) * t->ntiles)) != hipSuccess) return oom("tile sums", e);
    for (int c = 0; c < 2; c++)
        for (int l = 1; l < t->nlevels; l++) {
            if ((e = dmalloc(hook, &t->upper[c][l], sizeof(uint64_t) * t->level_size[l])) != hipSuccess)
                return oom("sum tree levels", e);
            if ((e = hipMemset(t->upper[c][l], 0, sizeof(uint64_t) * t->level_size[l])) != hipSuccess) {
                free_table(t);
                return hip_fail(e, "gear_table_create: clearing the sum tree");
            }
        }
    if ((e = dmalloc(hook, &t->wg_min, sizeof(uint32_t) * gear::kSearchMaxGrid)) != hipSuccess) return oom("batch minima", e);
    if ((e = dmalloc(hook, &t->chunk_min, sizeof(uint32_t) * t->nchunks)) != hipSuccess) return oom("chunk minima", e);
    if ((e = dmalloc(hook, &t->status, sizeof(uint32_t))) != hipSuccess) return oom("status word", e);
    // Staging for host index and priority lists (row writes, index manager).
    if ((e = dmalloc(hook, &t->stage_idx, sizeof(int64_t) * gear::kStageRows)) != hipSuccess ||
        (e = hmalloc(hook, reinterpret_cast<void**>(&t->pin_host), (size_t)(gear::kStageSlotBytes * gear::kStageSlots),
                     hipHostMallocMapped | hipHostMallocCoherent)) != hipSuccess)
        return oom("index staging", e);
    {
        void* d = nullptr;
        if ((e = hipHostGetDevicePointer(&d, t->pin_host, 0)) != hipSuccess) return oom("a device view of the staging", e);
        t->pin_dev = static_cast<uint8_t*>(d);
    }
    for (int k = 0; k < gear::kStageSlots; k++)
        if ((e = hipEventCreateWithFlags(&t->pin_free[k], hipEventDisableTiming)) != hipSuccess) {
            free_table(t);
            return hip_fail(e, "gear_table_create: staging events");
        }
    if ((e = dmalloc(hook, &t->topk_hist, sizeof(uint32_t) * 3 * gear::kTopkBins)) != hipSuccess ||
        (e = dmalloc(hook, &t->topk_state, sizeof(uint32_t) * gear::kTopkStateWords)) != hipSuccess ||
        (e = dmalloc(hook, &t->topk_local, sizeof(uint32_t) * 3 * gear::kTopkMaxGrid * gear::kTopkBins)) != hipSuccess ||
        (e = dmalloc(hook, &t->topk_keys, sizeof(uint64_t) * gear::kTopkMaxK)) != hipSuccess)
        return oom("TopK scratch", e);

    if ((e = hipMemset(t->priority, 0, sizeof(uint32_t) * capacity)) != hipSuccess ||
        (e = hipMemset(t->tag, 0, sizeof(uint32_t) * capacity)) != hipSuccess ||
        (e = hipMemset(t->tile_sums, 0, sizeof(uint64_t) * t->ntiles)) != hipSuccess ||
        (e = hipMemset(t->wg_min, 0xFF, sizeof(uint32_t) * gear::kSearchMaxGrid)) != hipSuccess ||
        (e = hipMemset(t->status, 0, sizeof(uint32_t))) != hipSuccess ||
        (e = hipMemset(t->topk_hist, 0, sizeof(uint32_t) * 3 * gear::kTopkBins)) != hipSuccess ||
        (e = hipMemset(t->topk_state, 0, sizeof(uint32_t) * gear::kTopkStateWords)) != hipSuccess ||
        (e = hipDeviceSynchronize()) != hipSuccess) {
        free_table(t);
        return hip_fail(e, "gear_table_create: initialising table state");
    }
    *out = reinterpret_cast<gear_table*>(t);
    return GEAR_OK;
}

}  // namespace

extern "C" int gear_table_destroy(gear_table* h) {
    if (h == nullptr) return GEAR_OK;
    Table* t = reinterpret_cast<Table*>(h);
    gear::DeviceGuard guard(t->device);
    hipError_t e = hipDeviceSynchronize();
    free_table(t);
    if (e != hipSuccess) return hip_fail(e, "gear_table_destroy: hipDeviceSynchronize");
    return GEAR_OK;
}

extern "C" int gear_insert(gear_table* h, int64_t n, const void* const* col_src, const uint32_t* priorities,
                           void* stream) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_insert: table is NULL");
    Table* t = reinterpret_cast<Table*>(h);
    if (n < 0) return fail(GEAR_E_INVAL, "gear_insert: n < 0");
    if (n == 0) return GEAR_OK;
    if (priorities == nullptr) return fail(GEAR_E_INVAL, "gear_insert: priorities is NULL");
    if (t->ncols > 0) {
        if (col_src == nullptr) return fail(GEAR_E_INVAL, "gear_insert: col_src is NULL");
        for (int c = 0; c < t->ncols; c++)
            if (col_src[c] == nullptr) return fail(GEAR_E_INVAL, "gear_insert: a column source is NULL");
    }
    gear::DeviceGuard guard(t->device);
    if (guard.error() != hipSuccess) return hip_fail(guard.error(), "gear_insert: hipSetDevice");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (t->managed) return gear::managed_insert(*t, n, col_src, priorities, s);

    // Rows written one after another into slot k mod N: only the last N
    // of a longer batch survive, so copy those.
    const int64_t skip = n > t->N ? n - t->N : 0;
    const int64_t rows = n - skip;
    const int64_t slot0 = (int64_t)((t->next_seq + (uint64_t)skip) % (uint64_t)t->N);
    const int64_t first = rows < t->N - slot0 ? rows : t->N - slot0;
    const int64_t second = rows - first;

    for (int c = 0; c < t->ncols; c++) {
        const size_t rb = (size_t)t->T * (size_t)t->elem_bytes[c];
        uint8_t* base = t->residency == GEAR_HOST_PINNED ? t->col_host[c] : t->col_dev[c];
        const uint8_t* src = static_cast<const uint8_t*>(col_src[c]) + (size_t)skip * rb;
        hipError_t e = hipMemcpyAsync(base + (size_t)slot0 * rb, src, (size_t)first * rb, hipMemcpyDefault, s);
        if (e == hipSuccess && second > 0)
            e = hipMemcpyAsync(base, src + (size_t)first * rb, (size_t)second * rb, hipMemcpyDefault, s);
        if (e != hipSuccess) return hip_fail(e, "gear_insert: column copy");
    }
    const uint32_t* psrc = priorities + skip;
    hipError_t e = hipMemcpyAsync(t->priority + slot0, psrc, sizeof(uint32_t) * first, hipMemcpyDefault, s);
    if (e == hipSuccess && second > 0)
        e = hipMemcpyAsync(t->priority, psrc + first, sizeof(uint32_t) * second, hipMemcpyDefault, s);
    if (e != hipSuccess) return hip_fail(e, "gear_insert: priority copy");
    t->next_seq += (uint64_t)n;
    t->cdf_dirty = true;
    return GEAR_OK;
}

extern "C" int gear_table_set_options(gear_table* h, uint32_t options) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_table_set_options: table is NULL");
    if (options & ~(GEAR_OPT_INCREMENTAL_TREE | GEAR_OPT_IS_GLOBAL_MIN | GEAR_OPT_GATHER_SHARE_CU))
        return fail(GEAR_E_INVAL, "gear_table_set_options: unknown option bits");
    Table* t = reinterpret_cast<Table*>(h);
    // Chunk minima are exact only right after a scan: switching the global
    // normalisation on forces the next prioritized select to rescan.
    if ((options & GEAR_OPT_IS_GLOBAL_MIN) && !(t->options & GEAR_OPT_IS_GLOBAL_MIN)) t->cdf_dirty = true;
    t->options = options;
    return GEAR_OK;
}

extern "C" int gear_table_sync(gear_table* h, void* stream, int32_t* device_status) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_table_sync: table is NULL");
    Table* t = reinterpret_cast<Table*>(h);
    gear::DeviceGuard guard(t->device);
    if (guard.error() != hipSuccess) return hip_fail(guard.error(), "gear_table_sync: hipSetDevice");
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint32_t st = 0;
    hipError_t e = hipMemcpyAsync(&st, t->status, sizeof(uint32_t), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemsetAsync(t->status, 0, sizeof(uint32_t), s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "gear_table_sync");
    if (device_status) *device_status = (int32_t)st;
    return GEAR_OK;
}

extern "C" int gear_table_info(const gear_table* h, int64_t* count, uint64_t* next_seq) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_table_info: table is NULL");
    const Table* t = reinterpret_cast<const Table*>(h);
    if (count) *count = gear::live_count(*t);
    if (next_seq) *next_seq = t->next_seq;
    return GEAR_OK;
}

extern "C" int gear_table_column(const gear_table* h, int32_t c, void** base, void** host_ptr,
                                 int64_t* elem_bytes) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_table_column: table is NULL");
    const Table* t = reinterpret_cast<const Table*>(h);
    if (c < 0 || c >= t->ncols) return fail(GEAR_E_INVAL, "gear_table_column: no such column");
    if (base) *base = t->col_dev[c];
    if (host_ptr) *host_ptr = t->col_host[c];
    if (elem_bytes) *elem_bytes = t->elem_bytes[c];
    return GEAR_OK;
}

extern "C" int gear_table_column_info(const gear_table* h, int32_t c, const char** name, int32_t* dtype,
                                      int32_t* elems_per_step) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_table_column_info: table is NULL");
    const Table* t = reinterpret_cast<const Table*>(h);
    if (c < 0 || c >= t->ncols) return fail(GEAR_E_INVAL, "gear_table_column_info: no such column");
    if (name) *name = t->col_name[c].c_str();
    if (dtype) *dtype = t->col_dtype[c];
    if (elems_per_step) *elems_per_step = t->col_elems[c];
    return GEAR_OK;
}

extern "C" int gear_table_find_column(const gear_table* h, const char* name, int32_t* c) {
    if (c != nullptr) *c = -1;
    if (h == nullptr || name == nullptr || c == nullptr) return fail(GEAR_E_INVAL, "gear_table_find_column: NULL argument");
    const Table* t = reinterpret_cast<const Table*>(h);
    for (int j = 0; j < t->ncols; j++)
        if (t->col_name[j] == name) {
            *c = j;
            return GEAR_OK;
        }
    return fail(GEAR_E_INVAL, std::string("gear_table_find_column: no column called ") + name);
}

extern "C" int gear_table_priorities(const gear_table* h, uint32_t** d_priority) {
    if (h == nullptr || d_priority == nullptr) return fail(GEAR_E_INVAL, "gear_table_priorities: NULL argument");
    *d_priority = reinterpret_cast<const Table*>(h)->priority;
    return GEAR_OK;
}

extern "C" const char* gear_last_error(void) {
    return gear::g_last_error.c_str();
}
