// Window collection on gfx950 (GEAR Sec. 3.2 storage format; Sec. 3.4).
//
// For draw b, step t < L and requested column j:
//     out_j[b][t][:] = column c_j, block idx[b], step start[b] + t
// Each window is one contiguous byte range of its column,
//     base_c + (idx[b]*T + start[b]) * E_c,  length W_c = L * E_c,
// and each column's batch [B][L][E_c] is one contiguous range, so the copy
// is driven by the output: a workgroup owns a contiguous piece of one
// column's output.  Wide columns (a window at least a piece long) are cut
// into equal pieces of the whole batch, so a piece may run from the end of
// one window into the start of the next (never further); a launch of a few
// hundred MB then runs in equal pieces instead of ending on the short last
// pieces of every window.  Narrow windows are packed several to a piece with
// their source offsets staged in LDS.  All requested columns run in one
// launch.  A column table in pinned host memory is read by the same kernel
// through its mapped address, so the loads go over the host link without a
// CPU copy.
//
// gear_select_collect runs the same kernel for FIFO, LIFO or uniform draws
// (Sec. 3.3): instead of reading idx[b] and start[b], each piece computes its
// windows' draws from the ring state and the seed, and the piece holding a
// window's first element in the first requested column writes the draw's
// slot, start and weight.  A step then needs no separate selection launch.
//
// Element width per column: 16 bytes when every window source and output
// address is 16-byte aligned, else 4 bytes when 4-byte aligned, else 1.
// Sources are aligned when the column base and the step size are, or, for
// full-trajectory windows (L = T, every start 0), the trajectory size.
#include "gear_internal.h"

namespace gear {
namespace {

constexpr int kThreads = 256;
// Elements in flight per thread (U), so a piece is kThreads * U elements.
// HBM tables: 8 (32 KiB pieces at 16-byte elements) for batches of at least
// kLargeBatch bytes, 2 (8 KiB) below.  Measured on gfx950 in one process,
// each variant alternating on the same table and buffers: the DT-shaped
// whole trajectories (51 MB) 20.6-20.7 us with 2 against 20.9-21.2 with 4
// and 21.5-22.1 with 8; 8.7 MB and 2 MB batches 4.8 and 4.5 us with 2
// against 5.5 and 5.1 with 8.  The MAT batch (278 MB) took 103.6 us with 2
// and 94.6 with 4 against 96.0 with 8 back to back, but with the next
// steps' selection running beside it on another stream, as in the replay
// loop, 4 was the slower (gather 94.1 against 92.7 us, step 97.9 against
// 97.2 over 100 steps).  Pinned host tables: 4 (8 was 4% slower over the host
// link; 2 no faster).
constexpr int kUnrollLarge = 8;
constexpr int kUnrollSmall = 2;
constexpr int64_t kLargeBatch = 128ll << 20;
constexpr int kUnrollHost = 4;
// A long gather from an HBM table (at least kCapRounds rounds of the
// workgroups that fit the device) reserves kCapLds bytes of LDS per
// workgroup that it does not use: with the kernel's own LDS that is about
// 39 KB, so at most 4 of its workgroups share a CU (160 KiB of LDS).  It
// keeps HBM as busy with 4 as with 8 (MAT batch: 92.0-93.1 us with 2, 4 or 5
// per CU, 92.6 us uncapped), and kernels of other streams find free slots:
// with the next step's selection on another stream the MAT step went from
// 103 to 99.4-99.6 us.  Shorter launches take every slot.
// GEAR_OPT_GATHER_SHARE_CU reserves kShareLds instead (about 71 KB with the
// kernel's own LDS, so 2 per CU).  Beside such a gather the MAT selection and
// update take about half as long as beside one with 4 per CU, while the
// gather takes 1-1.5 us longer: worth it only while another stream has to
// catch up, as at the start of a pipeline.
constexpr unsigned kCapLds = 32 * 1024;
constexpr unsigned kShareLds = 64 * 1024;
constexpr int64_t kCapRounds = 4;
constexpr int64_t kResidentWorkgroups = 2048;  // 256 CUs x 8 workgroups of 256 threads
constexpr int kMaxLaunchCols = 16;  // columns per launch (more take several launches)

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

struct ColTask {
    const uint8_t* src;   // device-visible column base
    uint8_t* out;         // batch output [B][W]
    int64_t E;            // bytes per step
    int64_t W;            // window bytes, L*E
    int64_t task0;        // first task (workgroup) of this column
    int64_t piece;        // bytes per piece: kThreads * unroll * width
    int64_t n;            // elements per window, W / width
    int32_t width;        // element bytes: 16, 4 or 1
    int32_t wide;         // 1: equal pieces of the batch, each within one or two windows;
                          // 0: several whole windows per piece
    int32_t wpp;          // windows per piece (narrow)
    uint32_t epw;         // elements per window (narrow)
    uint32_t magic;       // ceil(2^32 / epw) for epw > 1: exact quotient for operands < 2^16
    int32_t draws_out;    // 1: this column's pieces write the selected slots, starts and weights
};

// A gather that selects its own windows (FIFO, LIFO or uniform draws): a
// kernel argument of its own, beside CollectArgs.
struct DrawArgs {
    int32_t computed;       // 1: the windows are `draws`, computed per piece; 0: from CollectArgs::idx, start
    SimpleDraws draws;
    int64_t* idx_out;       // the draws, written by the pieces of a draws_out column
    int32_t* start_out;
    float* w_out;           // ... and weight 1 per draw, when not NULL
};

struct CollectArgs {
    ColTask col[kMaxLaunchCols];
    int32_t ncols;
    const int64_t* idx;     // the caller's draws, unless DrawArgs::computed
    const int32_t* start;
    int32_t B;
    int32_t T;
    int32_t L;
    int64_t N;
    uint32_t* status;
};

template <int WIDTH>
struct Elem;
template <>
struct Elem<16> {
    typedef u32x4 type;
};
template <>
struct Elem<4> {
    typedef uint32_t type;
};
template <>
struct Elem<1> {
    typedef uint8_t type;
};

// Table bytes are read once per collection and the batch is written once:
// loads and stores are both non-temporal.  Measured on gfx950 with the
// MAT-shaped batch (278 MB each way) and output buffers that alternate, so
// that no batch line is still cached from an earlier launch: 89.8 us with
// non-temporal stores against 94.8 us with plain ones, level with a plain
// copy of the same bytes.  Plain stores win (81 us) only when the same
// output buffer is rewritten while the last-level cache still holds it.
template <int WIDTH>
__device__ inline typename Elem<WIDTH>::type load_stream(const typename Elem<WIDTH>::type* p) {
    return __builtin_nontemporal_load(p);
}

template <int WIDTH>
__device__ inline void store_stream(typename Elem<WIDTH>::type* p, typename Elem<WIDTH>::type v) {
    __builtin_nontemporal_store(v, p);
}

template <int WIDTH>
__device__ inline typename Elem<WIDTH>::type zero_elem() {
    return typename Elem<WIDTH>::type(0);
}

// Element k (< U) of this thread within its piece of kThreads * U elements.
// Each wave owns 64 * U consecutive elements and its k-th load covers the
// k-th 64 of them, so every wave reads and writes one contiguous run instead
// of the four waves interleaving every 64 elements.  On gfx950 a 278 MB copy
// with 4 KiB per wave took 88.5-88.9 us, against 96.4-96.9 us with 32 KiB
// pieces interleaved that way.  In the gather it is worth less: the MAT
// batch with 8 elements per thread 91.1-96.0 us against 91.2-96.7
// interleaved (two machines), and no difference next to another stream's
// selection; the DT-shaped batch with 2, 20.6 against 20.9 us.
template <int U>
__device__ __forceinline__ int64_t lane_elem(int k) {
    return (int64_t)(threadIdx.x >> 6) * (64 * U) + k * 64 + (threadIdx.x & 63);
}

// Source byte offset of window b's first step; kNoWindow for index -1 (a
// draw with no trajectory: a missing TopK entry, a draw another shard
// owns), kBadWindow for an index or start out of range.  Both read as zeros.
constexpr int64_t kNoWindow = -1;
constexpr int64_t kBadWindow = -2;

__device__ __forceinline__ int64_t window_offset(const CollectArgs& a, const DrawArgs& g, const ColTask& c,
                                                 int64_t b) {
    if (g.computed) return (simple_slot(g.draws, b) * a.T + simple_start(g.draws, b)) * c.E;
    const int64_t i = a.idx[b];
    const int32_t s = a.start[b];
    if (i == -1) return kNoWindow;
    if (i < 0 || i >= a.N || s < 0 || s > a.T - a.L) return kBadWindow;
    return (i * a.T + s) * c.E;
}

// A gather that selects its own windows writes draw b's slot, start and
// weight once: from the piece of the draws_out column that holds the
// window's first element.
__device__ __forceinline__ void write_draw(const DrawArgs& g, int64_t b) {
    g.idx_out[b] = simple_slot(g.draws, b);
    g.start_out[b] = simple_start(g.draws, b);
    if (g.w_out) g.w_out[b] = 1.0f;
}

// Piece q of a wide column: output elements [q*P, q*P + m) of the column's
// batch, P = kThreads * U, m = P except in the batch's last piece.  A
// window has n >= P elements, so the piece lies in window w0 from element r0
// on and, if r0 + m > n, runs into window w0 + 1.
template <int WIDTH, int U>
__device__ void copy_wide(const CollectArgs& a, const DrawArgs& g, const ColTask& c, int64_t q) {
    typedef typename Elem<WIDTH>::type V;
    constexpr int64_t P = (int64_t)kThreads * U;
    const int64_t o0 = q * P;
    const int64_t w0 = o0 / c.n;
    const int64_t r0 = o0 - w0 * c.n;
    const int64_t total = (int64_t)a.B * c.n;
    const int64_t m = (total - o0) < P ? (total - o0) : P;
    const bool two = r0 + m > c.n;
    const int64_t so0 = window_offset(a, g, c, w0);
    const int64_t so1 = two ? window_offset(a, g, c, w0 + 1) : kNoWindow;
    if (threadIdx.x == 0 && (so0 == kBadWindow || so1 == kBadWindow)) atomicOr(a.status, GEAR_STATUS_BAD_INDEX);
    if (c.draws_out && threadIdx.x == 0) {  // a piece holds at most one window's first element
        if (r0 == 0) write_draw(g, w0);
        else if (two) write_draw(g, w0 + 1);
    }
    const V* src = reinterpret_cast<const V*>(c.src);
    V* dst = reinterpret_cast<V*>(c.out) + o0;
    // Element offsets of the two windows' sources, shifted so that element
    // r of the piece (r = r0 + e) reads base + r in either window.
    const int64_t b0 = so0 / WIDTH, b1 = so1 / WIDTH - c.n;
    V v[U];
    if (m == P && so0 >= 0 && (!two || so1 >= 0)) {
        // Every element valid: the loads go out unconditionally, all in flight.
#pragma unroll
        for (int k = 0; k < U; k++) {
            const int64_t r = r0 + lane_elem<U>(k);
            v[k] = load_stream<WIDTH>(src + (r < c.n ? b0 : b1) + r);
        }
#pragma unroll
        for (int k = 0; k < U; k++) store_stream<WIDTH>(dst + lane_elem<U>(k), v[k]);
        return;
    }
    // The batch's last piece, or a piece touching a missing or invalid
    // window (whose elements are zero).
#pragma unroll
    for (int k = 0; k < U; k++) {
        const int64_t e = lane_elem<U>(k);
        const int64_t r = r0 + e;
        const bool second = r >= c.n;
        v[k] = zero_elem<WIDTH>();
        if (e < m && (second ? so1 : so0) >= 0) v[k] = load_stream<WIDTH>(src + (second ? b1 : b0) + r);
    }
#pragma unroll
    for (int k = 0; k < U; k++) {
        const int64_t e = lane_elem<U>(k);
        if (e < m) store_stream<WIDTH>(dst + e, v[k]);
    }
}

template <int WIDTH, int U>
__device__ void copy_narrow(const CollectArgs& a, const DrawArgs& g, const ColTask& c, int64_t q) {
    typedef typename Elem<WIDTH>::type V;
    __shared__ int64_t s_off[kThreads];   // source element offset per window, -1 if invalid
    __shared__ int s_bad;
    const int64_t b0 = q * c.wpp;
    const int nb = (int)((a.B - b0) < c.wpp ? (a.B - b0) : c.wpp);
    if (threadIdx.x == 0) s_bad = 0;
    __syncthreads();
    if ((int)threadIdx.x < nb) {
        const int64_t so = window_offset(a, g, c, b0 + threadIdx.x);
        s_off[threadIdx.x] = so < 0 ? -1 : so / WIDTH;
        if (so == kBadWindow) s_bad = 1;
        if (c.draws_out) write_draw(g, b0 + threadIdx.x);
    }
    __syncthreads();
    if (threadIdx.x == 0 && s_bad) atomicOr(a.status, GEAR_STATUS_BAD_INDEX);
    const uint32_t total = (uint32_t)nb * c.epw;
    const V* src = reinterpret_cast<const V*>(c.src);
    V* dst = reinterpret_cast<V*>(c.out) + b0 * (int64_t)c.epw;
    V v[U];
#pragma unroll
    for (int k = 0; k < U; k++) {
        const uint32_t e = (uint32_t)lane_elem<U>(k);
        v[k] = zero_elem<WIDTH>();
        if (e < total) {
            const uint32_t w = c.epw == 1 ? e : __umulhi(e, c.magic);
            const int64_t so = s_off[w];
            if (so >= 0) v[k] = load_stream<WIDTH>(src + so + (e - w * c.epw));
        }
    }
#pragma unroll
    for (int k = 0; k < U; k++) {
        const uint32_t e = (uint32_t)lane_elem<U>(k);
        if (e < total) store_stream<WIDTH>(dst + e, v[k]);
    }
}

template <int U>
__global__ __launch_bounds__(kThreads) void collect_kernel(CollectArgs a, DrawArgs g) {
    const int64_t task = blockIdx.x;
    int j = 0;
    while (j + 1 < a.ncols && a.col[j + 1].task0 <= task) j++;
    const ColTask& c = a.col[j];
    const int64_t q = task - c.task0;
    if (c.wide) {
        if (c.width == 16) copy_wide<16, U>(a, g, c, q);
        else if (c.width == 4) copy_wide<4, U>(a, g, c, q);
        else copy_wide<1, U>(a, g, c, q);
    } else {
        if (c.width == 16) copy_narrow<16, U>(a, g, c, q);
        else if (c.width == 4) copy_narrow<4, U>(a, g, c, q);
        else copy_narrow<1, U>(a, g, c, q);
    }
}

// The collect launches over ncols requested columns (kMaxLaunchCols per
// launch).  With `draws`, the windows are those FIFO, LIFO or uniform draws,
// computed in the kernel, and the first launch's first column writes them to
// idx_out, start_out and w_out; otherwise they come from idx and start.
int launch_collect(Table* t, const int64_t* d_idx, const int32_t* d_start, const SimpleDraws* draws,
                   int64_t* idx_out, int32_t* start_out, float* w_out, int32_t B, int32_t L,
                   const int32_t* col_ids, int32_t ncols, void* const* d_out, hipStream_t s, const char* who) {
    const bool pinned = t->residency == GEAR_HOST_PINNED;
    int64_t batch_bytes = 0;
    for (int j = 0; j < ncols; j++) batch_bytes += (int64_t)B * L * t->elem_bytes[col_ids ? col_ids[j] : j];
    const int unroll = pinned ? kUnrollHost : batch_bytes >= kLargeBatch ? kUnrollLarge : kUnrollSmall;

    for (int j0 = 0; j0 < ncols; j0 += kMaxLaunchCols) {
        CollectArgs a{};
        a.idx = d_idx;
        a.start = d_start;
        DrawArgs g{};
        g.computed = draws != nullptr;
        if (draws) {
            g.draws = *draws;
            g.idx_out = idx_out;
            g.start_out = start_out;
            g.w_out = w_out;
        }
        a.B = B;
        a.T = t->T;
        a.L = L;
        a.N = t->N;
        a.status = t->status;
        a.ncols = 0;
        int64_t tasks = 0;
        // Tasks are numbered from the last requested column to the first:
        // the wide columns, listed first in the common layouts, then end
        // the launch with full pieces instead of small packed ones
        // (measured 1.6% faster on whole 68 KB trajectories).
        const int jend = ncols < j0 + kMaxLaunchCols ? ncols : j0 + kMaxLaunchCols;
        for (int j = jend - 1; j >= j0; j--) {
            const int c = col_ids ? col_ids[j] : j;
            ColTask& ct = a.col[a.ncols++];
            ct.src = t->col_dev[c];
            ct.out = static_cast<uint8_t*>(d_out[j]);
            ct.E = t->elem_bytes[c];
            ct.W = (int64_t)L * ct.E;
            ct.draws_out = draws != nullptr && j == 0;
            const uintptr_t sa = reinterpret_cast<uintptr_t>(ct.src), oa = reinterpret_cast<uintptr_t>(ct.out);
            // Window sources lie E bytes apart, or T*E when L = T (every
            // window then starts at step 0); outputs lie W bytes apart.
            const int64_t stride = L == t->T ? (int64_t)t->T * ct.E : ct.E;
            if (stride % 16 == 0 && ct.W % 16 == 0 && sa % 16 == 0 && oa % 16 == 0) ct.width = 16;
            else if (stride % 4 == 0 && ct.W % 4 == 0 && sa % 4 == 0 && oa % 4 == 0) ct.width = 4;
            else ct.width = 1;
            ct.piece = (int64_t)kThreads * unroll * ct.width;
            ct.n = ct.W / ct.width;
            ct.task0 = tasks;
            if (ct.W >= ct.piece) {
                ct.wide = 1;
                ct.wpp = 1;
                ct.epw = 0;
                ct.magic = 0;
                tasks += ((int64_t)B * ct.n + kThreads * unroll - 1) / (kThreads * unroll);
            } else {
                ct.wide = 0;
                int64_t wpp = ct.piece / ct.W;
                if (wpp > kThreads) wpp = kThreads;
                ct.wpp = (int32_t)wpp;
                ct.epw = (uint32_t)(ct.W / ct.width);
                ct.magic = ct.epw > 1 ? (uint32_t)(((1ull << 32) + ct.epw - 1) / ct.epw) : 0u;
                tasks += (B + wpp - 1) / wpp;
            }
        }
        if (tasks > 0x7FFFFFFF) return fail(GEAR_E_INVAL, std::string(who) + ": batch too large for one launch");
        const unsigned cap = (t->options & GEAR_OPT_GATHER_SHARE_CU) ? kShareLds : kCapLds;
        const unsigned lds = !pinned && tasks >= kCapRounds * kResidentWorkgroups ? cap : 0u;
        if (unroll == kUnrollLarge)
            hipLaunchKernelGGL(collect_kernel<kUnrollLarge>, dim3((unsigned)tasks), dim3(kThreads), lds, s, a, g);
        else if (unroll == kUnrollHost)
            hipLaunchKernelGGL(collect_kernel<kUnrollHost>, dim3((unsigned)tasks), dim3(kThreads), lds, s, a, g);
        else
            hipLaunchKernelGGL(collect_kernel<kUnrollSmall>, dim3((unsigned)tasks), dim3(kThreads), lds, s, a, g);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(e, (std::string(who) + ": launch").c_str());
    }
    return GEAR_OK;
}

// Argument checks shared by gear_collect and gear_select_collect.
int check_columns(const Table* t, const int32_t* col_ids, int32_t ncols, void* const* d_out, const char* who) {
    if (d_out == nullptr) return fail(GEAR_E_INVAL, std::string(who) + ": NULL pointer argument");
    if (col_ids == nullptr && ncols != t->ncols)
        return fail(GEAR_E_INVAL, std::string(who) + ": ncols must equal the table's column count when col_ids is NULL");
    if (ncols < 1 || ncols > GEAR_MAX_COLUMNS) return fail(GEAR_E_INVAL, std::string(who) + ": ncols out of range");
    for (int j = 0; j < ncols; j++) {
        const int c = col_ids ? col_ids[j] : j;
        if (c < 0 || c >= t->ncols) return fail(GEAR_E_INVAL, std::string(who) + ": no such column");
        if (d_out[j] == nullptr) return fail(GEAR_E_INVAL, std::string(who) + ": output pointer is NULL");
    }
    return GEAR_OK;
}

}  // namespace
}  // namespace gear

using gear::fail;
using gear::hip_fail;

extern "C" int gear_collect(gear_table* h, const int64_t* d_idx, const int32_t* d_start, int32_t B, int32_t L,
                            const int32_t* col_ids, int32_t ncols, void* const* d_out, void* stream) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_collect: table is NULL");
    gear::Table* t = reinterpret_cast<gear::Table*>(h);
    if (B < 1 || B > GEAR_MAX_BATCH) return fail(GEAR_E_INVAL, "gear_collect: B out of range");
    if (L < 1 || L > t->T) return fail(GEAR_E_INVAL, "gear_collect: L must lie in [1, T]");
    if (d_idx == nullptr || d_start == nullptr) return fail(GEAR_E_INVAL, "gear_collect: NULL pointer argument");
    int rc = gear::check_columns(t, col_ids, ncols, d_out, "gear_collect");
    if (rc != GEAR_OK) return rc;
    gear::DeviceGuard guard(t->device);
    if (guard.error() != hipSuccess) return hip_fail(guard.error(), "gear_collect: hipSetDevice");
    return gear::launch_collect(t, d_idx, d_start, nullptr, nullptr, nullptr, nullptr, B, L, col_ids, ncols, d_out,
                                static_cast<hipStream_t>(stream), "gear_collect");
}

extern "C" int gear_select_collect(gear_table* h, int32_t strategy, int32_t B, int32_t L, uint64_t seed,
                                   int64_t* d_idx, int32_t* d_start, float* d_weights, const int32_t* col_ids,
                                   int32_t ncols, void* const* d_out, void* stream) {
    if (h == nullptr) return fail(GEAR_E_INVAL, "gear_select_collect: table is NULL");
    gear::Table* t = reinterpret_cast<gear::Table*>(h);
    if (strategy != GEAR_FIFO && strategy != GEAR_LIFO && strategy != GEAR_UNIFORM)
        return fail(GEAR_E_INVAL, "gear_select_collect: strategy must be GEAR_FIFO, GEAR_LIFO or GEAR_UNIFORM");
    if (B < 1 || B > GEAR_MAX_BATCH) return fail(GEAR_E_INVAL, "gear_select_collect: B out of range");
    if (L < 1 || L > t->T) return fail(GEAR_E_INVAL, "gear_select_collect: L must lie in [1, T]");
    if (d_idx == nullptr || d_start == nullptr)
        return fail(GEAR_E_INVAL, "gear_select_collect: NULL pointer argument");
    int rc = gear::check_columns(t, col_ids, ncols, d_out, "gear_select_collect");
    if (rc != GEAR_OK) return rc;
    const int64_t live = gear::live_count(*t);
    if (live == 0) return fail(GEAR_E_EMPTY, "gear_select_collect: nothing inserted");
    if ((strategy == GEAR_FIFO || strategy == GEAR_LIFO) && (int64_t)B > live)
        return fail(GEAR_E_INSUFFICIENT, "gear_select_collect: FIFO/LIFO batch larger than the live count");
    gear::DeviceGuard guard(t->device);
    if (guard.error() != hipSuccess) return hip_fail(guard.error(), "gear_select_collect: hipSetDevice");
    const gear::SimpleDraws d = gear::simple_draws(*t, strategy, L, seed);
    return gear::launch_collect(t, nullptr, nullptr, &d, d_idx, d_start, d_weights, B, L, col_ids, ncols, d_out,
                                static_cast<hipStream_t>(stream), "gear_select_collect");
}
