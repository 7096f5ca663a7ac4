// Internal declarations of the gfx950 experience-replay library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "gear.h"
#include "wave.h"

namespace gear {

// Priority scan geometry.  A tile is 256 priorities: one wave64, four per
// lane, one 16-byte load per lane.  A chunk (one workgroup of the scan) is
// 32 tiles.  Selection walks a 256-ary sum tree: level 0 holds the sum of
// every tile, level l the sum of every 256^l tiles; the top level has at most
// 256 nodes.
constexpr int kTile = 256;
constexpr int kTilesPerChunk = 32;
constexpr int kFanout = 256;
constexpr int kMaxLevels = 6;
// The search runs at most this many workgroups; each leaves the smallest
// priority its draws selected in one slot of Table::wg_min.
constexpr int kSearchMaxGrid = 2048;
constexpr int64_t kSmallN = GEAR_SMALL_SELECT_MAX_N;  // tables this small select in one launch (prefix in LDS)
constexpr int32_t kSmallMaxB = GEAR_SMALL_SELECT_MAX_B;  // ... for batches up to this size
// TopK: at most this many workgroups per digit pass.
constexpr int kTopkMaxGrid = 256;
constexpr int kTopkBins = 4096;       // bins of one TopK digit pass (12-bit digits)
constexpr int kTopkStateWords = 32;   // TopK selection states after 0 .. 3 digit passes
constexpr int kTopkMaxK = GEAR_MAX_TOPK;
// Host index and priority lists (row writes, allocation, commits) are
// handled in chunks of kStageRows entries, through a ring of kStageSlots
// pinned, mapped slots that kernels read in place (a slot is refilled only
// after its last reader has run).
constexpr int64_t kStageRows = 1 << 16;
constexpr int kStageSlots = 4;
constexpr int64_t kStageSlotBytes = kStageRows * (int64_t)(sizeof(int64_t) + sizeof(uint32_t));

// Per-slot state of the index manager (host side).
enum : uint8_t { kSlotFree = 0, kSlotPending = 1, kSlotCommitted = 2, kSlotMark = 3 };

struct Table {
    int device = 0;
    int residency = GEAR_DEVICE;
    int64_t N = 0;
    int32_t T = 0;
    int32_t ncols = 0;
    std::vector<int64_t> elem_bytes;
    std::vector<std::string> col_name;  // column names ("c<index>" for byte columns)
    std::vector<int32_t> col_dtype;     // GEAR_DTYPE_* per column
    std::vector<int32_t> col_elems;     // elements per step per column
    std::vector<uint8_t*> col_dev;    // device-visible base of each column
    std::vector<uint8_t*> col_host;   // host base (pinned tables), else null

    uint64_t next_seq = 0;            // insertions so far (host-side ring state)

    uint32_t* priority = nullptr;     // [N]
    uint32_t* tag = nullptr;          // [N] scatter winner tags, kept zero between calls

    // Scan / search state.
    int64_t ntiles = 0, nchunks = 0;
    int nlevels = 0;                  // levels of the sum tree (level 0 = per tile)
    int64_t level_size[kMaxLevels] = {};
    uint64_t* tile_sums = nullptr;    // level 0, rewritten by every scan
    uint64_t* upper[2][kMaxLevels] = {};  // levels >= 1, two copies: a scan adds into
                                      // one and zeroes the other for the next scan
    int tree_parity = 0;              // copy filled by the last scan
    uint32_t* wg_min = nullptr;       // [kSearchMaxGrid] per-workgroup minimum selected priority
    uint32_t* chunk_min = nullptr;    // [nchunks] smallest non-zero priority of each scan chunk
    uint32_t* status = nullptr;       // device status word
    bool cdf_dirty = true;            // the tree does not reflect the priorities
    uint32_t options = 0;             // GEAR_OPT_* bits

    // TopK scratch (fixed sizes).
    uint32_t* topk_hist = nullptr;    // [3][kTopkBins] digit histograms, zero between calls
    uint32_t* topk_state = nullptr;   // [kTopkStateWords] selection states after 0 .. 3 digit passes
    uint32_t* topk_local = nullptr;   // [3][kTopkMaxGrid][kTopkBins] per-workgroup suffix sums of each digit pass
    // Index manager (allocate / commit insertion), off for ring tables.  The
    // host keeps the free-index queue, every slot's state and the committed
    // slots in commit order (a ring: ord_head is the oldest); the device
    // keeps the same commit-order ring and a committed flag per slot.
    bool managed = false;
    int32_t removal = GEAR_FIFO;
    int64_t max_selectable = 0;
    std::vector<int32_t> free_q;      // ring [N], front at fq_head
    int64_t fq_head = 0, n_free = 0;
    std::vector<uint8_t> slot_state;  // kSlot* per slot
    std::vector<int32_t> order_h;     // ring [N] of committed slots, oldest at ord_head
    int64_t ord_head = 0, n_committed = 0, n_pending = 0;
    int32_t* order = nullptr;         // device copy of order_h (same positions)
    uint8_t* committed = nullptr;     // device [N]: 1 for committed slots
    // Staging of host index and priority lists (every table): a ring of
    // pinned, mapped, coherent host slots that kernels read directly (small
    // host-to-device copies left the GPU idle for about 25 us each), and an
    // HBM copy of a slot list for the row scatter, which reads it once per
    // workgroup.
    int64_t* stage_idx = nullptr;     // device [kStageRows]
    uint8_t* pin_host = nullptr;      // [kStageSlots][kStageSlotBytes]: int64 indices, then uint32 priorities
    uint8_t* pin_dev = nullptr;       // the same ring's device address
    hipEvent_t pin_free[kStageSlots] = {};  // recorded after the last kernel that reads each slot
    int pin_next = 0;                 // slot the next chunk uses

    uint64_t* topk_keys = nullptr;    // [kTopkMaxK] selected keys (p << 32 | ~slot), equal priorities in slot order
};

// Thread-local error reporting.
int fail(int code, const std::string& msg);
int hip_fail(hipError_t e, const char* what);

// Allocation failures on demand, for tests of the cleanup paths: with
// GEAR_TEST_FAIL_ALLOC=n (n >= 1) in the environment, the n-th allocation
// made through one hook fails as if memory were exhausted.  Each
// gear_table_create and gear_table_use_allocator call counts its own
// allocations.  Without the variable nothing fails.
class AllocHook {
  public:
    AllocHook();
    // True when the next allocation is to fail.
    bool fail_next() { return ++count_ == fail_at_; }

  private:
    long fail_at_ = 0;
    long count_ = 0;
};

// Makes the table's device current for the lifetime of the guard.
class DeviceGuard {
  public:
    explicit DeviceGuard(int dev);
    ~DeviceGuard();
    hipError_t error() const { return err_; }

  private:
    int prev_ = -1;
    hipError_t err_ = hipSuccess;
};

// Kernel launchers (each returns hipSuccess or the launch error).
hipError_t launch_scan(Table& t, hipStream_t s);
// With shard_totals (device uint64[G]), the table is shard g of G: draws are
// numbers over the sum of all totals, and only those in this shard's range
// are resolved (slot + base); the rest get slot -1.
hipError_t launch_search(Table& t, int32_t B, int32_t L, uint64_t seed, bool want_min,
                         int64_t* idx, int32_t* start, uint32_t* sel_prio, int* grid_out, hipStream_t s,
                         const uint64_t* shard_totals = nullptr, int G = 1, int g = 0, int64_t base = 0);
hipError_t launch_is_weights(Table& t, int32_t B, float beta, int search_grid, float* w, hipStream_t s,
                             bool global_min = false);
hipError_t launch_topk(Table& t, int32_t K, int32_t L, uint64_t seed, int64_t* idx, int32_t* start, float* w,
                       hipStream_t s);
hipError_t launch_simple_select(Table& t, int32_t strategy, int32_t B, int32_t L, uint64_t seed,
                                int64_t* idx, int32_t* start, float* w, hipStream_t s);
// The arguments of FIFO, LIFO or uniform draws from the table's current ring
// (or commit-order) state; the table must have a live entry.
SimpleDraws simple_draws(const Table& t, int32_t strategy, int32_t L, uint64_t seed);
// With maintain_tree, the scatter also adds new - old of every changed
// slot into the sum tree the last scan filled.
hipError_t launch_scatter(Table& t, const int64_t* idx, const uint32_t* newp, int32_t B, bool maintain_tree,
                          hipStream_t s);
// Index manager: release the memory of a managed table's extra arrays.
void free_index_manager(Table& t);
// Managed insertion used by gear_insert: allocate n, copy the rows into the
// allocated slots, commit them with their priorities.
int managed_insert(Table& t, int64_t n, const void* const* col_src, const uint32_t* priorities, hipStream_t s);
// Writes row r of each column source into slot idx[r] (host list) in place.
int write_rows(Table& t, int64_t n, const int64_t* idx, const void* const* col_src, hipStream_t s);
// Live count of a table: committed slots (managed) or min(next_seq, N) (ring).
inline int64_t live_count(const Table& t) {
    if (t.managed) return t.n_committed;
    return t.next_seq < (uint64_t)t.N ? (int64_t)t.next_seq : t.N;
}

}  // namespace gear
