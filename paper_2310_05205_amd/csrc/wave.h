// Device helpers shared by the selection kernels: the splitmix64 draw,
// the bounding map, and wave-level DPP scans.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gear.h"

namespace gear {

// splitmix64 (Steele, Lea & Flood, OOPSLA 2014): output c of the stream
// seeded with `seed` is the finaliser applied to seed + (c+1)*gamma.
__device__ __forceinline__ uint64_t splitmix64_out(uint64_t seed, uint64_t c) {
    uint64_t z = seed + (c + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// floor(u * n / 2^64): the high word of the 128-bit product.
__device__ __forceinline__ uint64_t scale_draw(uint64_t u, uint64_t n) { return __umul64hi(u, n); }

// Draw b of a FIFO, LIFO or uniform selection (Sec. 3.3): a slot from
// index arithmetic on the ring of live slots (or on the commit order of a
// table with an index manager, when `order` is not NULL), and a window start
// drawn from splitmix64 output 2b + 1.  gear_select's kernel and the gather
// that selects its own windows both call these, so the two agree bit for bit.
struct SimpleDraws {
    int32_t strategy;       // GEAR_FIFO, GEAR_LIFO or GEAR_UNIFORM
    int64_t N;              // capacity
    int64_t live;           // live count (>= 1)
    int64_t oldest;         // ring (or commit-order) position of the oldest live entry
    int64_t newest;         // ... and of the newest
    const int32_t* order;   // commit order [N] of a managed table, else NULL
    uint64_t span;          // T - L + 1 window starts
    uint64_t seed;
};

__device__ __forceinline__ int64_t simple_slot(const SimpleDraws& d, int64_t b) {
    int64_t i;
    if (d.strategy == GEAR_FIFO) {
        i = d.oldest + b;
        if (i >= d.N) i -= d.N;
    } else if (d.strategy == GEAR_LIFO) {
        i = d.newest - b;
        if (i < 0) i += d.N;
    } else {
        i = (int64_t)scale_draw(splitmix64_out(d.seed, 2 * (uint64_t)b), (uint64_t)d.live);
        if (d.order) {
            i += d.oldest;
            if (i >= d.N) i -= d.N;
        }
    }
    return d.order ? (int64_t)d.order[i] : i;
}

__device__ __forceinline__ int32_t simple_start(const SimpleDraws& d, int64_t b) {
    return (int32_t)scale_draw(splitmix64_out(d.seed, 2 * (uint64_t)b + 1), d.span);
}

// Wave-level scans with DPP (gfx9 data-parallel primitives, all 64 lanes
// active): row shifts by 1, 2, 4, 8 scan each row of 16 lanes, then the
// row broadcasts of lanes 15 and 31 carry row totals forward.  A lane whose
// DPP source is outside its row receives 0.  64-bit values move as two
// 32-bit halves.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, CTRL, ROW_MASK, 0xf, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), CTRL, ROW_MASK, 0xf, false);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_inclusive_scan(uint64_t v) {
    v += dpp_u64<0x111, 0xf>(v);  // row_shr:1
    v += dpp_u64<0x112, 0xf>(v);  // row_shr:2
    v += dpp_u64<0x114, 0xf>(v);  // row_shr:4
    v += dpp_u64<0x118, 0xf>(v);  // row_shr:8
    v += dpp_u64<0x142, 0xa>(v);  // row_bcast:15 into rows 1 and 3
    v += dpp_u64<0x143, 0xc>(v);  // row_bcast:31 into rows 2 and 3
    return v;
}

// The same scan on 32-bit values.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp32(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROW_MASK, 0xf, false);
}

__device__ __forceinline__ uint32_t wave_inclusive_scan32(uint32_t v) {
    v += dpp32<0x111, 0xf>(v);  // row_shr:1
    v += dpp32<0x112, 0xf>(v);  // row_shr:2
    v += dpp32<0x114, 0xf>(v);  // row_shr:4
    v += dpp32<0x118, 0xf>(v);  // row_shr:8
    v += dpp32<0x142, 0xa>(v);  // row_bcast:15 into rows 1 and 3
    v += dpp32<0x143, 0xc>(v);  // row_bcast:31 into rows 2 and 3
    return v;
}

// Value of v in lane `src` (src is the same in every lane).
__device__ __forceinline__ uint64_t read_lane(uint64_t v, int src) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, src);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), src);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_sum(uint64_t v) { return read_lane(wave_inclusive_scan(v), 63); }

__device__ __forceinline__ uint64_t pick4(uint64_t a, uint64_t b, uint64_t c, uint64_t d, int q) {
    return q == 0 ? a : (q == 1 ? b : (q == 2 ? c : d));
}

}  // namespace gear
