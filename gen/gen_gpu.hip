// GPU implementation of the synthetic-input generator defined in gen.c.
//
// Fills trajectory columns of large synthetic tables directly in device (or
// mapped host) memory.  Every value follows the definitions at the top of
// gen.c exactly: Philox4x32-10 words, Irwin-Hall normals in exact integer
// arithmetic, bf16 round-to-nearest-even, fp64 return-to-go sums.  It is an
// input generator only and shares nothing with the replay library.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

enum {
    GEN_BYTES = 0, GEN_NORMAL_F32 = 1, GEN_UNIFORM_F32 = 2, GEN_INT_MOD = 3,
    GEN_NORMAL_BF16 = 4, GEN_DONE_U8 = 5, GEN_RTG_F32 = 6, GEN_STAMP = 7
};

struct Stream {
    uint32_t key0, key1, k_lo, k_hi, col;
};

__device__ inline void philox_block(const Stream& s, uint32_t blk, uint32_t out[4]) {
    uint32_t c0 = blk, c1 = s.k_lo, c2 = s.k_hi, c3 = s.col;
    uint32_t k0 = s.key0, k1 = s.key1;
#pragma unroll
    for (int r = 0; r < 10; r++) {
        uint32_t hi0 = __umulhi(0xD2511F53u, c0), lo0 = 0xD2511F53u * c0;
        uint32_t hi1 = __umulhi(0xCD9E8D57u, c2), lo1 = 0xCD9E8D57u * c2;
        c0 = hi1 ^ c1 ^ k0;
        c1 = lo1;
        c2 = hi0 ^ c3 ^ k1;
        c3 = lo0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

__device__ inline uint32_t word_at(const Stream& s, uint64_t j) {
    uint32_t w[4];
    philox_block(s, (uint32_t)(j >> 2), w);
    return w[j & 3];
}

// Words 6n .. 6n+5 always span exactly two Philox blocks.
__device__ inline float normal_f32(const Stream& s, uint64_t n) {
    uint64_t j0 = 6 * n;
    uint32_t a[4], b[4];
    philox_block(s, (uint32_t)(j0 >> 2), a);
    philox_block(s, (uint32_t)(j0 >> 2) + 1u, b);
    uint32_t w[8] = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    int off = (int)(j0 & 3);
    int64_t sum = 0;
#pragma unroll
    for (int i = 0; i < 6; i++) {
        uint32_t x = w[off + i];
        sum += (int64_t)(x & 0xFFFFu) + (int64_t)(x >> 16);
    }
    return (float)(int32_t)(sum - 393210) * (1.0f / 65536.0f);
}

__device__ inline uint16_t bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ inline Stream make_stream(uint64_t seed, uint32_t col, uint64_t k) {
    Stream s;
    s.key0 = (uint32_t)seed; s.key1 = (uint32_t)(seed >> 32);
    s.k_lo = (uint32_t)k; s.k_hi = (uint32_t)(k >> 32); s.col = col;
    return s;
}

// One workgroup per row (grid-stride over rows); threads stride over the
// row's elements.  row_bytes = T*m*esz.
__global__ void gen_fill_kernel(int kind, int64_t param, int32_t m, uint64_t seed, uint32_t col,
                                int32_t T, uint64_t k0, int64_t nrows, int64_t row_bytes,
                                uint8_t* __restrict__ out) {
    for (int64_t row = blockIdx.x; row < nrows; row += gridDim.x) {
        uint64_t k = k0 + (uint64_t)row;
        uint8_t* dst = out + row * row_bytes;
        int64_t total = (int64_t)T * m;
        if (kind == GEN_RTG_F32) {
            if (threadIdx.x == 0) {
                Stream s = make_stream(seed, (uint32_t)param, k);
                double acc = 0.0;
                for (int32_t t = T - 1; t >= 0; t--) {
                    acc += (double)normal_f32(s, (uint64_t)t);
                    ((float*)dst)[t] = (float)acc;
                }
            }
            continue;
        }
        Stream s = make_stream(seed, col, k);
        if (kind == GEN_BYTES) {
            if ((row_bytes & 3) == 0) {
                for (int64_t q = threadIdx.x; q < (row_bytes >> 2); q += blockDim.x)
                    ((uint32_t*)dst)[q] = word_at(s, (uint64_t)q);
            } else {
                for (int64_t n = threadIdx.x; n < row_bytes; n += blockDim.x)
                    dst[n] = (uint8_t)(word_at(s, (uint64_t)n >> 2) >> (8 * (n & 3)));
            }
            continue;
        }
        for (int64_t n = threadIdx.x; n < total; n += blockDim.x) {
            switch (kind) {
            case GEN_NORMAL_F32:
                ((float*)dst)[n] = normal_f32(s, (uint64_t)n);
                break;
            case GEN_UNIFORM_F32:
                ((float*)dst)[n] = (float)((int32_t)(word_at(s, (uint64_t)n) >> 8) - 8388608) * (1.0f / 8388608.0f);
                break;
            case GEN_INT_MOD:
                ((int32_t*)dst)[n] = (int32_t)(uint32_t)((uint64_t)word_at(s, (uint64_t)n) % (uint64_t)param);
                break;
            case GEN_NORMAL_BF16:
                ((uint16_t*)dst)[n] = bf16_rne(normal_f32(s, (uint64_t)n));
                break;
            case GEN_DONE_U8:
                dst[n] = (uint8_t)((n / m) == T - 1);
                break;
            case GEN_STAMP:
                ((uint32_t*)dst)[2 * n] = (uint32_t)k;
                ((uint32_t*)dst)[2 * n + 1] = (uint32_t)n;
                break;
            default:
                break;
            }
        }
    }
}

}  // namespace

extern "C" int gen_fill_rows_gpu(int kind, int64_t param, int32_t m, uint64_t seed, uint32_t col,
                                 int32_t T, uint64_t k0, int64_t nrows, void* out, void* stream) {
    int esz = (kind == GEN_BYTES || kind == GEN_DONE_U8) ? 1 : (kind == GEN_NORMAL_BF16 ? 2 : (kind == GEN_STAMP ? 8 : 4));
    if (m <= 0 || T <= 0 || nrows < 0 || out == nullptr) return -1;
    if ((kind == GEN_STAMP || kind == GEN_RTG_F32) && m != 1) return -1;
    if (kind == GEN_INT_MOD && param <= 0) return -1;
    if (kind < GEN_BYTES || kind > GEN_STAMP) return -1;
    if (nrows == 0) return 0;
    int64_t row_bytes = (int64_t)T * m * esz;
    int grid = (int)(nrows < 65536 ? nrows : 65536);
    hipLaunchKernelGGL(gen_fill_kernel, dim3(grid), dim3(256), 0, (hipStream_t)stream,
                       kind, param, m, seed, col, T, k0, nrows, row_bytes, (uint8_t*)out);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}
