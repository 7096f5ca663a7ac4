/*
 * Seeded synthetic inputs for the experience-replay library and its oracle.
 *
 * This module produces INPUTS only: trajectory column contents, initial
 * priorities and the new priorities fed to updates.  It holds none of the
 * replay method's arithmetic (no prefix sums, draws of the method, searches
 * or gathers).  Its random numbers come from Philox4x32-10 (Salmon, Moraes,
 * Dror & Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011), a
 * counter-based generator different from the method's own splitmix64 draws.
 *
 * The contents of every trajectory are a pure function of
 * (seed, column id, insertion number k), so any selected trajectory can be
 * regenerated on its own.  gen_gpu.hip implements the same definitions on
 * the GPU for filling large tables; the two must agree byte for byte.
 *
 * Word stream: word j of stream (seed, col, k) is element j % 4 of
 *   philox4x32_10(counter = {j / 4, k_lo, k_hi, col}, key = {seed_lo, seed_hi}).
 *
 * Column kinds (element n = t * m + e of a trajectory with m elements/step):
 *   GEN_BYTES       uint8: byte n % 4 (little-endian) of word n / 4
 *   GEN_NORMAL_F32  fp32 ~N(0,1) (Irwin-Hall): the twelve 16-bit halves h of
 *                   words 6n..6n+5 give (sum h - 393210) / 65536, exact in fp32
 *   GEN_UNIFORM_F32 fp32 uniform on [-1, 1): ((word n >> 8) - 2^23) / 2^23
 *   GEN_INT_MOD     int32: word n mod param
 *   GEN_NORMAL_BF16 bf16: GEN_NORMAL_F32 rounded to bfloat16, nearest-even
 *   GEN_DONE_U8     uint8: 1 at the last step (t == T-1), else 0
 *   GEN_RTG_F32     fp32 return-to-go: sum over t' >= t of the GEN_NORMAL_F32
 *                   reward of column id `param`, summed in fp64 (exact: the
 *                   terms are multiples of 2^-16 bounded by 6), rounded once
 *   GEN_STAMP       8 bytes per step: uint32 k (low word of the insertion
 *                   number), then uint32 t; a marker for order/window checks
 *
 * Priority distributions (value i of stream (seed, stream, k0 + i)):
 *   GEN_PRIO_UNIFORM   a + word0 mod (b - a + 1)
 *   GEN_PRIO_PARETO    floor(U^(-1/a)) clamped to [1, b], U in (0,1] from 53 bits
 *   GEN_PRIO_LOGNORMAL round-half-even(exp(a + b*Z)) clamped to [1, c],
 *                      Z ~ N(0,1) by Box-Muller from two 53-bit uniforms
 */
#include <stdint.h>
#include <stddef.h>
#include <string.h>
#include <math.h>

enum {
    GEN_BYTES = 0, GEN_NORMAL_F32 = 1, GEN_UNIFORM_F32 = 2, GEN_INT_MOD = 3,
    GEN_NORMAL_BF16 = 4, GEN_DONE_U8 = 5, GEN_RTG_F32 = 6, GEN_STAMP = 7
};
enum { GEN_PRIO_UNIFORM = 0, GEN_PRIO_PARETO = 1, GEN_PRIO_LOGNORMAL = 2 };

void gen_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4])
{
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    int r;
    for (r = 0; r < 10; r++) {
        uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        c0 = hi1 ^ c1 ^ k0;
        c1 = lo1;
        c2 = hi0 ^ c3 ^ k1;
        c3 = lo0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Caches the last Philox block so sequential word reads cost one call per 4. */
typedef struct {
    uint32_t key[2];
    uint32_t ctr_hi[3];
    uint64_t block;
    int valid;
    uint32_t w[4];
} gen_stream;

static void stream_init(gen_stream *s, uint64_t seed, uint32_t col, uint64_t k)
{
    s->key[0] = (uint32_t)seed;
    s->key[1] = (uint32_t)(seed >> 32);
    s->ctr_hi[0] = (uint32_t)k;
    s->ctr_hi[1] = (uint32_t)(k >> 32);
    s->ctr_hi[2] = col;
    s->valid = 0;
}

static uint32_t stream_word(gen_stream *s, uint64_t j)
{
    uint64_t blk = j >> 2;
    if (!s->valid || blk != s->block) {
        uint32_t ctr[4];
        ctr[0] = (uint32_t)blk;  /* trajectories hold < 2^34 words */
        ctr[1] = s->ctr_hi[0];
        ctr[2] = s->ctr_hi[1];
        ctr[3] = s->ctr_hi[2];
        gen_philox4x32_10(ctr, s->key, s->w);
        s->block = blk;
        s->valid = 1;
    }
    return s->w[j & 3];
}

static float normal_f32(gen_stream *s, uint64_t n)
{
    int64_t sum = 0;
    int i;
    for (i = 0; i < 6; i++) {
        uint32_t w = stream_word(s, 6 * n + (uint64_t)i);
        sum += (int64_t)(w & 0xFFFFu) + (int64_t)(w >> 16);
    }
    return (float)(int32_t)(sum - 393210) * (1.0f / 65536.0f);
}

static uint16_t f32_to_bf16_rne(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

int gen_elem_size(int kind)
{
    switch (kind) {
    case GEN_BYTES: case GEN_DONE_U8: return 1;
    case GEN_NORMAL_BF16: return 2;
    case GEN_STAMP: return 8;
    default: return 4;
    }
}

/* Rows k0 .. k0+nrows-1 of one column into out[nrows][T][m * elem_size]. */
int gen_fill_rows_cpu(int kind, int64_t param, int32_t m, uint64_t seed, uint32_t col,
                      int32_t T, uint64_t k0, int64_t nrows, uint8_t *out)
{
    int64_t row;
    int esz = gen_elem_size(kind);
    int64_t row_bytes = (int64_t)T * m * esz;
    if (m <= 0 || T <= 0 || nrows < 0 || (kind == GEN_STAMP && m != 1) || (kind == GEN_RTG_F32 && m != 1))
        return -1;
    if (kind == GEN_INT_MOD && param <= 0)
        return -1;
#pragma omp parallel for schedule(dynamic, 1)
    for (row = 0; row < nrows; row++) {
        uint64_t k = k0 + (uint64_t)row;
        uint8_t *dst = out + row * row_bytes;
        gen_stream s;
        int64_t n, total = (int64_t)T * m;
        stream_init(&s, seed, (kind == GEN_RTG_F32) ? (uint32_t)param : col, k);
        switch (kind) {
        case GEN_BYTES:
            for (n = 0; n < total; n++)
                dst[n] = (uint8_t)(stream_word(&s, (uint64_t)n >> 2) >> (8 * (n & 3)));
            break;
        case GEN_NORMAL_F32:
            for (n = 0; n < total; n++) {
                float v = normal_f32(&s, (uint64_t)n);
                memcpy(dst + 4 * n, &v, 4);
            }
            break;
        case GEN_UNIFORM_F32:
            for (n = 0; n < total; n++) {
                float v = (float)((int32_t)(stream_word(&s, (uint64_t)n) >> 8) - 8388608) * (1.0f / 8388608.0f);
                memcpy(dst + 4 * n, &v, 4);
            }
            break;
        case GEN_INT_MOD:
            for (n = 0; n < total; n++) {
                int32_t v = (int32_t)(uint32_t)((uint64_t)stream_word(&s, (uint64_t)n) % (uint64_t)param);
                memcpy(dst + 4 * n, &v, 4);
            }
            break;
        case GEN_NORMAL_BF16:
            for (n = 0; n < total; n++) {
                uint16_t v = f32_to_bf16_rne(normal_f32(&s, (uint64_t)n));
                memcpy(dst + 2 * n, &v, 2);
            }
            break;
        case GEN_DONE_U8:
            for (n = 0; n < total; n++)
                dst[n] = (uint8_t)((n / m) == T - 1);
            break;
        case GEN_RTG_F32: {
            double acc = 0.0;
            int32_t t;
            for (t = T - 1; t >= 0; t--) {
                float v;
                acc += (double)normal_f32(&s, (uint64_t)t);
                v = (float)acc;
                memcpy(dst + 4 * t, &v, 4);
            }
            break;
        }
        case GEN_STAMP: {
            int32_t t;
            for (t = 0; t < T; t++) {
                uint32_t lo = (uint32_t)k, tt = (uint32_t)t;
                memcpy(dst + 8 * t, &lo, 4);
                memcpy(dst + 8 * t + 4, &tt, 4);
            }
            break;
        }
        default:
            break;
        }
    }
    return 0;
}

static double unit53_open0(gen_stream *s, uint64_t j)
{
    /* (x + 1) / 2^53 for a 53-bit x built from words j, j+1: lies in (0, 1]. */
    uint64_t x = ((uint64_t)stream_word(s, j + 1) << 32 | stream_word(s, j)) >> 11;
    return (double)(x + 1u) * (1.0 / 9007199254740992.0);
}

int gen_priorities(int dist, double a, double b, double c, uint64_t seed, uint32_t stream,
                   uint64_t k0, int64_t n, uint32_t *out)
{
    int64_t i;
    if (n < 0)
        return -1;
    for (i = 0; i < n; i++) {
        gen_stream s;
        double v;
        stream_init(&s, seed, stream, k0 + (uint64_t)i);
        switch (dist) {
        case GEN_PRIO_UNIFORM: {
            uint64_t lo = (uint64_t)a, hi = (uint64_t)b;
            out[i] = (uint32_t)(lo + (uint64_t)stream_word(&s, 0) % (hi - lo + 1u));
            break;
        }
        case GEN_PRIO_PARETO:
            v = floor(pow(unit53_open0(&s, 0), -1.0 / a));
            if (v < 1.0) v = 1.0;
            if (v > b) v = b;
            out[i] = (uint32_t)v;
            break;
        case GEN_PRIO_LOGNORMAL: {
            double u1 = unit53_open0(&s, 0), u2 = unit53_open0(&s, 2);
            double z = sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2);
            v = nearbyint(exp(a + b * z));
            if (v < 1.0) v = 1.0;
            if (v > c) v = c;
            out[i] = (uint32_t)v;
            break;
        }
        default:
            return -1;
        }
    }
    return 0;
}

/* Rows for an arbitrary list of insertion numbers ks[0..n) into
 * out[n][T][m * elem_size]: row i is the row of insertion ks[i]. */
int gen_fill_rows_list_cpu(int kind, int64_t param, int32_t m, uint64_t seed, uint32_t col,
                           int32_t T, const uint64_t *ks, int64_t n, uint8_t *out)
{
    int64_t i;
    int64_t row_bytes = (int64_t)T * m * gen_elem_size(kind);
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (i = 0; i < n; i++)
        bad |= gen_fill_rows_cpu(kind, param, m, seed, col, T, ks[i], 1, out + i * row_bytes) != 0;
    return bad ? -1 : 0;
}
