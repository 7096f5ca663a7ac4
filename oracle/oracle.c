/*
 * Plain CPU oracle for GPU-centric experience replay selection and collection
 * (GEAR, Wang et al., arXiv 2310.05205).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously-correct
 * reference that the HIP library is checked against.  Only the test suite,
 * the package smoke check and the CPU-baseline leg of the benchmark may load
 * it.  It shares no code, header, table or constant with the HIP library: the
 * two sides each implement splitmix64 from its published definition.
 *
 * Everything here is single-threaded and written as the plain definition of
 * what the method computes:
 *   - the strategies FIFO, LIFO, uniform and prioritized (weighted) replay
 *     (Sec. 1 list of selection strategies; Sec. 3.3, centralized selection
 *     supports uniform and weighted sampling; decentralized selection names
 *     FIFO as deterministic);
 *   - weighted sampling as a prefix sum over the weights followed by a binary
 *     search for each uniformly drawn number (Sec. 3.3, centralized selection);
 *   - zero priority marks an index that must never be selected (Sec. 3.2,
 *     index manager / status table);
 *   - a collected item is a range of timesteps of a subset of fields, read
 *     from column tables whose blocks hold one field of one trajectory
 *     (Sec. 3.2, shard storage format; Sec. 3.4, collection example);
 *   - insertion into a fixed-capacity store with FIFO removal of the victim
 *     (Sec. 3.2, trajectory insertion and deletion).
 *
 * Readings where the paper is silent (each is listed in the design notes):
 *   - draws are with replacement, one search per random number;
 *   - the random number for a draw is floor(u * S / 2^64) for a 64-bit
 *     counter-based splitmix64 output u (exact integer arithmetic);
 *   - the scan is inclusive and the search returns the smallest i with
 *     C_i > r (an upper bound), so zero-priority slots are never chosen;
 *   - draw b uses stream counter 2b for the index and 2b+1 for the window start;
 *   - importance-sampling weights are (n*P(i))^-beta normalised by the batch
 *     maximum, with n the live count and P(i) = p_i/S, in fp64, rounded once;
 *   - a priority update applies the batch in order, so the last occurrence of
 *     a duplicated index wins.
 *
 * Parity pins: every function below is checked by the CPU test suite against
 * values fixed independently of this file (published splitmix64 outputs,
 * numpy library routines, closed forms and brute-force enumeration).
 */
#include <stdint.h>
#include <stddef.h>
#include <string.h>
#include <math.h>
#include <stdlib.h>

/* Oracle status codes (the oracle's own; deliberately not shared). */
#define ORC_OK            0
#define ORC_INVAL        -1
#define ORC_EMPTY        -3
#define ORC_INSUFFICIENT -4
#define ORC_NO_WEIGHT    -6  /* prioritized draw with all priorities zero */

#define ORC_FIFO        0
#define ORC_LIFO        1
#define ORC_UNIFORM     2
#define ORC_PRIORITIZED 3
#define ORC_TOPK        4

/* Index manager state (see oracle_im_init). */
#define ORC_IM_FREE      0
#define ORC_IM_PENDING   1   /* allocated, being written */
#define ORC_IM_COMMITTED 2

typedef struct {
    int64_t N;             /* indices (blocks per column table) */
    int removal;           /* ORC_FIFO or ORC_LIFO */
    int64_t max_sel;       /* preset maximum of selectable indices */
    int64_t *free_q;       /* free indices, front first */
    int64_t n_free;
    int64_t *committed;    /* committed indices, oldest commit first */
    int64_t n_committed;
    int64_t n_pending;     /* allocated, not yet committed */
    uint8_t *state;        /* ORC_IM_* per index */
} orc_im;

void oracle_im_free(orc_im *m);

/* ------------------------------------------------------------------------ */
/* splitmix64 (Steele, Lea & Flood, "Fast splittable pseudorandom number     */
/* generators", OOPSLA 2014).  The generator state advances by the golden    */
/* gamma 0x9E3779B97F4A7C15 and each output is the state passed through the  */
/* finaliser below.                                                          */
/* ------------------------------------------------------------------------ */
uint64_t oracle_mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* Output number c (0-based) of the sequential splitmix64 stream whose state
 * starts at `seed`: the state after c+1 advances is seed + (c+1)*gamma. */
uint64_t oracle_draw(uint64_t seed, uint64_t c)
{
    /* c+1 additions of gamma, taken mod 2^64 in one multiplication. */
    uint64_t state = seed + (c + 1u) * 0x9E3779B97F4A7C15ull;
    return oracle_mix64(state);
}

/* floor(u * n / 2^64): maps a uniform 64-bit word onto [0, n). */
uint64_t oracle_bounded(uint64_t u, uint64_t n)
{
    unsigned __int128 prod = (unsigned __int128)u * (unsigned __int128)n;
    return (uint64_t)(prod >> 64);
}

/* ------------------------------------------------------------------------ */
/* Weighted sampling, step 1: inclusive prefix sum of the priorities         */
/* (Sec. 3.3: a prefix-sum array over the weights).  C[i] = p[0] + ... + p[i]. */
/* Returns the total S = C[n-1] (0 for n == 0).                              */
/* ------------------------------------------------------------------------ */
uint64_t oracle_prefix_sum(const uint32_t *p, int64_t n, uint64_t *C)
{
    uint64_t acc = 0;
    int64_t i;
    for (i = 0; i < n; i++) {
        acc += (uint64_t)p[i];
        C[i] = acc;
    }
    return acc;
}

/* Weighted sampling, step 2: binary search for the bin holding r
 * (Sec. 3.3).  Returns the smallest i in [0, n) with C[i] > r, or n if there
 * is none.  C must be non-decreasing.  Textbook lower/upper-bound bisection. */
int64_t oracle_upper_bound(const uint64_t *C, int64_t n, uint64_t r)
{
    int64_t lo = 0, hi = n;           /* answer lies in [lo, hi] */
    while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        if (C[mid] > r)
            hi = mid;
        else
            lo = mid + 1;
    }
    return lo;
}

/* ------------------------------------------------------------------------ */
/* TopK order (Sec. 3.3, decentralized selection: the top-K priority          */
/* trajectories): higher priority first, the lower slot first among equal     */
/* priorities.                                                               */
/* ------------------------------------------------------------------------ */
typedef struct {
    uint32_t p;
    int64_t i;
} orc_cand;

static int orc_topk_cmp(const void *a, const void *b)
{
    const orc_cand *x = (const orc_cand *)a, *y = (const orc_cand *)b;
    if (x->p != y->p)
        return x->p > y->p ? -1 : 1;
    return x->i < y->i ? -1 : (x->i > y->i ? 1 : 0);
}

/* ------------------------------------------------------------------------ */
/* Selection (Sec. 1 strategies; Sec. 3.3).                                   */
/*                                                                          */
/* State of the store: capacity N slots, `next_seq` insertions so far, the  */
/* live count n = min(next_seq, N); insertion k lives in slot k mod N, so   */
/* the live slots are always [0, n) and the oldest live insertion is        */
/* next_seq - n.                                                            */
/*                                                                          */
/* Outputs, per draw b in [0, B):                                           */
/*   idx[b]   slot of the selected trajectory                               */
/*   start[b] first timestep of the L-step window, uniform on [0, T-L]      */
/*   w[b]     importance-sampling weight (prioritized) or 1, if w != NULL   */
/* ------------------------------------------------------------------------ */
/* With an index manager (below), `order` lists the committed slots, oldest */
/* commit first, and n = norder; FIFO, LIFO and uniform then pick from that  */
/* list.  With order == NULL the ring state above applies.                   */
/* ------------------------------------------------------------------------ */
/*                                                                          */
/* IS weights normalise by the largest weight: of the batch (global_min = 0, */
/* the reading used by default), or of every live trajectory with non-zero   */
/* priority (global_min = 1, the variant of prioritized replay that divides  */
/* by the largest weight in the whole buffer).                               */
/* ------------------------------------------------------------------------ */
int oracle_select(int strategy, const uint32_t *priority, int64_t N,
                  uint64_t next_seq, const int64_t *order, int64_t norder,
                  int32_t T, int32_t B, int32_t L,
                  uint64_t seed, float beta, int global_min,
                  int64_t *idx, int32_t *start, float *w,
                  uint64_t *C_scratch /* N entries, prioritized only */)
{
    int64_t n;
    int32_t b;

    if (N <= 0 || T <= 0 || B <= 0 || L <= 0 || L > T || idx == NULL || start == NULL)
        return ORC_INVAL;
    if (strategy < ORC_FIFO || strategy > ORC_TOPK)
        return ORC_INVAL;
    if (order != NULL)
        n = norder;
    else
        n = (next_seq < (uint64_t)N) ? (int64_t)next_seq : N;
    if (n == 0)
        return ORC_EMPTY;

    if (strategy == ORC_FIFO || strategy == ORC_LIFO) {
        /* Insertion order: FIFO yields the B oldest live insertions, oldest
         * first; LIFO the B newest, newest first.  Selection never evicts. */
        if ((int64_t)B > n)
            return ORC_INSUFFICIENT;
        for (b = 0; b < B; b++) {
            if (order != NULL) {
                idx[b] = strategy == ORC_FIFO ? order[b] : order[n - 1 - b];
            } else {
                uint64_t k;   /* insertion number of the b-th selected trajectory */
                if (strategy == ORC_FIFO)
                    k = next_seq - (uint64_t)n + (uint64_t)b;
                else
                    k = next_seq - 1u - (uint64_t)b;
                idx[b] = (int64_t)(k % (uint64_t)N);
            }
        }
    } else if (strategy == ORC_UNIFORM) {
        /* Uniform over the n live trajectories: the live slots [0, n) of the
         * ring, or the committed list of an index manager. */
        for (b = 0; b < B; b++) {
            int64_t r = (int64_t)oracle_bounded(oracle_draw(seed, 2u * (uint64_t)b), (uint64_t)n);
            idx[b] = order != NULL ? order[r] : r;
        }
    } else if (strategy == ORC_TOPK) {
        /* The B highest-priority selectable slots (priority > 0), higher
         * priority first, lower slot first among equals.  Missing draws
         * (fewer than B selectable slots) get slot -1 and weight 0. */
        int64_t ncand = 0, i;
        orc_cand *cand = (orc_cand *)malloc(sizeof(orc_cand) * (size_t)(N > 0 ? N : 1));
        if (cand == NULL)
            return ORC_INVAL;
        for (i = 0; i < N; i++) {
            if (priority[i] > 0) {
                cand[ncand].p = priority[i];
                cand[ncand].i = i;
                ncand++;
            }
        }
        qsort(cand, (size_t)ncand, sizeof(orc_cand), orc_topk_cmp);
        for (b = 0; b < B; b++)
            idx[b] = (int64_t)b < ncand ? cand[b].i : -1;
        free(cand);
        if (w != NULL)
            for (b = 0; b < B; b++)
                w[b] = idx[b] >= 0 ? 1.0f : 0.0f;
        for (b = 0; b < B; b++)
            start[b] = idx[b] >= 0 ? (int32_t)oracle_bounded(oracle_draw(seed, 2u * (uint64_t)b + 1u),
                                                             (uint64_t)(T - L + 1)) : 0;
        return ncand >= (int64_t)B ? ORC_OK : ORC_NO_WEIGHT;
    } else {
        /* Weighted: prefix sum over all N priorities, then one upper-bound
         * search per uniform number r in [0, S). */
        uint64_t S;
        if (C_scratch == NULL)
            return ORC_INVAL;
        S = oracle_prefix_sum(priority, N, C_scratch);
        if (S == 0)
            return ORC_NO_WEIGHT;
        for (b = 0; b < B; b++) {
            uint64_t r = oracle_bounded(oracle_draw(seed, 2u * (uint64_t)b), S);
            idx[b] = oracle_upper_bound(C_scratch, N, r);
        }
        if (w != NULL) {
            /* x_b = n * P(idx_b) with P(i) = p_i / S; w'_b = x_b^-beta;
             * w_b = w'_b / max of w' over the batch, or over every slot
             * with non-zero priority (every such slot is live). */
            double wmax = 0.0;
            if (global_min) {
                int64_t i;
                for (i = 0; i < N; i++) {
                    if (priority[i] > 0) {
                        double x = (double)n * (double)priority[i] / (double)S;
                        double v = pow(x, -(double)beta);
                        if (v > wmax)
                            wmax = v;
                    }
                }
            } else {
                for (b = 0; b < B; b++) {
                    double x = (double)n * (double)priority[idx[b]] / (double)S;
                    double v = pow(x, -(double)beta);
                    if (v > wmax)
                        wmax = v;
                }
            }
            for (b = 0; b < B; b++) {
                double x = (double)n * (double)priority[idx[b]] / (double)S;
                double v = pow(x, -(double)beta);
                w[b] = (float)(v / wmax);
            }
        }
    }

    /* Window start for every strategy: uniform over [0, T-L]. */
    for (b = 0; b < B; b++)
        start[b] = (int32_t)oracle_bounded(oracle_draw(seed, 2u * (uint64_t)b + 1u),
                                           (uint64_t)(T - L + 1));
    if (w != NULL && strategy != ORC_PRIORITIZED)
        for (b = 0; b < B; b++)
            w[b] = 1.0f;
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Collection (Sec. 3.2 storage format; Sec. 3.4 collection example).        */
/* Column c is an array of N blocks; a block is T steps of elem_bytes[c]     */
/* bytes.  For each draw b and step t < L:                                   */
/*   out[c][b][t] = column c, block idx[b], step start[b] + t                */
/* Output per column is contiguous [B][L][elem_bytes[c]].                    */
/* Index -1 marks a draw with no trajectory (a missing TopK entry, a draw    */
/* owned by another shard): its window is all zeros.  Returns ORC_INVAL on   */
/* any other out-of-range index, or an out-of-range start.                   */
/* ------------------------------------------------------------------------ */
int oracle_collect(int32_t ncols, const uint8_t *const *col_base, const int64_t *elem_bytes,
                   int64_t N, int32_t T, const int64_t *idx, const int32_t *start,
                   int32_t B, int32_t L, uint8_t *const *out)
{
    int32_t c, b, t;
    if (ncols <= 0 || B <= 0 || L <= 0 || L > T)
        return ORC_INVAL;
    for (b = 0; b < B; b++)
        if (idx[b] != -1 && (idx[b] < 0 || idx[b] >= N || start[b] < 0 || start[b] > T - L))
            return ORC_INVAL;
    for (c = 0; c < ncols; c++) {
        int64_t E = elem_bytes[c];
        for (b = 0; b < B; b++) {
            if (idx[b] == -1) {
                memset(out[c] + (int64_t)b * L * E, 0, (size_t)(L * E));
                continue;
            }
            for (t = 0; t < L; t++) {
                const uint8_t *src = col_base[c] + ((idx[b] * (int64_t)T) + start[b] + t) * E;
                uint8_t *dst = out[c] + (((int64_t)b * L) + t) * E;
                memcpy(dst, src, (size_t)E);
            }
        }
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Priority update (Sec. 3.2: the status table holds the priorities;       */
/* changes are gathered, then applied).  Applied in batch order, so the     */
/* last write to a slot wins.  Indices must lie in [0, N).                  */
/* ------------------------------------------------------------------------ */
int oracle_update(uint32_t *priority, int64_t N, const int64_t *idx, const uint32_t *newp, int32_t B)
{
    int32_t b;
    if (B < 0)
        return ORC_INVAL;
    for (b = 0; b < B; b++)
        if (idx[b] < 0 || idx[b] >= N)
            return ORC_INVAL;
    for (b = 0; b < B; b++)
        priority[idx[b]] = newp[b];
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Insertion with FIFO removal (Sec. 3.2, insertion and deletion): the       */
/* store holds at most N trajectories; insertion k overwrites slot k mod N,  */
/* i.e. the oldest trajectory is the victim once the store is full.          */
/* src[c] holds n blocks of T*elem_bytes[c] bytes; prio holds n priorities.  */
/* Rows are written one after another, so when n > N the last N survive.     */
/* Returns the new insertion count.                                          */
/* ------------------------------------------------------------------------ */
uint64_t oracle_insert(int32_t ncols, uint8_t *const *col_base, const int64_t *elem_bytes,
                       int64_t N, int32_t T, uint64_t next_seq, int64_t n,
                       const uint8_t *const *src, uint32_t *priority, const uint32_t *prio)
{
    int64_t r;
    int32_t c;
    for (r = 0; r < n; r++) {
        uint64_t slot = (next_seq + (uint64_t)r) % (uint64_t)N;
        for (c = 0; c < ncols; c++) {
            int64_t block = (int64_t)T * elem_bytes[c];
            memcpy(col_base[c] + (int64_t)slot * block, src[c] + r * block, (size_t)block);
        }
        priority[slot] = prio[r];
    }
    return next_seq + (uint64_t)n;
}

/* ------------------------------------------------------------------------ */
/* Index manager (Sec. 3.2): a block allocator with one queue of free        */
/* indices (allocation dequeues, release enqueues) and a status table whose  */
/* priority is 0 for indices that are free or still being written.          */
/*                                                                          */
/* Insertion (Sec. 3.2, trajectory insertion and deletion): `allocate`      */
/* hands out free indices; the client writes the blocks of those indices in */
/* place; `commit` sets their priorities and makes them selectable.  When   */
/* an index is requested and none is free, or the number of selectable      */
/* indices has reached the preset maximum, a victim is released by the      */
/* removal strategy: FIFO releases the oldest committed index, LIFO the     */
/* newest.                                                                   */
/*                                                                          */
/* Reading: pending (allocated, uncommitted) indices count toward the        */
/* maximum, so a victim is released while committed + pending >= max_sel;   */
/* with max_sel = N this is exactly "no free index".  Pending indices are    */
/* never released.                                                           */
/*                                                                          */
/* Plain arrays and linear work: the committed list is kept oldest first    */
/* and shifted on removal; the free queue likewise.                          */
/* ------------------------------------------------------------------------ */
int oracle_im_init(orc_im *m, int64_t N, int removal, int64_t max_sel)
{
    int64_t i;
    m->free_q = NULL;
    m->committed = NULL;
    m->state = NULL;
    if (N <= 0 || (removal != ORC_FIFO && removal != ORC_LIFO) || max_sel < 1 || max_sel > N)
        return ORC_INVAL;
    m->N = N;
    m->removal = removal;
    m->max_sel = max_sel;
    m->free_q = (int64_t *)malloc(sizeof(int64_t) * (size_t)N);
    m->committed = (int64_t *)malloc(sizeof(int64_t) * (size_t)N);
    m->state = (uint8_t *)malloc((size_t)N);
    if (m->free_q == NULL || m->committed == NULL || m->state == NULL) {
        oracle_im_free(m);
        return ORC_INVAL;
    }
    for (i = 0; i < N; i++) {
        m->free_q[i] = i;            /* every index starts free, in index order */
        m->state[i] = ORC_IM_FREE;
    }
    m->n_free = N;
    m->n_committed = 0;
    m->n_pending = 0;
    return ORC_OK;
}

void oracle_im_free(orc_im *m)
{
    free(m->free_q);
    free(m->committed);
    free(m->state);
    m->free_q = NULL;
    m->committed = NULL;
    m->state = NULL;
}

/* Release one victim by the removal strategy: its priority becomes 0 and
 * the index joins the back of the free queue. */
static void orc_im_release_victim(orc_im *m, uint32_t *priority)
{
    int64_t v, k;
    if (m->removal == ORC_FIFO) {
        v = m->committed[0];
        for (k = 1; k < m->n_committed; k++)
            m->committed[k - 1] = m->committed[k];
    } else {
        v = m->committed[m->n_committed - 1];
    }
    m->n_committed--;
    m->state[v] = ORC_IM_FREE;
    priority[v] = 0;
    m->free_q[m->n_free++] = v;
}

/* Allocate n indices into idx_out, releasing victims as needed.  Fails
 * with ORC_INSUFFICIENT, changing nothing, when the pending indices alone
 * would exceed the maximum. */
int oracle_im_allocate(orc_im *m, int64_t n, int64_t *idx_out, uint32_t *priority)
{
    int64_t r, k;
    if (n < 0)
        return ORC_INVAL;
    if (m->n_pending + n > m->max_sel)
        return ORC_INSUFFICIENT;
    for (r = 0; r < n; r++) {
        while (m->n_free == 0 || m->n_committed + m->n_pending >= m->max_sel)
            orc_im_release_victim(m, priority);
        idx_out[r] = m->free_q[0];
        for (k = 1; k < m->n_free; k++)
            m->free_q[k - 1] = m->free_q[k];
        m->n_free--;
        m->state[idx_out[r]] = ORC_IM_PENDING;
        m->n_pending++;
    }
    return ORC_OK;
}

/* Commit n pending indices, in the given order, with their priorities.
 * Every index must be pending and appear once; otherwise nothing changes. */
int oracle_im_commit(orc_im *m, int64_t n, const int64_t *idx, const uint32_t *prio, uint32_t *priority)
{
    int64_t r, q;
    if (n < 0)
        return ORC_INVAL;
    for (r = 0; r < n; r++) {
        if (idx[r] < 0 || idx[r] >= m->N || m->state[idx[r]] != ORC_IM_PENDING)
            return ORC_INVAL;
        for (q = 0; q < r; q++)
            if (idx[q] == idx[r])
                return ORC_INVAL;
    }
    for (r = 0; r < n; r++) {
        m->state[idx[r]] = ORC_IM_COMMITTED;
        m->committed[m->n_committed++] = idx[r];
        m->n_pending--;
        priority[idx[r]] = prio[r];
    }
    return ORC_OK;
}

/* Priority update under an index manager: as oracle_update, except that an
 * index that is not committed (released, or being written) keeps its zero
 * priority, so a late update never makes it selectable. */
int oracle_im_update(const orc_im *m, uint32_t *priority, const int64_t *idx, const uint32_t *newp, int32_t B)
{
    int32_t b;
    if (B < 0)
        return ORC_INVAL;
    for (b = 0; b < B; b++)
        if (idx[b] < 0 || idx[b] >= m->N)
            return ORC_INVAL;
    for (b = 0; b < B; b++)
        if (m->state[idx[b]] == ORC_IM_COMMITTED)
            priority[idx[b]] = newp[b];
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Index translation (Sec. 3.4): shards have equal capacity, so a global     */
/* index belongs to shard global / capacity at local index global mod        */
/* capacity.  Used by the multi-GPU sharding design only.                    */
/* ------------------------------------------------------------------------ */
int oracle_translate(int64_t global, int64_t capacity, int64_t *shard, int64_t *local)
{
    if (capacity <= 0 || global < 0)
        return ORC_INVAL;
    *shard = global / capacity;
    *local = global % capacity;
    return ORC_OK;
}
