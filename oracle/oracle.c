/*
 * CPU oracle for the scratchpad embedding-training step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do.  It shares no code, header, table or constant with the HIP
 * path.  Plain, slow and sequential per table on purpose: every loop follows
 * the definition it cites, with fp64 accumulation and one rounding to fp32 per
 * stored value.
 *
 * Two parts:
 *   O1  uncached embedding-bag training over the full tables
 *       (Sec. II-B "Forward propagation" and "Backpropagation"; plain SGD as
 *        stated in Sec. VI, the method leaves the optimiser unchanged).
 *   O2  reference planner for the GPU scratchpad: Hit-Map query, hold set
 *       from the look-forward window, victims among unheld slots by the
 *       replacement policy (LRU, the default, or LFU or random eviction, the
 *       alternatives of Sec. VI-E), Hit-Map update (Sec. IV-C hazard windows,
 *       Sec. IV-D Algorithm 1).
 *
 * Batch layout (both parts): one mini-batch is a table-major CSR.  ids[] holds
 * table 0's row IDs first, then table 1's, ...; bag g = t*B + b spans
 * ids[bag_off[g] .. bag_off[g+1]).  Row IDs are local to their table.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_ERR_INVALID (-1)
#define ORC_ERR_CAPACITY (-3)

/* replacement policies (Sec. VI-E) */
#define ORC_POLICY_LRU 0
#define ORC_POLICY_LFU 1
#define ORC_POLICY_RANDOM 2

/* successor batches a plan may prefetch, at most */
#define ORC_MAX_PF 15

int orc_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------- O1 */

/*
 * Forward (Sec. II-B, "Forward propagation"): every bag gathers the rows its
 * IDs name and reduces them element-wise into one vector.  The reduction is a
 * sum; an empty bag yields zeros; an ID repeated inside a bag counts each time.
 * out is [T*B][D].
 */
void orc_forward(int32_t T, int32_t B, int32_t D, float *const *tables,
                 const int32_t *ids, const int32_t *bag_off, float *out)
{
    int32_t t;
#pragma omp parallel for schedule(dynamic, 1)
    for (t = 0; t < T; ++t) {
        double *acc = (double *)malloc(sizeof(double) * (size_t)D);
        for (int32_t b = 0; b < B; ++b) {
            int64_t g = (int64_t)t * B + b;
            for (int32_t d = 0; d < D; ++d) acc[d] = 0.0;
            for (int32_t j = bag_off[g]; j < bag_off[g + 1]; ++j) {
                const float *w = tables[t] + (int64_t)ids[j] * D;
                for (int32_t d = 0; d < D; ++d) acc[d] += (double)w[d];
            }
            for (int32_t d = 0; d < D; ++d) out[g * D + d] = (float)acc[d];
        }
        free(acc);
    }
}

typedef struct {
    int32_t row;
    int32_t pos;
} orc_pair;

static int orc_cmp_pair(const void *a, const void *b)
{
    const orc_pair *x = (const orc_pair *)a, *y = (const orc_pair *)b;
    if (x->row != y->row) return x->row < y->row ? -1 : 1;
    if (x->pos != y->pos) return x->pos < y->pos ? -1 : 1;
    return 0;
}

/*
 * Backward + update (Sec. II-B, "Backpropagation"): the gradient of bag g is
 * routed to every row the bag gathered; a row gathered several times (in one
 * bag or in several) receives the sum of those gradients (duplication and
 * coalescing).  The sum runs over the row's positions in ascending order.
 * The row is then overwritten with W - lr * g (plain SGD).
 * grad is [T*B][D].
 */
void orc_backward_sgd(int32_t T, int32_t B, int32_t D, float *const *tables,
                      const int32_t *ids, const int32_t *bag_off, const float *grad,
                      float lr)
{
    int32_t t;
#pragma omp parallel for schedule(dynamic, 1)
    for (t = 0; t < T; ++t) {
        int32_t j0 = bag_off[(int64_t)t * B], j1 = bag_off[(int64_t)(t + 1) * B];
        int32_t n = j1 - j0;
        if (n <= 0) continue;
        orc_pair *p = (orc_pair *)malloc(sizeof(orc_pair) * (size_t)n);
        int64_t *bag_of = (int64_t *)malloc(sizeof(int64_t) * (size_t)n);
        double *acc = (double *)malloc(sizeof(double) * (size_t)D);
        for (int32_t b = 0; b < B; ++b) {
            int64_t g = (int64_t)t * B + b;
            for (int32_t j = bag_off[g]; j < bag_off[g + 1]; ++j) bag_of[j - j0] = g;
        }
        for (int32_t j = j0; j < j1; ++j) {
            p[j - j0].row = ids[j];
            p[j - j0].pos = j;
        }
        qsort(p, (size_t)n, sizeof(orc_pair), orc_cmp_pair);
        int32_t s = 0;
        while (s < n) {
            int32_t e = s;
            for (int32_t d = 0; d < D; ++d) acc[d] = 0.0;
            while (e < n && p[e].row == p[s].row) {
                const float *gr = grad + bag_of[p[e].pos - j0] * D;
                for (int32_t d = 0; d < D; ++d) acc[d] += (double)gr[d];
                ++e;
            }
            float *w = tables[t] + (int64_t)p[s].row * D;
            for (int32_t d = 0; d < D; ++d)
                w[d] = (float)((double)w[d] - (double)lr * acc[d]);
            s = e;
        }
        free(acc);
        free(bag_of);
        free(p);
    }
}

/* One uncached training step: forward on the weights left by the previous
 * step's update (RAW-1 honoured by plain sequencing), then backward+SGD. */
void orc_train_step(int32_t T, int32_t B, int32_t D, float *const *tables,
                    const int32_t *ids, const int32_t *bag_off, const float *grad,
                    float lr, float *out_or_null)
{
    if (out_or_null) orc_forward(T, B, D, tables, ids, bag_off, out_or_null);
    orc_backward_sgd(T, B, D, tables, ids, bag_off, grad, lr);
}

/* ------------------------------------------------------------------------- O2 */

/*
 * SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
 * generators", OOPSLA 2014): the state advances by the golden-ratio gamma and
 * each output is the state passed through the variant-13 64-bit finaliser.
 * orc_splitmix64_nth returns output number n (n >= 1) of the generator
 * started from state `seed`, i.e. the finaliser applied to seed + n * gamma.
 */
uint64_t orc_splitmix64_nth(uint64_t seed, uint64_t n)
{
    uint64_t z = seed + n * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/*
 * Random-eviction priority of global slot g at plan u: a slot that never
 * held a row gets 0 (free slots are used before anything is evicted); any
 * other gets 1 + the top 24 bits of output number u * 2^31 + g + 1 of the
 * seeded SplitMix64 stream, a fresh draw for every plan.  The victims are
 * the unheld slots with the smallest (priority, slot): a uniformly random
 * choice among the occupied candidates, up to ties of the 24-bit draws,
 * which go to the lower slot.
 */
uint32_t orc_random_priority(uint64_t seed, int32_t u, int64_t g, int32_t last_use)
{
    if (last_use < 0) return 0;
    uint64_t n = ((uint64_t)(uint32_t)u << 31) + (uint64_t)g + 1;
    return 1u + (uint32_t)(orc_splitmix64_nth(seed, n) >> 40);
}

/*
 * Planner state per table t (Sec. IV-D, "GPU scratchpad design"):
 *   key_of_slot[s]  row cached in slot s, or -1 if the slot never held one;
 *   slot_of_row[r]  slot caching row r, or -1 (the Hit-Map, kept as a plain
 *                   array indexed by row);
 *   last_use[s]     index of the last plan whose current batch used slot s,
 *                   -1 for a slot that never held a row;
 *   uses[s]         plans whose current batch used slot s since its current
 *                   row was placed there (the placing plan included), 0 for a
 *                   slot that never held a row: the LFU frequency.
 */
typedef struct {
    int32_t T;
    int32_t policy;
    uint64_t seed;
    int64_t *rows, *slots, *slot_base;
    int32_t **key_of_slot, **last_use, **slot_of_row, **uses;
    int32_t u; /* plans committed so far = index of the next plan */
} orc_planner;

orc_planner *orc_planner_create(int32_t T, const int64_t *rows, const int64_t *slots,
                                int32_t policy, uint64_t seed)
{
    if (policy < ORC_POLICY_LRU || policy > ORC_POLICY_RANDOM) return NULL;
    orc_planner *p = (orc_planner *)calloc(1, sizeof(orc_planner));
    p->T = T;
    p->policy = policy;
    p->seed = seed;
    p->rows = (int64_t *)malloc(sizeof(int64_t) * T);
    p->slots = (int64_t *)malloc(sizeof(int64_t) * T);
    p->slot_base = (int64_t *)malloc(sizeof(int64_t) * (T + 1));
    p->key_of_slot = (int32_t **)malloc(sizeof(int32_t *) * T);
    p->last_use = (int32_t **)malloc(sizeof(int32_t *) * T);
    p->slot_of_row = (int32_t **)malloc(sizeof(int32_t *) * T);
    p->uses = (int32_t **)malloc(sizeof(int32_t *) * T);
    p->slot_base[0] = 0;
    for (int32_t t = 0; t < T; ++t) {
        p->rows[t] = rows[t];
        p->slots[t] = slots[t];
        p->slot_base[t + 1] = p->slot_base[t] + slots[t];
        p->key_of_slot[t] = (int32_t *)malloc(sizeof(int32_t) * slots[t]);
        p->last_use[t] = (int32_t *)malloc(sizeof(int32_t) * slots[t]);
        p->slot_of_row[t] = (int32_t *)malloc(sizeof(int32_t) * rows[t]);
        p->uses[t] = (int32_t *)calloc((size_t)slots[t], sizeof(int32_t));
        for (int64_t s = 0; s < slots[t]; ++s) p->key_of_slot[t][s] = -1, p->last_use[t][s] = -1;
        for (int64_t r = 0; r < rows[t]; ++r) p->slot_of_row[t][r] = -1;
    }
    p->u = 0;
    return p;
}

void orc_planner_destroy(orc_planner *p)
{
    if (!p) return;
    for (int32_t t = 0; t < p->T; ++t) {
        free(p->key_of_slot[t]);
        free(p->last_use[t]);
        free(p->slot_of_row[t]);
        free(p->uses[t]);
    }
    free(p->uses);
    free(p->key_of_slot);
    free(p->last_use);
    free(p->slot_of_row);
    free(p->rows);
    free(p->slots);
    free(p->slot_base);
    free(p);
}

int32_t orc_planner_step(const orc_planner *p) { return p->u; }

/* Read access to the committed state, for invariant checks. */
void orc_planner_state(const orc_planner *p, int32_t t, int32_t *key_of_slot,
                       int32_t *last_use, int32_t *slot_of_row, int32_t *uses)
{
    if (uses) memcpy(uses, p->uses[t], sizeof(int32_t) * p->slots[t]);
    if (key_of_slot) memcpy(key_of_slot, p->key_of_slot[t], sizeof(int32_t) * p->slots[t]);
    if (last_use) memcpy(last_use, p->last_use[t], sizeof(int32_t) * p->slots[t]);
    if (slot_of_row) memcpy(slot_of_row, p->slot_of_row[t], sizeof(int32_t) * p->rows[t]);
}

static int orc_cmp_i32(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/* A candidate slot and its eviction priority: smaller goes first. */
typedef struct {
    int64_t prio;
    int32_t slot;
} orc_cand;

static int orc_cmp_cand(const void *a, const void *b)
{
    const orc_cand *x = (const orc_cand *)a, *y = (const orc_cand *)b;
    if (x->prio != y->prio) return x->prio < y->prio ? -1 : 1;
    return (x->slot > y->slot) - (x->slot < y->slot);
}

/* Eviction priority of slot s of table t under the planner's policy:
 * LRU the last use (never used = -1, first), LFU the use count (never used =
 * 0, first), random the seeded draw of orc_random_priority. */
static int64_t orc_priority(const orc_planner *p, int32_t t, int64_t s)
{
    switch (p->policy) {
    case ORC_POLICY_LFU: return p->uses[t][s];
    case ORC_POLICY_RANDOM:
        return orc_random_priority(p->seed, p->u, p->slot_base[t] + s, p->last_use[t][s]);
    default: return p->last_use[t][s];
    }
}

/* Sorted unique rows of table t in one batch; returns the count. */
static int32_t orc_unique_rows(const int32_t *ids, int32_t j0, int32_t j1, int32_t *out)
{
    int32_t n = j1 - j0, m = 0;
    if (n <= 0) return 0;
    memcpy(out, ids + j0, sizeof(int32_t) * (size_t)n);
    qsort(out, (size_t)n, sizeof(int32_t), orc_cmp_i32);
    for (int32_t i = 0; i < n; ++i)
        if (i == 0 || out[i] != out[m - 1]) out[m++] = out[i];
    return m;
}

static int32_t orc_find(const int32_t *sorted, int32_t n, int32_t key)
{
    int32_t lo = 0, hi = n;
    while (lo < hi) {
        int32_t mid = lo + (hi - lo) / 2;
        if (sorted[mid] < key) lo = mid + 1; else hi = mid;
    }
    return lo;
}

/*
 * Rows of table t that a plan prefetching npf batches ahead also fills (the
 * earlier fill of future misses that Sec. IV-C's multi-stage overlap allows):
 * for each successor batch win[w], w = 1..npf in turn, its sorted unique rows
 * that are neither cached nor in an earlier batch of the window (win[0] ..
 * win[w-1]; rows of win[0] are filled as the planned batch's own misses,
 * rows of a closer successor were taken with it).  Batch by batch, each
 * ascending.  Returns the count; P needs room for the IDs of table t in
 * win[1..npf]; tmp for those of table t in win[0..npf] (each batch's sorted
 * unique rows, kept for the membership tests).
 */
static int32_t orc_prefetch_rows(const orc_planner *p, int32_t t, int32_t npf,
                                 const int32_t *const *win_ids, const int32_t *const *win_off,
                                 int32_t B, int32_t *P, int32_t *tmp)
{
    int32_t k = 0;
    int32_t start[ORC_MAX_PF + 2], len[ORC_MAX_PF + 1];
    start[0] = 0;
    for (int32_t w = 0; w <= npf; ++w) {
        const int32_t *off = win_off[w];
        len[w] = orc_unique_rows(win_ids[w], off[(int64_t)t * B], off[(int64_t)(t + 1) * B],
                                 tmp + start[w]);
        start[w + 1] = start[w] + len[w];
    }
    for (int32_t w = 1; w <= npf; ++w) {
        const int32_t *rows = tmp + start[w];
        for (int32_t i = 0; i < len[w]; ++i) {
            int32_t earlier = 0;
            for (int32_t e = 0; e < w && !earlier; ++e) {
                const int32_t at = orc_find(tmp + start[e], len[e], rows[i]);
                earlier = at < len[e] && tmp[start[e] + at] == rows[i];
            }
            if (p->slot_of_row[t][rows[i]] < 0 && !earlier) P[k++] = rows[i];
        }
    }
    return k;
}

/*
 * Held slots of table t for this plan (Sec. IV-C, "Removing RAW-4" and
 * "Putting everything together"): a slot is held when the row it caches is
 * used by any batch of the window (the batch being planned, its visible
 * successors and, when the caller passes them, earlier batches still in
 * flight: the past window).  Rows not resident hold nothing.  held[] is
 * zeroed here.
 */
static void orc_mark_held(const orc_planner *p, int32_t t, int32_t nwin,
                          const int32_t *const *win_ids, const int32_t *const *win_off,
                          int32_t B, uint8_t *held)
{
    memset(held, 0, (size_t)p->slots[t]);
    for (int32_t w = 0; w < nwin; ++w) {
        int32_t j0 = win_off[w][(int64_t)t * B], j1 = win_off[w][(int64_t)(t + 1) * B];
        for (int32_t j = j0; j < j1; ++j) {
            int32_t s = p->slot_of_row[t][win_ids[w][j]];
            if (s >= 0) held[s] = 1;
        }
    }
}

/*
 * Plan the batch win[0] with hold window win[0..nwin-1] (its look-forward
 * successors, and any past batches the caller wants held, in any order after
 * win[0]).
 *
 * For each table t (Algorithm 1, canonicalised):
 *   U      sorted unique rows of win[0] in table t; inv[j] indexes U;
 *   hit    U[i] is cached (Hit-Map query, Step C);
 *   M      the missing rows of U in ascending order;
 *   C      unheld slots (never used, or caching a row no window batch uses);
 *   V      the |M| slots of C with the smallest (priority, slot), in that
 *          order: ChooseVictim under the policy (orc_priority), ties by slot
 *          index;
 *   M[i] is placed in V[i]; V[i]'s previous row (if any) is evicted and
 *   leaves the Hit-Map; V[i]'s use count restarts at 0;
 *   every slot of U gets last_use = u and one more use; slot_of[j] = slot of
 *   ids[j].
 * If any table has |M| > |C| the plan fails with ORC_ERR_CAPACITY and no
 * state changes (the worst-case sizing of Sec. IV-D is not met).
 *
 * Prefetch (orc_planner_plan_pf with npf >= 1 successors): M is extended,
 * per table, by the rows of win[1..npf] that are neither cached nor in an
 * earlier window batch (orc_prefetch_rows: batch by batch, each ascending),
 * after the planned batch's misses; they take the next victims in the same
 * order.  A prefetched row is placed with last_use = u and no use (it is not
 * part of this plan's batch); it has no slot_of entry.  The capacity check
 * counts both kinds of misses.
 *
 * Outputs (caller allocates; capacity NNZ of win[0] unless noted, slots are
 * global = slot_base[t] + local slot):
 *   u_table,u_row [nU]   U over all tables, ascending (table, row)
 *   inv [NNZ]            index into U
 *   hit [nU]             1 = hit
 *   m_table,m_row [nM]   misses, ascending (table, row)
 *   v_slot [nM]          slot given to miss i
 *   v_old_row [nM]       row evicted from that slot, -1 if it was empty
 *   v_old_use [nM]       that slot's last_use before this plan
 *   slot_u [nU]          slot of U[i] after the plan
 *   slot_of [NNZ]        slot of ids[j] after the plan
 *   counts[3]            nU, nM, number of evictions of occupied slots
 */
static int32_t orc_batch_valid(const orc_planner *p, const int32_t *ids, const int32_t *off, int32_t B)
{
    if (off[0] != 0) return 0;
    for (int64_t g = 0; g < (int64_t)p->T * B; ++g)
        if (off[g + 1] < off[g]) return 0;
    for (int32_t t = 0; t < p->T; ++t)
        for (int32_t j = off[(int64_t)t * B]; j < off[(int64_t)(t + 1) * B]; ++j)
            if (ids[j] < 0 || ids[j] >= p->rows[t]) return 0;
    return 1;
}

static int32_t orc_plan_core(orc_planner *p, int32_t nwin, const int32_t *const *win_ids,
                             const int32_t *const *win_off, int32_t B, int32_t npf,
                             int32_t *u_table, int32_t *u_row,
                             int32_t *inv, uint8_t *hit, int32_t *m_table, int32_t *m_row,
                             int32_t *v_slot, int32_t *v_old_row, int32_t *v_old_use,
                             int32_t *slot_u, int32_t *slot_of, int64_t *counts)
{
    const int32_t T = p->T;
    const int32_t *ids = win_ids[0], *off = win_off[0];
    if (nwin < 1) return ORC_ERR_INVALID;

    /* validate every window batch before anything else */
    if (npf < 0 || npf > nwin - 1 || npf > ORC_MAX_PF) return ORC_ERR_INVALID;
    for (int32_t w = 0; w < nwin; ++w)
        if (!orc_batch_valid(p, win_ids[w], win_off[w], B)) return ORC_ERR_INVALID;

    int64_t maxS = 0;
    for (int32_t t = 0; t < T; ++t) if (p->slots[t] > maxS) maxS = p->slots[t];
    int32_t nnz = off[(int64_t)T * B];
    int32_t pf_nnz = 0;  /* IDs of the prefetched batches */
    for (int32_t w = 1; w <= npf; ++w) pf_nnz += win_off[w][(int64_t)T * B];
    int32_t *U = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nnz > 0 ? nnz : 1));
    int32_t *P = (int32_t *)malloc(sizeof(int32_t) * (size_t)(pf_nnz > 0 ? pf_nnz : 1));
    int32_t *tmp = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nnz + pf_nnz > 0 ? nnz + pf_nnz : 1));
    uint8_t *held = (uint8_t *)malloc((size_t)(maxS > 0 ? maxS : 1));
    orc_cand *cand = (orc_cand *)malloc(sizeof(orc_cand) * (size_t)(maxS > 0 ? maxS : 1));
    int32_t status = ORC_OK;

    /* pass 1: capacity check on every table, no state change */
    for (int32_t t = 0; t < T && status == ORC_OK; ++t) {
        int32_t j0 = off[(int64_t)t * B], j1 = off[(int64_t)(t + 1) * B];
        int32_t nu = orc_unique_rows(ids, j0, j1, U);
        int64_t nmiss = 0, ncand = 0;
        for (int32_t i = 0; i < nu; ++i) nmiss += p->slot_of_row[t][U[i]] < 0;
        nmiss += orc_prefetch_rows(p, t, npf, win_ids, win_off, B, P, tmp);
        orc_mark_held(p, t, nwin, win_ids, win_off, B, held);
        for (int64_t s = 0; s < p->slots[t]; ++s) ncand += !held[s];
        if (nmiss > ncand) status = ORC_ERR_CAPACITY;
    }

    /* pass 2: commit */
    int64_t nU = 0, nM = 0, nEv = 0, nPf = 0;
    for (int32_t t = 0; t < T && status == ORC_OK; ++t) {
        int32_t j0 = off[(int64_t)t * B], j1 = off[(int64_t)(t + 1) * B];
        int32_t nu = orc_unique_rows(ids, j0, j1, U);
        int64_t ubase = nU, mbase = nM;
        for (int32_t i = 0; i < nu; ++i) {
            u_table[ubase + i] = t;
            u_row[ubase + i] = U[i];
            hit[ubase + i] = p->slot_of_row[t][U[i]] >= 0;
        }
        for (int32_t j = j0; j < j1; ++j) inv[j] = (int32_t)(ubase + orc_find(U, nu, ids[j]));
        int64_t nmiss = 0;
        for (int32_t i = 0; i < nu; ++i)
            if (!hit[ubase + i]) {
                m_table[mbase + nmiss] = t;
                m_row[mbase + nmiss] = U[i];
                ++nmiss;
            }
        const int64_t nown = nmiss;  /* the planned batch's own misses come first */
        {
            int32_t nfetch = orc_prefetch_rows(p, t, npf, win_ids, win_off, B, P, tmp);
            for (int32_t i = 0; i < nfetch; ++i) {
                m_table[mbase + nmiss] = t;
                m_row[mbase + nmiss] = P[i];
                ++nmiss;
            }
            nPf += nfetch;
        }
        orc_mark_held(p, t, nwin, win_ids, win_off, B, held);
        int64_t nc = 0;
        for (int64_t s = 0; s < p->slots[t]; ++s)
            if (!held[s]) {
                cand[nc].prio = orc_priority(p, t, s);
                cand[nc].slot = (int32_t)s;
                ++nc;
            }
        qsort(cand, (size_t)nc, sizeof(orc_cand), orc_cmp_cand);
        for (int64_t i = 0; i < nmiss; ++i) {
            int32_t v = cand[i].slot;
            int32_t old = p->key_of_slot[t][v];
            v_slot[mbase + i] = (int32_t)(p->slot_base[t] + v);
            v_old_row[mbase + i] = old;
            v_old_use[mbase + i] = p->last_use[t][v];
            if (old >= 0) {
                p->slot_of_row[t][old] = -1;
                ++nEv;
            }
            p->key_of_slot[t][v] = m_row[mbase + i];
            p->slot_of_row[t][m_row[mbase + i]] = v;
            p->uses[t][v] = 0;
            if (i >= nown) p->last_use[t][v] = p->u;  /* prefetched: placed now, not used */
        }
        for (int32_t i = 0; i < nu; ++i) {
            int32_t s = p->slot_of_row[t][U[i]];
            slot_u[ubase + i] = (int32_t)(p->slot_base[t] + s);
            p->last_use[t][s] = p->u;
            p->uses[t][s] += 1;
        }
        for (int32_t j = j0; j < j1; ++j) slot_of[j] = slot_u[inv[j]];
        nU += nu;
        nM += nmiss;
    }
    if (status == ORC_OK) {
        counts[0] = nU;
        counts[1] = nM;
        counts[2] = nEv;
        counts[3] = nPf;
        p->u += 1;
    }
    free(cand);
    free(held);
    free(tmp);
    free(P);
    free(U);
    return status;
}

/* Plan without prefetch; counts[3] as described above. */
int32_t orc_planner_plan(orc_planner *p, int32_t nwin, const int32_t *const *win_ids,
                         const int32_t *const *win_off, int32_t B,
                         int32_t *u_table, int32_t *u_row, int32_t *inv, uint8_t *hit,
                         int32_t *m_table, int32_t *m_row, int32_t *v_slot,
                         int32_t *v_old_row, int32_t *v_old_use, int32_t *slot_u,
                         int32_t *slot_of, int64_t *counts)
{
    int64_t c4[4] = {0, 0, 0, 0};
    int32_t st = orc_plan_core(p, nwin, win_ids, win_off, B, 0, u_table, u_row, inv, hit,
                               m_table, m_row, v_slot, v_old_row, v_old_use, slot_u, slot_of, c4);
    if (st == ORC_OK) memcpy(counts, c4, sizeof(int64_t) * 3);
    return st;
}

/* Plan that also prefetches the first npf successors of the window (win[1..npf]
 * must be look-forward batches; past batches follow them); m_* and v_* need
 * room for the NNZ of win[0..npf] together; counts[4] = nU, nM (prefetched
 * included), evictions, prefetched rows. */
int32_t orc_planner_plan_pf(orc_planner *p, int32_t nwin, const int32_t *const *win_ids,
                            const int32_t *const *win_off, int32_t B, int32_t npf,
                            int32_t *u_table, int32_t *u_row,
                            int32_t *inv, uint8_t *hit, int32_t *m_table, int32_t *m_row,
                            int32_t *v_slot, int32_t *v_old_row, int32_t *v_old_use,
                            int32_t *slot_u, int32_t *slot_of, int64_t *counts)
{
    return orc_plan_core(p, nwin, win_ids, win_off, B, npf, u_table, u_row, inv, hit,
                         m_table, m_row, v_slot, v_old_row, v_old_use, slot_u, slot_of, counts);
}
