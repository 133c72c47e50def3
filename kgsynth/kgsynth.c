/*
 * kgsynth.c -- seeded synthetic knowledge-graph generator.
 *
 * This file produces input triples only.  It holds none of the sampling
 * method's arithmetic: no adjacency, no query evaluation, no random draws
 * of the sampler.  Both the CPU oracle and the GPU library consume its
 * output, which is why it lives in a module of its own.
 *
 * Recipe (documented with the configurations in kgsynth/__init__.py):
 *   candidate i (i = 0, 1, 2, ...) is a triple (h, r, t) with
 *     h = perm_h(rank_h(i)),  r = perm_r(rank_r(i)),  t = perm_t(rank_t(i))
 *   where each rank is either uniform on [0, n) or rank-Zipf(s)
 *   (P(rank k) proportional to (k+1)^-s, k = 0..n-1), sampled exactly with
 *   Walker/Vose alias tables, and each perm is a keyed Feistel bijection of
 *   [0, n) with cycle walking.  With shared_perm the head and tail
 *   permutations coincide, so in- and out-degree correlate.
 *   The graph is the first E distinct candidates in index order, skipping a
 *   candidate whose head already has deg_cap out-edges or whose tail already
 *   has deg_cap in-edges (deg_cap = 0: no cap).
 *   Random words come from SplitMix64 (Steele, Lea, Flood, OOPSLA 2014) over
 *   the counter (seed, stream, i), so the result does not depend on the
 *   number of threads.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>
#include <omp.h>
#include <stdio.h>

static inline uint64_t splitmix64(uint64_t z)
{
    z += 0x9E3779B97F4A7C15ULL;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static inline uint64_t word(uint64_t seed, uint64_t stream, uint64_t i)
{
    return splitmix64(splitmix64(seed ^ (stream * 0xD1B54A32D192ED03ULL)) + i * 0x9E3779B97F4A7C15ULL);
}

/* ---------------------------------------------------------------- Feistel */
typedef struct {
    uint64_t n;
    int half;        /* bits per half */
    uint32_t mask;
    uint64_t key[4];
} perm_t;

static void perm_init(perm_t *p, uint64_t n, uint64_t key)
{
    int bits = 2;
    while ((1ULL << bits) < n) bits++;
    if (bits & 1) bits++;
    p->n = n;
    p->half = bits / 2;
    p->mask = (uint32_t)((1ULL << p->half) - 1);
    for (int k = 0; k < 4; k++) p->key[k] = splitmix64(key + (uint64_t)k * 0x632BE59BD9B4E019ULL);
}

static inline uint64_t perm_apply(const perm_t *p, uint64_t x)
{
    do {
        uint32_t l = (uint32_t)(x >> p->half) & p->mask;
        uint32_t r = (uint32_t)x & p->mask;
        for (int k = 0; k < 4; k++) {
            uint32_t f = (uint32_t)splitmix64(p->key[k] ^ r) & p->mask;
            uint32_t nl = r;
            r = l ^ f;
            l = nl;
        }
        x = ((uint64_t)l << p->half) | r;
    } while (x >= p->n);     /* cycle walking keeps the map a bijection of [0, n) */
    return x;
}

/* ------------------------------------------------------------- alias table */
typedef struct {
    uint64_t n;
    int zipf;
    double *prob;    /* acceptance probability of column k */
    int32_t *alias;  /* alternative outcome of column k */
} dist_t;

static int dist_init(dist_t *d, uint64_t n, int zipf, double s)
{
    d->n = n;
    d->zipf = zipf;
    d->prob = NULL;
    d->alias = NULL;
    if (!zipf) return 0;
    d->prob = (double *)malloc(n * sizeof(double));
    d->alias = (int32_t *)malloc(n * sizeof(int32_t));
    int32_t *small = (int32_t *)malloc(n * sizeof(int32_t));
    int32_t *large = (int32_t *)malloc(n * sizeof(int32_t));
    if (!d->prob || !d->alias || !small || !large) return -1;
    /* weights, then their sum over fixed chunks combined in chunk order, so
       the table does not depend on the thread count */
    const uint64_t CH = 1u << 20;
    uint64_t nch = (n + CH - 1) / CH;
    double *part = (double *)calloc(nch, sizeof(double));
    if (!part) return -1;
#pragma omp parallel for schedule(static)
    for (uint64_t c = 0; c < nch; c++) {
        uint64_t lo = c * CH, hi = lo + CH < n ? lo + CH : n;
        double acc = 0.0;
        for (uint64_t k = hi; k-- > lo;) {
            d->prob[k] = pow((double)(k + 1), -s);
            acc += d->prob[k];
        }
        part[c] = acc;
    }
    double total = 0.0;
    for (uint64_t c = nch; c-- > 0;) total += part[c];   /* small terms first */
    free(part);
    double scale = (double)n / total;
    uint64_t ns = 0, nl = 0;
    for (uint64_t k = 0; k < n; k++) {
        d->prob[k] *= scale;
        d->alias[k] = (int32_t)k;
        if (d->prob[k] < 1.0) small[ns++] = (int32_t)k; else large[nl++] = (int32_t)k;
    }
    /* Vose's method */
    while (ns > 0 && nl > 0) {
        int32_t a = small[--ns];
        int32_t g = large[nl - 1];
        d->alias[a] = g;
        d->prob[g] = (d->prob[g] + d->prob[a]) - 1.0;
        if (d->prob[g] < 1.0) { nl--; small[ns++] = g; }
    }
    while (nl > 0) d->prob[large[--nl]] = 1.0;
    while (ns > 0) d->prob[small[--ns]] = 1.0;
    free(small);
    free(large);
    return 0;
}

static void dist_free(dist_t *d)
{
    free(d->prob);
    free(d->alias);
}

static inline uint64_t dist_sample(const dist_t *d, uint64_t u)
{
    uint64_t col = ((u >> 32) * d->n) >> 32;
    if (!d->zipf) return col;
    double coin = (double)(u & 0xFFFFFFFFULL) * (1.0 / 4294967296.0);
    return coin < d->prob[col] ? col : (uint64_t)d->alias[col];
}

/* ------------------------------------------------------------ candidates */
typedef struct {
    uint64_t seed;
    dist_t dh, dr, dt;
    const dist_t *pdt;
    perm_t ph, pr, pt;
    const perm_t *ppt;
} gen_t;

/* Candidate i as ranks.  The permutations are bijections, so two candidates
   are the same triple iff their ranks agree, and a cap on an entity's degree
   is a cap on its rank's degree: distinctness and caps are decided on ranks
   and ids are produced only for the accepted triples. */
static inline void candidate(const gen_t *g, uint64_t i, int32_t *h, int32_t *r, int32_t *t)
{
    *h = (int32_t)dist_sample(&g->dh, word(g->seed, 1, i));
    *r = (int32_t)dist_sample(&g->dr, word(g->seed, 2, i));
    *t = (int32_t)dist_sample(g->pdt, word(g->seed, 3, i));
}

static inline void to_ids(const gen_t *g, int32_t *h, int32_t *r, int32_t *t)
{
    *h = (int32_t)perm_apply(&g->ph, (uint64_t)*h);
    *r = (int32_t)perm_apply(&g->pr, (uint64_t)*r);
    *t = (int32_t)perm_apply(g->ppt, (uint64_t)*t);
}

static inline uint32_t triple_key(int32_t h, int32_t r, int32_t t)
{
    uint64_t z = splitmix64(((uint64_t)(uint32_t)h << 32) ^ (uint64_t)(uint32_t)t);
    return (uint32_t)(splitmix64(z ^ (uint64_t)(uint32_t)r) >> 32);
}

/* stable LSD radix sort of (key, idx) pairs by key, 11-bit digits */
static void radix_sort(uint32_t *key, uint32_t *idx, uint32_t *key2, uint32_t *idx2, uint64_t n, int nth)
{
    const int B = 11, NB = 1 << 11;
    uint64_t *cnt = (uint64_t *)calloc((size_t)nth * NB, sizeof(uint64_t));
    for (int shift = 0; shift < 32; shift += B) {
        memset(cnt, 0, (size_t)nth * NB * sizeof(uint64_t));
#pragma omp parallel num_threads(nth)
        {
            int tid = omp_get_thread_num();
            uint64_t lo = n * tid / nth, hi = n * (tid + 1) / nth;
            uint64_t *c = cnt + (size_t)tid * NB;
            for (uint64_t i = lo; i < hi; i++) c[(key[i] >> shift) & (NB - 1)]++;
        }
        uint64_t run = 0;
        for (int d = 0; d < NB; d++)
            for (int p = 0; p < nth; p++) {
                uint64_t c = cnt[(size_t)p * NB + d];
                cnt[(size_t)p * NB + d] = run;
                run += c;
            }
#pragma omp parallel num_threads(nth)
        {
            int tid = omp_get_thread_num();
            uint64_t lo = n * tid / nth, hi = n * (tid + 1) / nth;
            uint64_t *c = cnt + (size_t)tid * NB;
            for (uint64_t i = lo; i < hi; i++) {
                uint64_t o = c[(key[i] >> shift) & (NB - 1)]++;
                key2[o] = key[i];
                idx2[o] = idx[i];
            }
        }
        uint32_t *tk = key; key = key2; key2 = tk;
        uint32_t *ti = idx; idx = idx2; idx2 = ti;
    }
    /* 3 passes: the sorted data ended in the second buffers; copy back */
#pragma omp parallel for num_threads(nth) schedule(static)
    for (uint64_t i = 0; i < n; i++) { key2[i] = key[i]; idx2[i] = idx[i]; }
    free(cnt);
}

/*
 * Mark first occurrences: flag[i] = 1 iff candidate i's triple differs from
 * every candidate with a smaller index.  Candidates with equal keys sit next
 * to each other in ascending index order after the stable sort.
 */
static void mark_first(const gen_t *g, const uint32_t *key, const uint32_t *idx, uint64_t n,
                       uint8_t *flag, int nth)
{
#pragma omp parallel num_threads(nth)
    {
        int tid = omp_get_thread_num();
        uint64_t lo = n * tid / nth, hi = n * (tid + 1) / nth;
        while (lo > 0 && lo < n && key[lo] == key[lo - 1]) lo++;   /* start at a group head */
        while (hi > 0 && hi < n && key[hi] == key[hi - 1]) hi++;
        int32_t rep[64][3];
        for (uint64_t a = lo; a < hi;) {
            uint64_t b = a + 1;
            while (b < n && key[b] == key[a]) b++;
            int nrep = 0;
            for (uint64_t i = a; i < b; i++) {
                int32_t h, r, t;
                candidate(g, idx[i], &h, &r, &t);
                int seen = 0;
                for (int k = 0; k < nrep; k++)
                    if (rep[k][0] == h && rep[k][1] == r && rep[k][2] == t) { seen = 1; break; }
                if (!seen && nrep == 64) {
                    /* pathological key collision: compare against every earlier member */
                    for (uint64_t k = a; k < i && !seen; k++) {
                        int32_t h2, r2, t2;
                        candidate(g, idx[k], &h2, &r2, &t2);
                        seen = (h2 == h && r2 == r && t2 == t);
                    }
                }
                flag[idx[i]] = (uint8_t)!seen;
                if (!seen && nrep < 64) { rep[nrep][0] = h; rep[nrep][1] = r; rep[nrep][2] = t; nrep++; }
            }
            a = b;
        }
    }
}

/*
 * Generate E triples into out[E*3] (row-major h, r, t).
 * Returns E on success, a negative value on error.
 */
int64_t kgs_generate(int64_t V, int64_t R, int64_t E,
                     int head_zipf, double head_s, int tail_zipf, double tail_s,
                     int rel_zipf, double rel_s, int shared_perm, int64_t deg_cap,
                     uint64_t seed, double overdraw, int32_t *out, int nthreads)
{
    if (V <= 0 || R <= 0 || E < 0 || V > 0x7FFFFFFF || R > 0x7FFFFFFF || !out) return -1;
    if ((double)E > 0.5 * (double)V * (double)R * (double)V) return -1;
    int nth = nthreads > 0 ? nthreads : omp_get_max_threads();
    gen_t g;
    g.seed = seed;
    if (dist_init(&g.dh, (uint64_t)V, head_zipf, head_s)) return -2;
    if (dist_init(&g.dr, (uint64_t)R, rel_zipf, rel_s)) return -2;
    int same_tail = shared_perm && tail_zipf == head_zipf && tail_s == head_s;
    if (same_tail) { g.pdt = &g.dh; g.dt.prob = NULL; g.dt.alias = NULL; }
    else { if (dist_init(&g.dt, (uint64_t)V, tail_zipf, tail_s)) return -2; g.pdt = &g.dt; }
    perm_init(&g.ph, (uint64_t)V, splitmix64(seed ^ 0x1111));
    perm_init(&g.pr, (uint64_t)R, splitmix64(seed ^ 0x2222));
    if (shared_perm) g.ppt = &g.ph;
    else { perm_init(&g.pt, (uint64_t)V, splitmix64(seed ^ 0x3333)); g.ppt = &g.pt; }

    int64_t result = -3;
    /* overdraw only sets the first stream length tried; the result is the
       same for any value */
    if (!(overdraw >= 1.0)) overdraw = 1.25;
    uint64_t n = (uint64_t)((double)E * overdraw) + 1024;
    for (int round = 0; round < 8; round++) {
        if (n > 0xFFFFFFF0ULL) n = 0xFFFFFFF0ULL;
        uint32_t *key = (uint32_t *)malloc(n * 4), *idx = (uint32_t *)malloc(n * 4);
        uint32_t *key2 = (uint32_t *)malloc(n * 4), *idx2 = (uint32_t *)malloc(n * 4);
        uint8_t *flag = (uint8_t *)malloc(n);
        if (!key || !idx || !key2 || !idx2 || !flag) {
            free(key); free(idx); free(key2); free(idx2); free(flag);
            result = -2;
            break;
        }
#pragma omp parallel for num_threads(nth) schedule(static)
        for (uint64_t i = 0; i < n; i++) {
            int32_t h, r, t;
            candidate(&g, i, &h, &r, &t);
            key[i] = triple_key(h, r, t);
            idx[i] = (uint32_t)i;
        }
        radix_sort(key, idx, key2, idx2, n, nth);
        free(key);
        free(idx);
        mark_first(&g, key2, idx2, n, flag, nth);
        free(key2);
        free(idx2);
        /* take the first E distinct candidates in index order, honouring the cap */
        int32_t *outdeg = NULL, *indeg = NULL;
        if (deg_cap > 0) {
            outdeg = (int32_t *)calloc((size_t)V, 4);
            indeg = (int32_t *)calloc((size_t)V, 4);
        }
        int64_t m = 0;
        uint64_t last = 0;
        for (uint64_t i = 0; i < n && m < E; i++) {
            if (!flag[i]) continue;
            if (deg_cap > 0) {
                int32_t h, r, t;
                candidate(&g, i, &h, &r, &t);
                if (outdeg[h] >= deg_cap || indeg[t] >= deg_cap) { flag[i] = 0; continue; }
                outdeg[h]++;
                indeg[t]++;
            }
            m++;
            last = i;
        }
        free(outdeg);
        free(indeg);
        if (getenv("KGS_DEBUG")) fprintf(stderr, "kgs round %d n=%llu accepted=%lld\n", round, (unsigned long long)n, (long long)m);
        if (m == E) {
            /* positions of the accepted candidates, then fill in parallel */
            uint64_t lim = E > 0 ? last + 1 : 0;
            int64_t *pos = (int64_t *)malloc(((size_t)nth + 1) * sizeof(int64_t));
#pragma omp parallel num_threads(nth)
            {
                int tid = omp_get_thread_num();
                uint64_t lo = lim * tid / nth, hi = lim * (tid + 1) / nth;
                int64_t c = 0;
                for (uint64_t i = lo; i < hi; i++) c += flag[i];
                pos[tid + 1] = c;
#pragma omp barrier
#pragma omp single
                {
                    pos[0] = 0;
                    for (int p = 0; p < nth; p++) pos[p + 1] += pos[p];
                }
                int64_t o = pos[tid];
                for (uint64_t i = lo; i < hi; i++) {
                    if (!flag[i]) continue;
                    candidate(&g, i, &out[3 * o], &out[3 * o + 1], &out[3 * o + 2]);
                    to_ids(&g, &out[3 * o], &out[3 * o + 1], &out[3 * o + 2]);
                    o++;
                }
            }
            free(pos);
            free(flag);
            result = E;
            break;
        }
        free(flag);
        if (n == 0xFFFFFFF0ULL) { result = -4; break; }
        double grow = m > 0 ? 1.2 * (double)E / (double)m : 4.0;
        if (grow < 1.25) grow = 1.25;
        if (grow > 4.0) grow = 4.0;
        n = (uint64_t)((double)n * grow);
    }
    dist_free(&g.dh);
    dist_free(&g.dr);
    if (!same_tail) dist_free(&g.dt);
    return result;
}
