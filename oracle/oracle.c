/*
 * oracle.c -- plain CPU oracle (test infrastructure only; see oracle.h).
 *
 * Written for clarity, not speed: sorted arrays, binary search, recursion
 * over the query's computation plan.  Every function names the passage of
 * the paper it follows.  Points the paper leaves open are taken as:
 *   - root of reverse sampling uniform over entities with an in-edge;
 *   - each projection step picks an in-relation uniformly among the
 *     entity's distinct in-relations, then an in-neighbour uniformly;
 *   - union branches are grounded from the same entity as intersection
 *     branches;
 *   - an attempt is rejected when a walk reaches an entity without
 *     in-edges, when two single-projection sibling branches get the same
 *     (anchor, relation), or when max_fanout > 0 and a grounded step's
 *     forward neighbour list under its relation exceeds max_fanout;
 *   - candidates are uniform over all V entities, kept iff outside A_q and
 *     not drawn before (the negative set is a set);
 *   - a negated operand of an intersection is grounded from a sibling
 *     entity: the intersection's positive operands are grounded first (from
 *     the intersection's entity e, in plan order); then one entity w is
 *     drawn uniformly from A_r(x), where (x, r) -> e is the step of the
 *     first positive operand; the negated operand's subtree is grounded
 *     from w by the same reverse walk; the attempt is rejected if e lies in
 *     the negated operand's set.  The root therefore stays an answer, and
 *     the negated set overlaps the positive operand's set (it holds w).
 */
#include "oracle.h"

#include <stdlib.h>
#include <string.h>
#include <omp.h>

/* ------------------------------------------------------------------ Philox */
/* Philox4x32-10, Salmon et al., "Parallel Random Numbers: As Easy as 1, 2, 3",
   SC'11: ten rounds of two 32x32->64 multiplies with a Weyl key schedule. */
void oracle_philox(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; round++) {
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

uint64_t oracle_pick(uint64_t u, uint64_t n)
{
    return (uint64_t)(((unsigned __int128)u * n) >> 64);
}

uint64_t oracle_draw(uint64_t seed, uint32_t tag, uint32_t qid, uint32_t t, uint32_t j)
{
    uint32_t ctr[4] = {j, t, qid, tag};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t x[4];
    oracle_philox(ctr, key, x);
    return ((uint64_t)x[1] << 32) | x[0];
}

#define TAG_POS 1u
#define TAG_NEG 2u
#define TAG_SHARED 3u   /* the candidate set shared by a minibatch */

/* ------------------------------------------------------------------- graph */
/* The KG is a set of triples (Sec. 2); A_r(v) is the set of tails of v under
   r (appendix on the query computation plan).  Forward edges are kept sorted
   by (head, relation, tail) and reverse edges by (tail, relation, head). */
struct okg {
    int32_t V, R;
    int64_t E;
    int64_t *f_off;             /* [V+1] */
    int32_t *f_rel, *f_nbr;     /* [E] */
    int64_t *r_off;             /* [V+1] */
    int32_t *r_rel, *r_nbr;     /* [E] */
    int64_t *rs_off;            /* [V+1] first reverse segment of each entity */
    int32_t *rs_rel;            /* [S_rev] */
    int64_t *rs_beg;            /* [S_rev+1] edge range of each reverse segment */
    int64_t *fs_off;            /* [V+1] first forward segment of each entity */
    int32_t *fs_rel;            /* [S_fwd] relation of each forward segment */
    int64_t S_fwd, S_rev;
    int32_t *active_in;
    int64_t n_active;
};

static int cmp_u64(const void *a, const void *b)
{
    uint64_t x = *(const uint64_t *)a, y = *(const uint64_t *)b;
    return x < y ? -1 : x > y;
}

static int cmp_i32(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return x < y ? -1 : x > y;
}

/* Group edges by a primary entity, sort each group by (relation, other end),
   drop duplicates.  prim/rel/oth give edge i. */
typedef void (*edge_fn)(const void *ctx, int64_t i, int32_t *p, int32_t *r, int32_t *o);

static int group_sort(const void *ctx, edge_fn edge, int64_t n, int32_t V, int nthreads,
                      int64_t **off_out, int32_t **rel_out, int32_t **nbr_out, int64_t *m_out)
{
    int64_t *off = (int64_t *)calloc((size_t)V + 1, sizeof(int64_t));
    int64_t *cur = (int64_t *)malloc(((size_t)V + 1) * sizeof(int64_t));
    uint64_t *key = (uint64_t *)malloc((size_t)(n > 0 ? n : 1) * sizeof(uint64_t));
    if (!off || !cur || !key) { free(off); free(cur); free(key); return -1; }
    for (int64_t i = 0; i < n; i++) {
        int32_t p, r, o;
        edge(ctx, i, &p, &r, &o);
        off[p + 1]++;
    }
    for (int32_t v = 0; v < V; v++) off[v + 1] += off[v];
    memcpy(cur, off, ((size_t)V + 1) * sizeof(int64_t));
    for (int64_t i = 0; i < n; i++) {
        int32_t p, r, o;
        edge(ctx, i, &p, &r, &o);
        key[cur[p]++] = ((uint64_t)(uint32_t)r << 32) | (uint32_t)o;
    }
#pragma omp parallel for schedule(dynamic, 1024) num_threads(nthreads)
    for (int32_t v = 0; v < V; v++)
        if (off[v + 1] - off[v] > 1) qsort(key + off[v], (size_t)(off[v + 1] - off[v]), 8, cmp_u64);
    /* remove duplicates inside each group */
    int64_t w = 0;
    for (int32_t v = 0; v < V; v++) {
        int64_t b = off[v], e = off[v + 1];
        cur[v] = w;
        for (int64_t k = b; k < e; k++)
            if (k == b || key[k] != key[k - 1]) key[w++] = key[k];
    }
    cur[V] = w;
    int32_t *rel = (int32_t *)malloc((size_t)(w > 0 ? w : 1) * 4);
    int32_t *nbr = (int32_t *)malloc((size_t)(w > 0 ? w : 1) * 4);
    if (!rel || !nbr) { free(off); free(cur); free(key); free(rel); free(nbr); return -1; }
    for (int64_t k = 0; k < w; k++) {
        rel[k] = (int32_t)(key[k] >> 32);
        nbr[k] = (int32_t)(uint32_t)key[k];
    }
    free(key);
    free(off);
    *off_out = cur;
    *rel_out = rel;
    *nbr_out = nbr;
    *m_out = w;
    return 0;
}

typedef struct { const int32_t *tr; int64_t n; int32_t R; } in_ctx;

/* input triple i, or for i >= n the inverse (t, r+R, h) of triple i-n */
static void in_edge(const void *c, int64_t i, int32_t *p, int32_t *r, int32_t *o)
{
    const in_ctx *x = (const in_ctx *)c;
    if (i < x->n) { *p = x->tr[3 * i]; *r = x->tr[3 * i + 1]; *o = x->tr[3 * i + 2]; }
    else { i -= x->n; *p = x->tr[3 * i + 2]; *r = x->tr[3 * i + 1] + x->R; *o = x->tr[3 * i]; }
}

typedef struct { const okg *g; const int32_t *head; } fwd_ctx;

/* forward edge i seen from its tail: (tail, relation, head) */
static void rev_edge(const void *c, int64_t i, int32_t *p, int32_t *r, int32_t *o)
{
    const fwd_ctx *x = (const fwd_ctx *)c;
    *p = x->g->f_nbr[i];
    *r = x->g->f_rel[i];
    *o = x->head[i];
}

void oracle_graph_free(okg *g)
{
    if (!g) return;
    free(g->f_off); free(g->f_rel); free(g->f_nbr);
    free(g->r_off); free(g->r_rel); free(g->r_nbr);
    free(g->rs_off); free(g->rs_rel); free(g->rs_beg);
    free(g->fs_off); free(g->fs_rel);
    free(g->active_in);
    free(g);
}

okg *oracle_graph_build(const int32_t *triples, int64_t n, int32_t V, int32_t R, int add_inverse,
                        int nthreads)
{
    if (V <= 0 || R <= 0 || n < 0 || (n > 0 && !triples)) return NULL;
    if (add_inverse && (int64_t)R * 2 > 0x7FFFFFFF) return NULL;
    for (int64_t i = 0; i < n; i++) {
        int32_t h = triples[3 * i], r = triples[3 * i + 1], t = triples[3 * i + 2];
        if (h < 0 || h >= V || t < 0 || t >= V || r < 0 || r >= R) return NULL;
    }
    if (nthreads <= 0) nthreads = omp_get_max_threads();
    okg *g = (okg *)calloc(1, sizeof(okg));
    if (!g) return NULL;
    g->V = V;
    g->R = add_inverse ? 2 * R : R;
    in_ctx ic = {triples, n, R};
    int64_t m;
    if (group_sort(&ic, in_edge, add_inverse ? 2 * n : n, V, nthreads, &g->f_off, &g->f_rel,
                   &g->f_nbr, &m)) { oracle_graph_free(g); return NULL; }
    g->E = m;
    /* head of every forward edge, for building the reverse lists */
    int32_t *head = (int32_t *)malloc((size_t)(m > 0 ? m : 1) * 4);
    if (!head) { oracle_graph_free(g); return NULL; }
    for (int32_t v = 0; v < V; v++)
        for (int64_t k = g->f_off[v]; k < g->f_off[v + 1]; k++) head[k] = v;
    fwd_ctx fc = {g, head};
    int64_t m2;
    int rc = group_sort(&fc, rev_edge, m, V, nthreads, &g->r_off, &g->r_rel, &g->r_nbr, &m2);
    free(head);
    if (rc || m2 != m) { oracle_graph_free(g); return NULL; }
    /* forward segments (runs of one relation per entity) and their relations */
    g->S_fwd = 0;
    for (int32_t v = 0; v < V; v++)
        for (int64_t k = g->f_off[v]; k < g->f_off[v + 1]; k++)
            if (k == g->f_off[v] || g->f_rel[k] != g->f_rel[k - 1]) g->S_fwd++;
    g->fs_off = (int64_t *)malloc(((size_t)V + 1) * 8);
    g->fs_rel = (int32_t *)malloc((size_t)(g->S_fwd > 0 ? g->S_fwd : 1) * 4);
    if (!g->fs_off || !g->fs_rel) { oracle_graph_free(g); return NULL; }
    {
        int64_t sf = 0;
        for (int32_t v = 0; v < V; v++) {
            g->fs_off[v] = sf;
            for (int64_t k = g->f_off[v]; k < g->f_off[v + 1]; k++)
                if (k == g->f_off[v] || g->f_rel[k] != g->f_rel[k - 1]) g->fs_rel[sf++] = g->f_rel[k];
        }
        g->fs_off[V] = sf;
    }
    int64_t S = 0;
    for (int32_t v = 0; v < V; v++)
        for (int64_t k = g->r_off[v]; k < g->r_off[v + 1]; k++)
            if (k == g->r_off[v] || g->r_rel[k] != g->r_rel[k - 1]) S++;
    g->S_rev = S;
    g->rs_off = (int64_t *)malloc(((size_t)V + 1) * 8);
    g->rs_rel = (int32_t *)malloc((size_t)(S > 0 ? S : 1) * 4);
    g->rs_beg = (int64_t *)malloc(((size_t)S + 1) * 8);
    if (!g->rs_off || !g->rs_rel || !g->rs_beg) { oracle_graph_free(g); return NULL; }
    S = 0;
    for (int32_t v = 0; v < V; v++) {
        g->rs_off[v] = S;
        for (int64_t k = g->r_off[v]; k < g->r_off[v + 1]; k++)
            if (k == g->r_off[v] || g->r_rel[k] != g->r_rel[k - 1]) {
                g->rs_rel[S] = g->r_rel[k];
                g->rs_beg[S] = k;
                S++;
            }
    }
    g->rs_off[V] = S;
    g->rs_beg[S] = m;
    int64_t na = 0;
    for (int32_t v = 0; v < V; v++) na += g->r_off[v + 1] > g->r_off[v];
    g->active_in = (int32_t *)malloc((size_t)(na > 0 ? na : 1) * 4);
    if (!g->active_in) { oracle_graph_free(g); return NULL; }
    na = 0;
    for (int32_t v = 0; v < V; v++)
        if (g->r_off[v + 1] > g->r_off[v]) g->active_in[na++] = v;
    g->n_active = na;
    return g;
}

void oracle_graph_stats(const okg *g, int64_t *st)
{
    int64_t mo = 0, mi = 0, ms = 0;
    for (int32_t v = 0; v < g->V; v++) {
        if (g->f_off[v + 1] - g->f_off[v] > mo) mo = g->f_off[v + 1] - g->f_off[v];
        if (g->r_off[v + 1] - g->r_off[v] > mi) mi = g->r_off[v + 1] - g->r_off[v];
    }
    for (int64_t s = 0; s < g->S_rev; s++)
        if (g->rs_beg[s + 1] - g->rs_beg[s] > ms) ms = g->rs_beg[s + 1] - g->rs_beg[s];
    st[0] = g->V; st[1] = g->R; st[2] = g->E; st[3] = g->S_fwd; st[4] = g->S_rev;
    st[5] = g->n_active; st[6] = mo; st[7] = mi; st[8] = ms;
}

int64_t oracle_graph_edges(const okg *g, int dir, int32_t v, int32_t *rel, int32_t *nbr)
{
    if (v < 0 || v >= g->V) return -1;
    const int64_t *off = dir ? g->r_off : g->f_off;
    const int32_t *r = dir ? g->r_rel : g->f_rel, *o = dir ? g->r_nbr : g->f_nbr;
    int64_t b = off[v], e = off[v + 1];
    if (rel) memcpy(rel, r + b, (size_t)(e - b) * 4);
    if (nbr) memcpy(nbr, o + b, (size_t)(e - b) * 4);
    return e - b;
}

int64_t oracle_graph_dump(const okg *g, int dir, int32_t *ent, int32_t *rel, int32_t *nbr)
{
    const int64_t *off = dir ? g->r_off : g->f_off;
    const int32_t *r = dir ? g->r_rel : g->f_rel, *o = dir ? g->r_nbr : g->f_nbr;
    for (int32_t v = 0; v < g->V; v++)
        for (int64_t k = off[v]; k < off[v + 1]; k++) {
            ent[k] = v;
            rel[k] = r[k];
            nbr[k] = o[k];
        }
    return g->E;
}

int64_t oracle_graph_active_in(const okg *g, int32_t *out)
{
    if (out) memcpy(out, g->active_in, (size_t)g->n_active * 4);
    return g->n_active;
}

/* [*b, *e): the edges of v under relation r in one direction (binary search
   for the run of relation r inside v's sorted edge list). */
static void rel_range(const int64_t *off, const int32_t *rel, int32_t v, int32_t r, int64_t *b,
                      int64_t *e)
{
    int64_t lo = off[v], hi = off[v + 1];
    while (lo < hi) {               /* first edge with relation >= r */
        int64_t mid = lo + (hi - lo) / 2;
        if (rel[mid] < r) lo = mid + 1; else hi = mid;
    }
    int64_t first = lo;
    hi = off[v + 1];
    while (lo < hi) {               /* first edge with relation > r */
        int64_t mid = lo + (hi - lo) / 2;
        if (rel[mid] <= r) lo = mid + 1; else hi = mid;
    }
    *b = first;
    *e = lo;
}

/* ---------------------------------------------------------- query plans */
/* Computation plans of the fourteen query structures of the experiments
   (Sec. 5.1: the structures of BetaE; the plan operators are those of the
   appendix on the computation plan): nine without negation and 2in, 3in,
   inp, pin, pni.  Nodes are listed children first.  Projection nodes carry
   a relation slot, anchors an anchor slot; intersection, union and
   complement edges carry no relation. */
enum { N_ANCHOR = 0, N_PROJ = 1, N_AND = 2, N_OR = 3, N_NOT = 4 };
typedef struct { int op, nch, ch[3], slot; } onode;
typedef struct { const char *name; int n, root; onode nd[8]; } otype;

#define A(s)       {N_ANCHOR, 0, {-1, -1, -1}, s}
#define P(c, s)    {N_PROJ, 1, {c, -1, -1}, s}
#define AND2(a, b) {N_AND, 2, {a, b, -1}, -1}
#define AND3(a, b, c) {N_AND, 3, {a, b, c}, -1}
#define OR2(a, b)  {N_OR, 2, {a, b, -1}, -1}
#define NOT(c)     {N_NOT, 1, {c, -1, -1}, -1}
#define NTYPES 14

static const otype TYPES[NTYPES] = {
    {"1p", 2, 1, {A(0), P(0, 0)}},
    {"2p", 3, 2, {A(0), P(0, 0), P(1, 1)}},
    {"3p", 4, 3, {A(0), P(0, 0), P(1, 1), P(2, 2)}},
    {"2i", 5, 4, {A(0), P(0, 0), A(1), P(2, 1), AND2(1, 3)}},
    {"3i", 7, 6, {A(0), P(0, 0), A(1), P(2, 1), A(2), P(4, 2), AND3(1, 3, 5)}},
    {"ip", 6, 5, {A(0), P(0, 0), A(1), P(2, 1), AND2(1, 3), P(4, 2)}},
    {"pi", 6, 5, {A(0), P(0, 0), P(1, 1), A(1), P(3, 2), AND2(2, 4)}},
    {"2u", 5, 4, {A(0), P(0, 0), A(1), P(2, 1), OR2(1, 3)}},
    {"up", 6, 5, {A(0), P(0, 0), A(1), P(2, 1), OR2(1, 3), P(4, 2)}},
    {"2in", 6, 5, {A(0), P(0, 0), A(1), P(2, 1), NOT(3), AND2(1, 4)}},
    {"3in", 8, 7, {A(0), P(0, 0), A(1), P(2, 1), A(2), P(4, 2), NOT(5), AND3(1, 3, 6)}},
    {"inp", 7, 6, {A(0), P(0, 0), A(1), P(2, 1), NOT(3), AND2(1, 4), P(5, 2)}},
    {"pin", 7, 6, {A(0), P(0, 0), P(1, 1), A(1), P(3, 2), NOT(4), AND2(2, 5)}},
    {"pni", 7, 6, {A(0), P(0, 0), P(1, 1), NOT(2), A(1), P(4, 2), AND2(3, 5)}},
};

int oracle_type_id(const char *name)
{
    for (int k = 0; k < NTYPES; k++)
        if (strcmp(TYPES[k].name, name) == 0) return k;
    return -1;
}

int oracle_type_plan(int qtype, int32_t *op, int32_t *child, int32_t *slot, int32_t *root)
{
    if (qtype < 0 || qtype >= NTYPES) return -1;
    const otype *T = &TYPES[qtype];
    for (int k = 0; k < T->n; k++) {
        op[k] = T->nd[k].op;
        slot[k] = T->nd[k].slot;
        for (int c = 0; c < 3; c++) child[3 * k + c] = c < T->nd[k].nch ? T->nd[k].ch[c] : -1;
    }
    *root = T->root;
    return T->n;
}

/* ------------------------------------------------------------ entity sets */
typedef struct { int32_t *v; int64_t n; } iset;

static int proj_mode = 0;   /* 0: auto, 1: always sort, 2: always bitmap (for tests) */
void oracle_set_proj_mode(int mode) { proj_mode = mode; }

/* Relation projection: union of A_r(v) over v in S, as a sorted set. */
static iset set_proj(const okg *g, iset S, int32_t r)
{
    int64_t total = 0;
    for (int64_t i = 0; i < S.n; i++) {
        int64_t b, e;
        rel_range(g->f_off, g->f_rel, S.v[i], r, &b, &e);
        total += e - b;
    }
    iset out = {NULL, 0};
    if (total == 0) return out;
    int use_bitmap = proj_mode == 2 || (proj_mode == 0 && total * 16 >= g->V);
    if (use_bitmap) {
        int64_t words = ((int64_t)g->V + 63) / 64;
        uint64_t *bits = (uint64_t *)calloc((size_t)words, 8);
        for (int64_t i = 0; i < S.n; i++) {
            int64_t b, e;
            rel_range(g->f_off, g->f_rel, S.v[i], r, &b, &e);
            for (int64_t k = b; k < e; k++) bits[g->f_nbr[k] >> 6] |= 1ULL << (g->f_nbr[k] & 63);
        }
        int64_t cnt = 0;
        for (int64_t w = 0; w < words; w++) cnt += __builtin_popcountll(bits[w]);
        out.v = (int32_t *)malloc((size_t)cnt * 4);
        for (int64_t w = 0; w < words; w++)
            for (uint64_t x = bits[w]; x; x &= x - 1) out.v[out.n++] = (int32_t)(w * 64 + __builtin_ctzll(x));
        free(bits);
    } else {
        out.v = (int32_t *)malloc((size_t)total * 4);
        for (int64_t i = 0; i < S.n; i++) {
            int64_t b, e;
            rel_range(g->f_off, g->f_rel, S.v[i], r, &b, &e);
            for (int64_t k = b; k < e; k++) out.v[out.n++] = g->f_nbr[k];
        }
        qsort(out.v, (size_t)out.n, 4, cmp_i32);
        int64_t w = 0;
        for (int64_t k = 0; k < out.n; k++)
            if (k == 0 || out.v[k] != out.v[k - 1]) out.v[w++] = out.v[k];
        out.n = w;
    }
    return out;
}

/* Intersection / union of two sorted sets by a linear merge (the appendix on
   the optimal cut notes sorted lists make both linear time). */
static iset set_merge(iset a, iset b, int is_union)
{
    iset o;
    o.v = (int32_t *)malloc((size_t)(a.n + b.n > 0 ? a.n + b.n : 1) * 4);
    o.n = 0;
    int64_t i = 0, j = 0;
    while (i < a.n && j < b.n) {
        if (a.v[i] < b.v[j]) { if (is_union) o.v[o.n++] = a.v[i]; i++; }
        else if (a.v[i] > b.v[j]) { if (is_union) o.v[o.n++] = b.v[j]; j++; }
        else { o.v[o.n++] = a.v[i]; i++; j++; }
    }
    if (is_union) {
        while (i < a.n) o.v[o.n++] = a.v[i++];
        while (j < b.n) o.v[o.n++] = b.v[j++];
    }
    return o;
}

/* a minus b for sorted sets (the delayed complement of the appendix on the
   optimal cut: an intersection with a complemented operand is computed as
   a set difference instead of materialising the complement). */
static iset set_minus(iset a, iset b)
{
    iset o;
    o.v = (int32_t *)malloc((size_t)(a.n > 0 ? a.n : 1) * 4);
    o.n = 0;
    int64_t j = 0;
    for (int64_t i = 0; i < a.n; i++) {
        while (j < b.n && b.v[j] < a.v[i]) j++;
        if (j < b.n && b.v[j] == a.v[i]) continue;
        o.v[o.n++] = a.v[i];
    }
    return o;
}

/* V minus s: the complement operator of the appendix on the computation
   plan, used where a complemented set is not an intersection operand. */
static iset set_complement(int32_t V, iset s)
{
    iset o;
    o.v = (int32_t *)malloc((size_t)(V - s.n > 0 ? V - s.n : 1) * 4);
    o.n = 0;
    int64_t j = 0;
    for (int32_t x = 0; x < V; x++) {
        if (j < s.n && s.v[j] == x) { j++; continue; }
        o.v[o.n++] = x;
    }
    return o;
}

static int set_has(iset s, int32_t x)
{
    int64_t lo = 0, hi = s.n;
    while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        if (s.v[mid] < x) lo = mid + 1; else hi = mid;
    }
    return lo < s.n && s.v[lo] == x;
}

/* Exhaustive execution of the plan from the anchors to node k (Sec. 2,
   "Traversing the KG using the computation plan to find answers"). */
static iset eval_node(const okg *g, const otype *T, int k, const int32_t *anchors,
                      const int32_t *relations)
{
    const onode *nd = &T->nd[k];
    iset out = {NULL, 0};
    if (nd->op == N_ANCHOR) {
        out.v = (int32_t *)malloc(4);
        out.v[0] = anchors[nd->slot];
        out.n = 1;
    } else if (nd->op == N_PROJ) {
        iset in = eval_node(g, T, nd->ch[0], anchors, relations);
        out = set_proj(g, in, relations[nd->slot]);
        free(in.v);
    } else if (nd->op == N_NOT) {
        iset in = eval_node(g, T, nd->ch[0], anchors, relations);
        out = set_complement(g->V, in);
        free(in.v);
    } else {
        /* an intersection with at least one positive operand subtracts its
           complemented operands after intersecting the others */
        int n_pos = 0;
        for (int c = 0; c < nd->nch; c++) n_pos += T->nd[nd->ch[c]].op != N_NOT;
        const int diff = nd->op == N_AND && n_pos > 0;
        int have = 0;
        for (int c = 0; c < nd->nch; c++) {
            if (diff && T->nd[nd->ch[c]].op == N_NOT) continue;
            iset b = eval_node(g, T, nd->ch[c], anchors, relations);
            if (!have) {
                out = b;
                have = 1;
                continue;
            }
            iset m = set_merge(out, b, nd->op == N_OR);
            free(out.v);
            free(b.v);
            out = m;
        }
        for (int c = 0; diff && c < nd->nch; c++) {
            if (T->nd[nd->ch[c]].op != N_NOT) continue;
            iset b = eval_node(g, T, T->nd[nd->ch[c]].ch[0], anchors, relations);
            iset m = set_minus(out, b);
            free(out.v);
            free(b.v);
            out = m;
        }
    }
    return out;
}

int64_t oracle_answer_set(const okg *g, int qtype, const int32_t *anchors,
                          const int32_t *relations, int32_t *out, int64_t cap)
{
    if (qtype < 0 || qtype >= NTYPES) return -1;
    const otype *T = &TYPES[qtype];
    for (int k = 0; k < T->n; k++) {
        const onode *nd = &T->nd[k];
        if (nd->op == N_ANCHOR && (anchors[nd->slot] < 0 || anchors[nd->slot] >= g->V)) return -1;
        if (nd->op == N_PROJ && (relations[nd->slot] < 0 || relations[nd->slot] >= g->R)) return -1;
    }
    iset s = eval_node(g, T, T->root, anchors, relations);
    if (out) memcpy(out, s.v, (size_t)(s.n < cap ? s.n : cap) * 4);
    int64_t n = s.n;
    free(s.v);
    return n;
}

/* ----------------------------------------------------- reverse sampling */
/* Reverse directional sampling (Sec. 3.1; appendix on reverse directional
   sampling): depth-first from the root to the anchors, children in index
   order.  A projection node whose output entity is e grounds its relation
   and input entity by g(e): an in-relation of e, then an in-neighbour of e
   under it.  Intersection and union children take the node's own entity;
   a complemented operand of an intersection is grounded from a sibling
   entity (reading in the header), after the positive operands. */
typedef struct {
    const okg *g;
    const otype *T;
    uint64_t seed;
    uint32_t qid, t, j;
    int32_t max_fanout;
    int32_t anchors[3], relations[3];
    int32_t ent[8];     /* entity each plan node was grounded with */
} walk;

static int ground(walk *w, const otype *T, int k, int32_t e)
{
    const onode *nd = &T->nd[k];
    const okg *g = w->g;
    w->ent[k] = e;
    if (nd->op == N_ANCHOR) {
        w->anchors[nd->slot] = e;
        return 1;
    }
    if (nd->op == N_PROJ) {
        int64_t nseg = g->rs_off[e + 1] - g->rs_off[e];
        uint64_t u0 = oracle_draw(w->seed, TAG_POS, w->qid, w->t, w->j);
        uint64_t u1 = oracle_draw(w->seed, TAG_POS, w->qid, w->t, w->j + 1);
        w->j += 2;
        if (nseg == 0) return 0;                         /* no in-edge: reject */
        int64_t s = g->rs_off[e] + (int64_t)oracle_pick(u0, (uint64_t)nseg);
        int64_t len = g->rs_beg[s + 1] - g->rs_beg[s];
        int32_t x = g->r_nbr[g->rs_beg[s] + (int64_t)oracle_pick(u1, (uint64_t)len)];
        int32_t r = g->rs_rel[s];
        if (w->max_fanout > 0) {
            int64_t b, en;
            rel_range(g->f_off, g->f_rel, x, r, &b, &en);
            if (en - b > w->max_fanout) return 0;         /* step expands too much */
        }
        w->relations[nd->slot] = r;
        return ground(w, T, nd->ch[0], x);
    }
    if (nd->op == N_NOT) return ground(w, T, nd->ch[0], e);
    int first_pos = -1;
    for (int c = 0; c < nd->nch; c++) {
        if (T->nd[nd->ch[c]].op == N_NOT) continue;
        if (first_pos < 0) first_pos = nd->ch[c];
        if (!ground(w, T, nd->ch[c], e)) return 0;
    }
    for (int c = 0; c < nd->nch; c++) {
        const int neg = nd->ch[c];
        if (T->nd[neg].op != N_NOT) continue;
        /* the sibling entity: uniform over A_r(x) of the first positive
           operand's step (x, r) -> e, which holds e, so it is never empty */
        const onode *p = &T->nd[first_pos];
        if (nd->op != N_AND || p->op != N_PROJ) return 0;
        const int32_t x = w->ent[p->ch[0]], r = w->relations[p->slot];
        int64_t b, en;
        rel_range(g->f_off, g->f_rel, x, r, &b, &en);
        uint64_t u = oracle_draw(w->seed, TAG_POS, w->qid, w->t, w->j);
        w->j += 1;
        const int32_t sib = g->f_nbr[b + (int64_t)oracle_pick(u, (uint64_t)(en - b))];
        if (!ground(w, T, neg, sib)) return 0;
        /* e must stay outside the complemented set */
        iset S = eval_node(g, T, T->nd[neg].ch[0], w->anchors, w->relations);
        const int inside = set_has(S, e);
        free(S.v);
        if (inside) return 0;
    }
    /* two single-projection branches grounded to the same (anchor, relation)
       make a degenerate intersection or union: reject */
    for (int a = 0; a < nd->nch; a++)
        for (int b = a + 1; b < nd->nch; b++) {
            const onode *x = &T->nd[nd->ch[a]], *y = &T->nd[nd->ch[b]];
            if (x->op != N_PROJ || y->op != N_PROJ) continue;
            const onode *xa = &T->nd[x->ch[0]], *ya = &T->nd[y->ch[0]];
            if (xa->op != N_ANCHOR || ya->op != N_ANCHOR) continue;
            if (w->anchors[xa->slot] == w->anchors[ya->slot] &&
                w->relations[x->slot] == w->relations[y->slot]) return 0;
        }
    return 1;
}

/* small open-addressing set of candidate ids (first-occurrence test) */
typedef struct { int32_t *slot; uint32_t mask; } hset;

static int hset_insert(hset *h, int32_t x)   /* 1 if newly inserted */
{
    uint32_t i = ((uint32_t)x * 0x9E3779B1u) & h->mask;
    while (h->slot[i] != -1) {
        if (h->slot[i] == x) return 0;
        i = (i + 1) & h->mask;
    }
    h->slot[i] = x;
    return 1;
}

/* Positive of query id qid: the first accepted attempt of reverse
   directional sampling (root uniform over entities with an in-edge, then
   the walk).  Returns 1 with the grounding in *w, the root in *root and the
   attempts used in *attempts; 0 when all pos_tries attempts are rejected. */
static int sample_positive(const okg *g, const otype *T, const oracle_args *a, uint32_t qid,
                           walk *w, int32_t *root, int32_t *attempts)
{
    for (uint32_t t = 0; t < (uint32_t)a->pos_tries; t++) {
        w->g = g; w->T = T; w->seed = a->seed; w->qid = qid; w->t = t; w->j = 1;
        w->max_fanout = a->max_fanout;
        for (int k = 0; k < 3; k++) { w->anchors[k] = -1; w->relations[k] = -1; }
        if (g->n_active == 0) continue;
        uint64_t u = oracle_draw(a->seed, TAG_POS, qid, t, 0);
        *root = g->active_in[oracle_pick(u, (uint64_t)g->n_active)];
        if (ground(w, T, T->root, *root)) {
            *attempts = (int32_t)t + 1;
            return 1;
        }
    }
    *attempts = a->pos_tries;
    return 0;
}

static void sample_one(const okg *g, const otype *T, const oracle_args *a, int64_t b,
                       int32_t *anchors, int32_t *relations, int32_t *positive, int32_t *negatives,
                       int32_t *n_valid, int32_t *pos_attempts, int32_t *neg_draws)
{
    uint32_t qid = (uint32_t)(a->query_offset + (uint64_t)b);
    for (int k = 0; k < 3; k++) { anchors[3 * b + k] = -1; relations[3 * b + k] = -1; }
    for (int k = 0; k < a->n_neg; k++) negatives[(int64_t)a->n_neg * b + k] = -1;
    positive[b] = -1;
    walk w;
    int32_t root = -1;
    if (!sample_positive(g, T, a, qid, &w, &root, &pos_attempts[b])) {
        n_valid[b] = -1;
        neg_draws[b] = -1;
        return;
    }
    positive[b] = root;
    for (int k = 0; k < 3; k++) { anchors[3 * b + k] = w.anchors[k]; relations[3 * b + k] = w.relations[k]; }
    if (a->n_neg == 0) {   /* no candidates: the answer set is not needed */
        n_valid[b] = 0;
        neg_draws[b] = 0;
        return;
    }
    /* negatives: rejection sampling against the full answer set */
    iset Aq = eval_node(g, T, T->root, w.anchors, w.relations);
    uint32_t cap = 16;
    while (cap < 2u * (uint32_t)a->neg_tries) cap <<= 1;
    hset seen = {(int32_t *)malloc((size_t)cap * 4), cap - 1};
    memset(seen.slot, 0xFF, (size_t)cap * 4);
    int32_t acc = 0, draws = a->neg_tries;
    if (a->n_neg == 0) draws = 0;
    for (int32_t j = 0; j < a->neg_tries && acc < a->n_neg; j++) {
        uint64_t u = oracle_draw(a->seed, TAG_NEG, qid, 0, (uint32_t)j);
        int32_t c = (int32_t)oracle_pick(u, (uint64_t)g->V);
        int first = hset_insert(&seen, c);
        if (first && !set_has(Aq, c)) {
            negatives[(int64_t)a->n_neg * b + acc] = c;
            acc++;
            if (acc == a->n_neg) draws = j + 1;
        }
    }
    n_valid[b] = acc;
    neg_draws[b] = draws;
    free(seen.slot);
    free(Aq.v);
}

int oracle_sample(const okg *g, int qtype, const oracle_args *a, int32_t *anchors,
                  int32_t *relations, int32_t *positive, int32_t *negatives, int32_t *n_valid,
                  int32_t *pos_attempts, int32_t *neg_draws, int nthreads)
{
    if (!g || !a || qtype < 0 || qtype >= NTYPES) return -1;
    if (a->batch < 0 || a->n_neg < 0 || a->pos_tries < 1 || a->neg_tries < a->n_neg) return -1;
    if (a->query_offset + (uint64_t)a->batch > (1ULL << 32)) return -1;
    if (nthreads <= 0) nthreads = omp_get_max_threads();
    const otype *T = &TYPES[qtype];
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
    for (int64_t b = 0; b < a->batch; b++)
        sample_one(g, T, a, b, anchors, relations, positive, negatives, n_valid, pos_attempts,
                   neg_draws);
    return 0;
}

/* ------------------------------------------------------ shared negatives */
/* Sharing negative samples within a minibatch (Sec. 4.3): one candidate set
   N for all queries and Mask[i][k] = 1 iff N[k] is a negative of query i,
   i.e. not in its answer set.  N holds the first n_neg distinct values of
   the draws c_j = pick(U(SHARED, qid0, 0, j), V), j < neg_tries, with qid0
   the minibatch's query_offset; the positives are those of oracle_sample. */
int oracle_sample_shared(const okg *g, int qtype, const oracle_args *a, int32_t *anchors,
                         int32_t *relations, int32_t *positive, int32_t *pos_attempts,
                         int32_t *shared, int32_t *n_shared, uint32_t *mask, int32_t *n_valid,
                         int nthreads)
{
    if (!g || !a || qtype < 0 || qtype >= NTYPES) return -1;
    if (a->batch < 0 || a->n_neg < 0 || a->pos_tries < 1 || a->neg_tries < a->n_neg) return -1;
    if (a->query_offset + (uint64_t)a->batch > (1ULL << 32)) return -1;
    if (nthreads <= 0) nthreads = omp_get_max_threads();
    const otype *T = &TYPES[qtype];
    /* the shared candidate set */
    uint32_t cap = 16;
    while (cap < 2u * (uint32_t)a->neg_tries) cap <<= 1;
    hset seen = {(int32_t *)malloc((size_t)cap * 4), cap - 1};
    memset(seen.slot, 0xFF, (size_t)cap * 4);
    int32_t cnt = 0;
    for (int32_t j = 0; j < a->neg_tries && cnt < a->n_neg; j++) {
        uint64_t u = oracle_draw(a->seed, TAG_SHARED, (uint32_t)a->query_offset, 0, (uint32_t)j);
        int32_t c = (int32_t)oracle_pick(u, (uint64_t)g->V);
        if (hset_insert(&seen, c)) shared[cnt++] = c;
    }
    free(seen.slot);
    for (int32_t k = cnt; k < a->n_neg; k++) shared[k] = -1;
    *n_shared = cnt;
    const int64_t words = (a->n_neg + 31) / 32;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
    for (int64_t b = 0; b < a->batch; b++) {
        uint32_t qid = (uint32_t)(a->query_offset + (uint64_t)b);
        uint32_t *row = mask + words * b;
        for (int64_t w = 0; w < words; w++) row[w] = 0;
        for (int k = 0; k < 3; k++) { anchors[3 * b + k] = -1; relations[3 * b + k] = -1; }
        positive[b] = -1;
        walk w;
        int32_t root = -1;
        if (!sample_positive(g, T, a, qid, &w, &root, &pos_attempts[b])) {
            n_valid[b] = -1;
            continue;
        }
        positive[b] = root;
        for (int k = 0; k < 3; k++) { anchors[3 * b + k] = w.anchors[k]; relations[3 * b + k] = w.relations[k]; }
        iset Aq = eval_node(g, T, T->root, w.anchors, w.relations);
        int32_t kept = 0;
        for (int32_t k = 0; k < cnt; k++)
            if (!set_has(Aq, shared[k])) {
                row[k / 32] |= 1u << (k % 32);
                kept++;
            }
        n_valid[b] = kept;
        free(Aq.v);
    }
    return 0;
}

/* ------------------------------------------------------------ verification */
/* Membership of given candidates in the answer sets of given queries (the
   test a rejection sampler makes, Sec. 3.2; used for evaluation, where the
   answers of a query differ between nested graphs, appendix on the task
   setup).  Candidate k of query i is c = candidates[i * n + k]; mask bit k
   of row i is set iff 0 <= c < V and c is not in A_q; n_valid[i] counts the
   set bits, or is -1 when an anchor or relation of the query is out of
   range (its row is zero). */
int oracle_verify(const okg *g, int qtype, int32_t batch, int32_t n, const int32_t *anchors,
                  const int32_t *relations, const int32_t *candidates, uint32_t *mask,
                  int32_t *n_valid, int nthreads)
{
    if (!g || qtype < 0 || qtype >= NTYPES || batch < 0 || n < 0) return -1;
    if (nthreads <= 0) nthreads = omp_get_max_threads();
    const otype *T = &TYPES[qtype];
    const int64_t words = ((int64_t)n + 31) / 32;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
    for (int64_t i = 0; i < batch; i++) {
        uint32_t *row = mask + words * i;
        for (int64_t w = 0; w < words; w++) row[w] = 0;
        const int32_t *a = anchors + 3 * i, *r = relations + 3 * i;
        int ok = 1;
        for (int k = 0; k < T->n; k++) {   /* every slot the plan uses is in range */
            const onode *nd = &T->nd[k];
            if (nd->op == N_ANCHOR) ok = ok && a[nd->slot] >= 0 && a[nd->slot] < g->V;
            if (nd->op == N_PROJ) ok = ok && r[nd->slot] >= 0 && r[nd->slot] < g->R;
        }
        if (!ok) {
            n_valid[i] = -1;
            continue;
        }
        iset Aq = eval_node(g, T, T->root, a, r);
        int32_t kept = 0;
        for (int32_t k = 0; k < n; k++) {
            const int32_t c = candidates[(int64_t)n * i + k];
            if (c >= 0 && c < g->V && !set_has(Aq, c)) {
                row[k / 32] |= 1u << (k % 32);
                kept++;
            }
        }
        n_valid[i] = kept;
        free(Aq.v);
    }
    return 0;
}

/* --------------------------------------------------- bidirectional check */
/* Sec. 3.2, bidirectional rejection sampling: the sets at the cut nodes are
   computed from the anchors (forward caching); the candidate is expanded
   from the root towards the cut (backward verification) and accepted as an
   answer iff the two sides meet. */
typedef struct {
    const okg *g;
    const otype *T;
    uint32_t cut;
    iset F[8];
    const int32_t *relations;
    const int32_t *anchors;
    int64_t visited;
} bidir;

static int member(bidir *B, int k, int32_t x)
{
    if (B->cut & (1u << k)) return set_has(B->F[k], x);
    const onode *nd = &B->T->nd[k];
    if (nd->op == N_ANCHOR) return x == B->anchors[nd->slot];
    if (nd->op == N_PROJ) {
        /* x is in A_r(S) iff some y with (y, r, x) in E lies in S */
        int64_t b, e;
        rel_range(B->g->r_off, B->g->r_rel, x, B->relations[nd->slot], &b, &e);
        B->visited += e - b;
        for (int64_t i = b; i < e; i++)
            if (member(B, nd->ch[0], B->g->r_nbr[i])) return 1;
        return 0;
    }
    if (nd->op == N_NOT) return !member(B, nd->ch[0], x);
    for (int c = 0; c < nd->nch; c++) {
        int in = member(B, nd->ch[c], x);
        if (nd->op == N_AND && !in) return 0;
        if (nd->op == N_OR && in) return 1;
    }
    return nd->op == N_AND;
}

/* Def. of a node cut: every anchor-to-root path meets the cut exactly once. */
static int is_node_cut(const otype *T, uint32_t mask)
{
    if (mask >> T->n) return 0;
    int parent[8];
    for (int k = 0; k < T->n; k++) parent[k] = -1;
    for (int k = 0; k < T->n; k++)
        for (int c = 0; c < T->nd[k].nch; c++) parent[T->nd[k].ch[c]] = k;
    for (int k = 0; k < T->n; k++) {
        if (T->nd[k].op != N_ANCHOR) continue;
        int hits = 0;
        for (int v = k; v != -1; v = parent[v]) hits += (mask >> v) & 1;
        if (hits != 1) return 0;
    }
    return 1;
}

int oracle_bidir_check(const okg *g, int qtype, const int32_t *anchors, const int32_t *relations,
                       uint32_t cut_mask, int32_t c, int64_t *counts)
{
    if (qtype < 0 || qtype >= NTYPES || c < 0 || c >= g->V) return -1;
    const otype *T = &TYPES[qtype];
    if (!is_node_cut(T, cut_mask)) return -1;
    bidir B;
    memset(&B, 0, sizeof(B));
    B.g = g; B.T = T; B.cut = cut_mask; B.relations = relations; B.anchors = anchors;
    int64_t fwd = 0;
    for (int k = 0; k < T->n; k++)
        if (cut_mask & (1u << k)) {
            B.F[k] = eval_node(g, T, k, anchors, relations);
            fwd += B.F[k].n;
        }
    int in = member(&B, T->root, c);
    for (int k = 0; k < T->n; k++) free(B.F[k].v);
    if (counts) { counts[0] = fwd; counts[1] = B.visited; }
    return in;
}

/* ------------------------------------------------- reads of the method */
/* Memory lines a bidirectional check reads (Sec. 3.2: the cost discussion
   and the optimal-scheduling equation count the entities each side
   expands; this counts the 64-byte lines of graph data behind them, the
   unit the memory system moves).  The adjacency is laid out per direction
   as node[V+1] (int32: an entity's first group), grp[S+1] (int32 pairs:
   relation, first edge) and nbr[E] (int32), each array starting on a
   64-byte boundary; a line is a 64-byte block of one array.  Group and edge
   indices are those of the canonical order (entity, relation, neighbour
   ascending), which this oracle's arrays share with any CSR of the same
   graph.  Reads:
   - an entity's groups: the node entries v and v + 1;
   - the group of relation r: a lower-bound binary search over the entity's
     groups (probe (lo + hi) / 2, compare its relation), then the edge
     bounds of the group found (its entry and the next one);
   - a neighbour list that is expanded: its entries in ascending order, up
     to the first one that decides the check;
   - a list met with a forward-cached set: the shorter side gives the keys
     in ascending order, each key is looked up in the other side by the
     same lower-bound search, up to the first common entity; list keys and
     list probes are read;
   - an entity tested for membership in a forward-cached set: the same
     lower-bound search of the set;
   - a cached set that fits the STAGE_BUDGET entries staged per query (each
     cut set in node order is staged when it fits in what the sets staged
     before it left of the budget) is held on chip, so its keys and probes
     are free, while a larger one is searched where it is stored: the
     forward group A_r(a) when the set is one projection of an anchor (the
     only kind the strict cut caches), else a sorted array of its own;
   - forward caching: every cut set once, from the anchors, with the same
     reads (node entries, group search, the whole list).
   The candidates of query qid are draws j < n_draws, c_j =
   pick(U(NEG, qid, 0, j), V).  Lines fall in two parts: part 0 holds the
   forward caching, each candidate's own node entries and group search,
   edge tests against an anchor, and the expansion of backward lists of at
   most LONG_LIST entries when every forward-cached set of the query is
   staged; part 1 holds everything read below a longer list, and every
   backward read of a query with a set that is not staged.  Each part counts
   its distinct lines; the total counts distinct lines over both. */
#define LONG_LIST 8
#define STAGE_BUDGET 1024
enum { L_FNODE = 0, L_FGRP, L_FNBR, L_RNODE, L_RGRP, L_RNBR };

typedef struct { int64_t *v; int64_t n, cap; } lineset;

static void ls_add(lineset *s, int arr, int64_t byte_off, int64_t nbytes)
{
    for (int64_t l = byte_off >> 6; l <= (byte_off + nbytes - 1) >> 6; l++) {
        if (s->n == s->cap) {
            s->cap = s->cap ? 2 * s->cap : 256;
            s->v = (int64_t *)realloc(s->v, (size_t)s->cap * 8);
        }
        s->v[s->n++] = ((int64_t)arr << 56) | l;
    }
}

static int cmp_i64(const void *a, const void *b)
{
    int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
    return x < y ? -1 : x > y;
}

static int64_t ls_distinct(int64_t *v, int64_t n)
{
    if (n == 0) return 0;
    qsort(v, (size_t)n, 8, cmp_i64);
    int64_t d = 1;
    for (int64_t i = 1; i < n; i++) d += v[i] != v[i - 1];
    return d;
}

typedef struct {
    const okg *g;
    const otype *T;
    uint32_t cut;
    iset F[8];
    int staged[8];          /* cut set k fits the staging budget */
    int64_t fbase[8];       /* first forward edge of an unstaged cut set that is
                               one forward group, else -1 (an array of its own) */
    int all_staged;
    const int32_t *anchors, *relations;
    lineset part[2];
} vlines;

/* a read of entry i of cut set k where it is stored (unstaged sets only) */
static void vset_read(vlines *L, int part, int k, int64_t i)
{
    if (L->staged[k]) return;
    if (L->fbase[k] >= 0) ls_add(&L->part[part], L_FNBR, (L->fbase[k] + i) * 4, 4);
    else ls_add(&L->part[part], 6 + k, i * 4, 4);
}

/* the group of relation r of entity v in one direction: [*b, *e), or 0 */
static int vgroup(vlines *L, int part, int dir, int32_t v, int32_t r, int64_t *b, int64_t *e)
{
    const okg *g = L->g;
    const int64_t *soff = dir ? g->rs_off : g->fs_off;
    const int32_t *srel = dir ? g->rs_rel : g->fs_rel;
    const int arr = dir ? L_RGRP : L_FGRP;
    ls_add(&L->part[part], dir ? L_RNODE : L_FNODE, (int64_t)v * 4, 8);
    int64_t lo = soff[v], hi = soff[v + 1];
    const int64_t end = hi;
    while (lo < hi) {
        const int64_t mid = lo + (hi - lo) / 2;
        ls_add(&L->part[part], arr, mid * 8, 4);
        if (srel[mid] < r) lo = mid + 1; else hi = mid;
    }
    if (lo == end || srel[lo] != r) return 0;
    ls_add(&L->part[part], arr, lo * 8 + 4, 4);
    ls_add(&L->part[part], arr, (lo + 1) * 8 + 4, 4);
    rel_range(dir ? g->r_off : g->f_off, dir ? g->r_rel : g->f_rel, v, r, b, e);
    return 1;
}

/* does the reverse list [b, e) share an entity with cut set k? */
static int vmeet(vlines *L, int part, int64_t b, int64_t e, int k_set)
{
    const int32_t *nbr = L->g->r_nbr;
    const iset F = L->F[k_set];
    if (e - b <= F.n) {
        for (int64_t i = b; i < e; i++) {
            ls_add(&L->part[part], L_RNBR, i * 4, 4);
            /* lower-bound search of the list's entry in the cached set */
            int64_t lo = 0, hi = F.n;
            while (lo < hi) {
                const int64_t mid = lo + (hi - lo) / 2;
                vset_read(L, part, k_set, mid);
                if (F.v[mid] < nbr[i]) lo = mid + 1; else hi = mid;
            }
            if (lo < F.n) {
                vset_read(L, part, k_set, lo);
                if (F.v[lo] == nbr[i]) return 1;
            }
        }
        return 0;
    }
    for (int64_t k = 0; k < F.n; k++) {
        vset_read(L, part, k_set, k);
        int64_t lo = b, hi = e;
        while (lo < hi) {
            const int64_t mid = lo + (hi - lo) / 2;
            ls_add(&L->part[part], L_RNBR, mid * 4, 4);
            if (nbr[mid] < F.v[k]) lo = mid + 1; else hi = mid;
        }
        if (lo < e) {
            ls_add(&L->part[part], L_RNBR, lo * 4, 4);
            if (nbr[lo] == F.v[k]) return 1;
        }
    }
    return 0;
}

static int vmember(vlines *L, int k, int32_t x, int part)
{
    if (L->cut & (1u << k)) {
        const iset F = L->F[k];
        if (L->staged[k]) return set_has(F, x);
        /* a set over the staging budget: the same lower-bound search, where
           it is stored */
        int64_t lo = 0, hi = F.n;
        while (lo < hi) {
            const int64_t mid = lo + (hi - lo) / 2;
            vset_read(L, part, k, mid);
            if (F.v[mid] < x) lo = mid + 1; else hi = mid;
        }
        if (lo == F.n) return 0;
        vset_read(L, part, k, lo);
        return F.v[lo] == x;
    }
    const onode *nd = &L->T->nd[k];
    if (nd->op == N_ANCHOR) return x == L->anchors[nd->slot];
    if (nd->op == N_NOT) return !vmember(L, nd->ch[0], x, part);
    if (nd->op == N_AND || nd->op == N_OR) {
        for (int c = 0; c < nd->nch; c++) {
            const int in = vmember(L, nd->ch[c], x, part);
            if (nd->op == N_AND && !in) return 0;
            if (nd->op == N_OR && in) return 1;
        }
        return nd->op == N_AND;
    }
    /* projection: x is in A_r(S) iff some y with (y, r, x) in E lies in S */
    int64_t b, e;
    if (!vgroup(L, part, 1, x, L->relations[nd->slot], &b, &e)) return 0;
    const int ch = nd->ch[0];
    const int edge_test = (L->cut & (1u << ch)) && L->T->nd[ch].op == N_ANCHOR;
    const int p = edge_test ? part : (e - b > LONG_LIST || !L->all_staged) ? 1 : part;
    if (L->cut & (1u << ch)) return vmeet(L, p, b, e, ch);
    for (int64_t i = b; i < e; i++) {
        ls_add(&L->part[p], L_RNBR, i * 4, 4);
        if (vmember(L, ch, L->g->r_nbr[i], p)) return 1;
    }
    return 0;
}

/* reads of forward caching: the set at node k computed from the anchors */
static void vforward(vlines *L, int k)
{
    const onode *nd = &L->T->nd[k];
    if (nd->op == N_ANCHOR) return;
    for (int c = 0; c < nd->nch; c++) vforward(L, nd->ch[c]);
    if (nd->op != N_PROJ) return;
    iset S = eval_node(L->g, L->T, nd->ch[0], L->anchors, L->relations);
    for (int64_t i = 0; i < S.n; i++) {
        int64_t b, e;
        if (vgroup(L, 0, 0, S.v[i], L->relations[nd->slot], &b, &e) && e > b)
            ls_add(&L->part[0], L_FNBR, b * 4, (e - b) * 4);
    }
    free(S.v);
}

int oracle_verify_lines(const okg *g, int qtype, const int32_t *anchors, const int32_t *relations,
                        uint32_t cut_mask, uint64_t seed, uint32_t qid, int32_t n_draws,
                        int64_t *lines)
{
    if (!g || qtype < 0 || qtype >= NTYPES || n_draws < 0) return -1;
    const otype *T = &TYPES[qtype];
    if (!is_node_cut(T, cut_mask)) return -1;
    for (int k = 0; k < T->n; k++) {
        const onode *nd = &T->nd[k];
        if (nd->op == N_ANCHOR && (anchors[nd->slot] < 0 || anchors[nd->slot] >= g->V)) return -1;
        if (nd->op == N_PROJ && (relations[nd->slot] < 0 || relations[nd->slot] >= g->R)) return -1;
    }
    vlines L;
    memset(&L, 0, sizeof(L));
    L.g = g; L.T = T; L.cut = cut_mask; L.anchors = anchors; L.relations = relations;
    int64_t staged = 0;
    L.all_staged = 1;
    for (int k = 0; k < T->n; k++) {
        L.staged[k] = 1;
        L.fbase[k] = -1;
        if (!(cut_mask & (1u << k))) continue;
        L.F[k] = eval_node(g, T, k, anchors, relations);
        vforward(&L, k);
        const onode *nd = &T->nd[k];
        if (nd->op == N_ANCHOR) continue;
        if (L.F[k].n <= STAGE_BUDGET - staged) staged += L.F[k].n;
        else {
            L.all_staged = 0;
            L.staged[k] = 0;
            if (nd->op == N_PROJ && T->nd[nd->ch[0]].op == N_ANCHOR) {
                int64_t fb, fe;
                rel_range(g->f_off, g->f_rel, anchors[T->nd[nd->ch[0]].slot], relations[nd->slot], &fb, &fe);
                L.fbase[k] = fb;
            }
        }
    }
    for (int32_t j = 0; j < n_draws; j++) {
        const int32_t c = (int32_t)oracle_pick(oracle_draw(seed, TAG_NEG, qid, 0, (uint32_t)j),
                                               (uint64_t)g->V);
        (void)vmember(&L, T->root, c, 0);
    }
    int64_t *all = (int64_t *)malloc((size_t)(L.part[0].n + L.part[1].n + 1) * 8);
    if (L.part[0].n) memcpy(all, L.part[0].v, (size_t)L.part[0].n * 8);
    if (L.part[1].n) memcpy(all + L.part[0].n, L.part[1].v, (size_t)L.part[1].n * 8);
    lines[0] = ls_distinct(L.part[0].v, L.part[0].n);
    lines[1] = ls_distinct(L.part[1].v, L.part[1].n);
    lines[2] = ls_distinct(all, L.part[0].n + L.part[1].n);
    free(all);
    free(L.part[0].v);
    free(L.part[1].v);
    for (int k = 0; k < T->n; k++) free(L.F[k].v);
    return 0;
}

int oracle_verify_lines_batch(const okg *g, int qtype, int32_t batch, const int32_t *anchors,
                              const int32_t *relations, const int32_t *positive, uint32_t cut_mask,
                              uint64_t seed, uint64_t query_offset, int32_t n_draws, int64_t *lines,
                              int nthreads)
{
    if (!g || qtype < 0 || qtype >= NTYPES || batch < 0) return -1;
    if (nthreads <= 0) nthreads = omp_get_max_threads();
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads) reduction(| : bad)
    for (int64_t b = 0; b < batch; b++) {
        int64_t *out = lines + 3 * b;
        out[0] = out[1] = out[2] = 0;
        if (positive[b] < 0) continue;   /* no query: nothing is verified */
        bad |= oracle_verify_lines(g, qtype, anchors + 3 * b, relations + 3 * b, cut_mask, seed,
                                   (uint32_t)(query_offset + (uint64_t)b), n_draws, out) != 0;
    }
    return bad ? -1 : 0;
}
