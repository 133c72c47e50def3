/*
 * oracle.h -- plain CPU oracle for batched query sampling with verified
 * negatives (SMORE, arXiv 2110.14890).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load or call this code.  It shares no code
 * with the GPU library: its Philox, adjacency, query plans and set algebra
 * are written here independently.
 *
 * What it computes, per query (all integer, no floating point):
 *   - a positive answer by reverse directional sampling (Sec. 3.1 and the
 *     appendix on reverse directional sampling): ground the root, then walk
 *     from the root to the anchors, each projection edge picking an
 *     in-relation of the current entity and then an in-neighbour under it;
 *   - the full answer set A_q by exhaustive execution of the computation plan
 *     (Sec. 2, "Traversing the KG"; appendix on the query computation plan:
 *     projection, intersection, union);
 *   - negatives: uniform candidates over V kept iff not in A_q and not drawn
 *     before (Sec. 3.2: the negative set is a subset of the complement of
 *     A_q; rejection with a constant candidate budget).
 * It also has a generic bidirectional checker (Sec. 3.2, forward caching to a
 * node cut then backward verification) used to pin the equivalence of the two
 * tests for every valid cut.
 */
#ifndef SMORE_ORACLE_H
#define SMORE_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct okg okg;

/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): out[4] from ctr[4], key[2]. */
void oracle_philox(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);
/* floor(u * n / 2^64) */
uint64_t oracle_pick(uint64_t u, uint64_t n);
/* U(tag, qid, t, j): low two Philox words of counter (j, t, qid, tag), key = seed halves */
uint64_t oracle_draw(uint64_t seed, uint32_t tag, uint32_t qid, uint32_t t, uint32_t j);

/* Build adjacency from n triples (h, r, t).  add_inverse appends (t, r+R, h).
   Returns NULL on invalid ids or allocation failure. */
okg *oracle_graph_build(const int32_t *triples, int64_t n, int32_t V, int32_t R, int add_inverse,
                        int nthreads);
void oracle_graph_free(okg *g);
/* stats[0..8] = V, R', E, S_fwd, S_rev, n_active_in, max_out, max_in, max_seg */
void oracle_graph_stats(const okg *g, int64_t *stats);
/* Copy the forward (dir=0) or reverse (dir=1) adjacency of entity v:
   rel[k], nbr[k] for its edges in canonical order; returns the count
   (call with NULL buffers to get the count). */
int64_t oracle_graph_edges(const okg *g, int dir, int32_t v, int32_t *rel, int32_t *nbr);
/* All edges of one direction in canonical order: ent[k] (head for dir 0,
   tail for dir 1), rel[k], nbr[k]; arrays of length E.  Returns E. */
int64_t oracle_graph_dump(const okg *g, int dir, int32_t *ent, int32_t *rel, int32_t *nbr);
/* Copy active_in (entities with at least one in-edge, ascending). */
int64_t oracle_graph_active_in(const okg *g, int32_t *out);

/* query types: 0..13 = 1p 2p 3p 2i 3i ip pi 2u up 2in 3in inp pin pni */
int oracle_type_id(const char *name);

typedef struct {
    int32_t batch, n_neg, pos_tries, neg_tries, max_fanout;
    uint64_t seed, query_offset;
} oracle_args;

/* Sample a batch.  Arrays: anchors/relations [batch*3], positive, n_valid,
   pos_attempts, neg_draws [batch], negatives [batch*n_neg].
   Returns 0, or -1 on invalid arguments. */
int oracle_sample(const okg *g, int qtype, const oracle_args *a, int32_t *anchors,
                  int32_t *relations, int32_t *positive, int32_t *negatives, int32_t *n_valid,
                  int32_t *pos_attempts, int32_t *neg_draws, int nthreads);

/* Shared negatives of a minibatch (Sec. 4.3): positives as oracle_sample;
   shared [n_neg] = the first n_neg distinct values of the draws
   pick(U(3, query_offset, 0, j), V), j < neg_tries, in draw order, -1 padded,
   *n_shared = their number; mask [batch * ceil(n_neg / 32)] bit k % 32 of
   word k / 32 of row i set iff shared[k] is not an answer of query i;
   n_valid [batch] = set bits of the row, -1 for a query without a positive.
   Returns 0, or -1 on invalid arguments. */
int oracle_sample_shared(const okg *g, int qtype, const oracle_args *a, int32_t *anchors,
                         int32_t *relations, int32_t *positive, int32_t *pos_attempts,
                         int32_t *shared, int32_t *n_shared, uint32_t *mask, int32_t *n_valid,
                         int nthreads);

/* Membership verification of given candidates: candidates [batch * n];
   mask [batch * ceil(n / 32)] bit k of row i set iff candidate k of query i
   is an entity (0 <= c < V) outside the query's answer set; n_valid [batch]
   = set bits, or -1 when an anchor or relation the shape uses is out of
   range.  anchors/relations [batch * 3] as in oracle_sample.  Returns 0, or
   -1 on invalid arguments. */
int oracle_verify(const okg *g, int qtype, int32_t batch, int32_t n, const int32_t *anchors,
                  const int32_t *relations, const int32_t *candidates, uint32_t *mask,
                  int32_t *n_valid, int nthreads);

/* Exhaustive answer set of a grounded query; writes up to cap sorted ids to
   out and returns |A_q| (or -1 on bad input). */
int64_t oracle_answer_set(const okg *g, int qtype, const int32_t *anchors,
                          const int32_t *relations, int32_t *out, int64_t cap);

/* Bidirectional membership test of candidate c for the node cut given as a
   bit mask over the type's plan nodes.  Returns 1/0, or -1 if the mask is
   not a node cut.  counts (optional, 2 entries) receives the number of
   entities materialised by forward caching and the number visited by the
   backward expansion. */
int oracle_bidir_check(const okg *g, int qtype, const int32_t *anchors, const int32_t *relations,
                       uint32_t cut_mask, int32_t c, int64_t *counts);

/* Memory lines a bidirectional check of one query reads (Sec. 3.2, the
   cost of forward caching plus backward verification), on the device
   layout node[V+1] / grp[S+1] pairs / nbr[E] per direction with 64-byte
   lines: forward caching of every set of the node cut cut_mask, then for
   each candidate draw j < n_draws (pick(U(NEG, qid, 0, j), V)) the
   backward check from the candidate.  The rules of each read are stated
   with the definition in oracle.c.  lines[0]: distinct lines of the part
   a first verification pass makes (forward caching, each candidate's
   entity range and group search, edge tests against anchors, backward
   lists of at most 8 entries when the query's cached sets fit 1,024
   staged entries); lines[1]: distinct lines read below a longer list or
   with a set that does not fit; lines[2]: distinct lines of both.
   Returns 0, or -1 for a bad shape, ids out of range or a mask that is
   not a node cut. */
int oracle_verify_lines(const okg *g, int qtype, const int32_t *anchors, const int32_t *relations,
                        uint32_t cut_mask, uint64_t seed, uint32_t qid, int32_t n_draws,
                        int64_t *lines);

/* oracle_verify_lines for queries b < batch (anchors / relations [batch*3],
   positive [batch]: a row with positive < 0 has no query and gets zeros),
   query ids query_offset + b; lines [batch*3]. */
int oracle_verify_lines_batch(const okg *g, int qtype, int32_t batch, const int32_t *anchors,
                              const int32_t *relations, const int32_t *positive, uint32_t cut_mask,
                              uint64_t seed, uint64_t query_offset, int32_t n_draws, int64_t *lines,
                              int nthreads);

/* Projection set-building mode, for tests: 0 auto, 1 always sort-unique,
   2 always a bitmap over V.  Results are identical in every mode. */
void oracle_set_proj_mode(int mode);

/* Plan of a query type: n nodes in children-before-parent order.
   op[k] (0 anchor, 1 projection, 2 and, 3 or, 4 complement), child[3k..3k+2] (-1 unused),
   slot[k] (anchor slot, relation slot, or -1).  Returns n. */
int oracle_type_plan(int qtype, int32_t *op, int32_t *child, int32_t *slot, int32_t *root);

#ifdef __cplusplus
}
#endif
#endif
