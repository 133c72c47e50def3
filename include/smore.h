/*
 * smore.h -- C ABI of the MI355X sampler for multi-hop query training data
 * (SMORE, arXiv 2110.14890: reverse directional sampling of queries, Sec. 3.1,
 * and bidirectional rejection sampling of verified negatives, Sec. 3.2).
 *
 * Conventions
 *  - Every call returns SMORE_OK (0) or a negative SMORE_E_* code; on error
 *    smore_last_error() returns a message for the calling thread.  No C++
 *    exception crosses this boundary.
 *  - Arguments are validated synchronously on the host before any launch;
 *    an invalid call launches nothing and writes nothing.
 *  - Pointers named *_host are host memory, all other buffers are device
 *    memory allocated by the caller (for example torch tensors on the same
 *    device).  The library never frees caller memory.
 *  - smore_sample is asynchronous on the caller's HIP stream and returns
 *    without synchronising; results are valid once that stream reaches them.
 *  - All ids and outputs are int32.  Entity ids are in [0, V), relation ids
 *    in [0, R') where R' = 2R when the graph adds inverse relations.
 */
#ifndef SMORE_H
#define SMORE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    SMORE_OK = 0,
    SMORE_E_INVALID_ARG = -1, /* null pointer, bad size, bad query plan */
    SMORE_E_RANGE = -2,       /* an id outside [0, V) or [0, R) */
    SMORE_E_UNSUPPORTED = -3, /* plan outside the fourteen shapes, limits */
    SMORE_E_NOMEM = -4,       /* device or host allocation failed */
    SMORE_E_HIP = -5,         /* a HIP runtime call failed */
    SMORE_E_OVERFLOW = -6     /* counts beyond the int32 / 32-bit query-id range, or
                                 batch x neg_tries of 2^31 or more */
};

/* flags of smore_build_graph */
#define SMORE_ADD_INVERSE 1u /* also insert (t, r + R, h) for every (h, r, t) */

/* Node operators of a query computation plan (Sec. 2, "Query computation
   plan"; appendix on the computation plan).  Each node is a set of
   entities; a projection node applies one relation to its single child, an
   intersection / union node combines its children, a complement node is
   V minus its single child, an anchor is a leaf. */
enum { SMORE_OP_ANCHOR = 0, SMORE_OP_PROJ = 1, SMORE_OP_AND = 2, SMORE_OP_OR = 3, SMORE_OP_NOT = 4 };

/* One plan node.  child[] index earlier nodes of the same plan (children
   before parents).  slot: the anchor slot (0..2) of an anchor, the relation
   slot (0..2) of a projection, -1 otherwise. */
typedef struct {
    int32_t op, n_child, child[3], slot;
} smore_dag_node;

/* A plan tree: n_nodes nodes, root = the answer node V_?. */
typedef struct {
    int32_t n_nodes, root;
    smore_dag_node node[16];
} smore_query_dag;

/* Arguments of one sampling call.
   batch        number of queries B (>= 1)
   n_neg        negatives wanted per query (>= 0)
   pos_tries    reverse-sampling attempts per query (>= 1)
   neg_tries    candidate draws per query (>= n_neg, <= SMORE_MAX_NEG_TRIES)
   max_fanout   0, or reject a grounding whose step (x, r) -> e has
                |A_r(x)| > max_fanout (the paper's per-relation expansion C)
   seed         64-bit key of the counter-based draws
   query_offset query q of this call has id query_offset + q; the result of
                a query depends only on (graph, plan, seed, id, counts), so a
                batch split over several calls gives identical rows
   flags        0 (reserved) */
typedef struct {
    int32_t batch, n_neg, pos_tries, neg_tries, max_fanout;
    uint64_t seed, query_offset;
    uint32_t flags;
} smore_sample_args;

#define SMORE_MAX_NEG_TRIES 4096

/* Caller-owned device outputs, int32, row-major.
   anchors   [B,3]   anchor entities by slot, -1 for unused slots
   relations [B,3]   relations by slot, -1 for unused slots
   positive  [B]     the answer entity grounded at the root
   negatives [B,n_neg] verified non-answers in draw order, -1 padded
   n_valid   [B]     number of negatives found; -1 if no positive was found
   pos_attempts [B]  attempts used (1-based); pos_tries when none succeeded
   neg_draws [B]     draws consumed: 1 + index of the n_neg-th accepted
                     draw, else neg_tries; 0 when n_neg = 0; -1 with no positive
   All seven pointers are required. */
typedef struct {
    int32_t *anchors, *relations, *positive, *negatives, *n_valid, *pos_attempts, *neg_draws;
} smore_sample_out;

typedef struct smore_graph smore_graph; /* opaque; owns its device arrays */

/* Build forward and reverse adjacency on the current HIP device from
   n_triples host triples (h, r, t) (int32 [n_triples, 3]).  The KG is a set
   of triples (Sec. 2), so duplicates are removed.  Adjacency is grouped by
   (entity, relation) with ascending relations per entity and ascending
   neighbours per group, as sorted lists (appendix on the optimal cut: sets
   kept as sorted lists).  Errors: SMORE_E_RANGE for an id outside
   [0, n_entities) / [0, n_relations); SMORE_E_OVERFLOW when the edge count
   (doubled with SMORE_ADD_INVERSE) reaches 2^31; SMORE_E_NOMEM; SMORE_E_HIP.
   Synchronous.  *out must be released with smore_free_graph. */
int smore_build_graph(const int32_t *triples_host, int64_t n_triples, int32_t n_entities,
                      int32_t n_relations, uint32_t flags, smore_graph **out);

/* Sizes of a built graph (any pointer may be NULL): entities, relations
   (after inverse), unique edges, forward and reverse (entity, relation)
   groups, device bytes held. */
int smore_graph_info(const smore_graph *g, int64_t *n_entities, int64_t *n_relations,
                     int64_t *n_edges, int64_t *n_seg_fwd, int64_t *n_seg_rev,
                     int64_t *device_bytes);

/* Copy one device array of the graph to host memory (for tests and
   inspection).  which: 0 fwd node_ptr [V+1], 1 fwd groups [2*(S_fwd+1)]
   (relation, first edge) pairs, 2 fwd neighbours [E], 3 rev node_ptr,
   4 rev groups, 5 rev neighbours, 6 active_in (entities with an in-edge,
   ascending), 7 in-edge mask [(V+31)/32] (bit v % 32 of word v / 32 set
   iff entity v has an in-edge), 8 coarse in-edge mask [(V+127)/128] (bit
   i % 32 of word i / 32 set iff one of entities 4i .. 4i+3 has an in-edge),
   9 in-relation signatures [(V+3)/4] (byte v % 4 of word v / 4, little
   endian, is entity v's: bit (r * 0x9E3779B1 mod 2^32) >> 29 set for each
   relation r of its in-edges, 0 for an entity without in-edges).
   count must equal the array length.
   Synchronous. */
int smore_graph_copy(const smore_graph *g, int32_t which, int32_t *host_dst, int64_t count);

/* Fill *out with one of the fourteen query structures of BetaE (Sec. 5.1):
   the nine without negation "1p" "2p" "3p" "2i" "3i" "ip" "pi" "2u" "up",
   and "2in" "3in" "inp" "pin" "pni", where one operand of the intersection
   is complemented (2in, 3in, inp, pin: the last one-hop operand; pni: the
   two-hop operand).  Anchor and relation slots follow branch order, and
   within a branch run from the anchor to the root. */
int smore_query_preset(const char *name, smore_query_dag *out);

/* Node cut of a plan tree minimising the worst per-anchor-path cost
   max(C^i, C^(t-i)) (Sec. 3.2, Def. "Node cut" and the optimal-scheduling
   equation), by the dynamic program of the appendix on the optimal cut
   (u = projections to the root, s = longest projection path to an anchor,
   o = best cost) and its top-down construction.  tie_break 0 adds a node
   when the children's best cost exceeds its own (as stated); 1 also adds it
   on equality, which caches as far forward as the same cost allows.
   cut_nodes receives up to 16 node indices; *n_cut their number. */
int smore_plan(const smore_query_dag *dag, int32_t tie_break, int32_t *cut_nodes, int32_t *n_cut);

/* Bytes of device workspace smore_sample / smore_sample_negatives need for
   these arguments (it grows with batch * neg_tries: per-draw candidate ids
   and states, the queue of long intersections, the lists of queries still
   short of n_neg).  The caller allocates it; its contents need no
   initialisation and are scratch after the call.  Calls that may overlap on
   the device must not share a workspace.  A call with n_neg = 0 draws no
   candidates and needs no workspace (NULL and 0 are accepted). */
int smore_sample_workspace_bytes(const smore_graph *g, const smore_query_dag *dag,
                                 const smore_sample_args *args, size_t *bytes);

/* Sample args->batch queries of shape dag with one positive each and up to
   n_neg verified negatives (Sec. 3.1 reverse directional sampling; Sec. 3.2
   bidirectional rejection sampling with a constant candidate budget).
   Per query id q: attempt t grounds the root uniformly among entities with
   an in-edge, then walks from the root to the anchors in pre-order, each
   projection picking an in-relation uniformly and then an in-neighbour
   uniformly; the first attempt without a dead end, a repeated
   (anchor, relation) pair among single-projection siblings, or a step wider
   than max_fanout wins.  Candidate j (j < neg_tries) is uniform over all V
   entities and is kept iff it is not an answer of the query and was not
   drawn earlier; the first n_neg kept are returned.  Draws come from
   Philox4x32-10 with counter (j, t, q, tag) and key seed.
   A complemented operand of an intersection (the negation shapes) is
   grounded after the positive operands, from a sibling entity w drawn
   uniformly from A_r(x) of the first positive operand's step (x, r) -> e;
   the attempt is also rejected when e lies in the complemented set, so the
   root is always an answer.  Draws are numbered in grounding order (root,
   two per projection, one for w).  The plan must be one of the fourteen
   presets (SMORE_E_UNSUPPORTED otherwise).  hip_stream: a hipStream_t, or
   NULL for the default stream. */
int smore_sample(const smore_graph *g, const smore_query_dag *dag, const smore_sample_args *args,
                 const smore_sample_out *out, void *workspace, size_t ws_bytes, void *hip_stream);

/* smore_sample for callers that cannot allocate device memory (code under
   HIP graph capture, tight serving loops, harnesses that forbid
   allocation): the same arguments, validation, outputs and stream
   semantics, but no workspace argument.  The scratch is a fixed array of
   SMORE_NOALLOC_SCRATCH_BYTES in device memory, one per GPU the library
   runs on, held until the process ends; the call itself allocates and
   frees nothing.  Every call on one GPU shares that array, so calls that
   may overlap on a GPU (different streams, different threads) race and
   must be serialised by the caller; the array keeps the last call's
   contents, and each call initialises whatever it reads.  Errors as for
   smore_sample, and SMORE_E_UNSUPPORTED when the arguments need more
   scratch than the fixed size (smore_sample_workspace_bytes gives the
   need; about 15 KB per query at 512 negatives and 2,048 draws, e.g.
   4,096 such queries, or 16,384 queries with 64 negatives and 256
   draws). */
#define SMORE_NOALLOC_SCRATCH_BYTES (64u << 20)
int smore_sample_noalloc(const smore_graph *g, const smore_query_dag *dag,
                         const smore_sample_args *args, const smore_sample_out *out,
                         void *hip_stream);

/* The two stages of smore_sample, for callers that time or feed them
   separately.  Same arguments and validation as smore_sample.
   smore_sample_positives writes anchors, relations, positive, pos_attempts
   and n_valid (-1 for a query without a positive, else 0).
   smore_sample_negatives reads anchors, relations and positive (a row with
   positive < 0, or with an anchor or relation id used by the shape outside
   the graph's range, is skipped: negatives -1, n_valid -1, neg_draws -1) and
   writes negatives, n_valid and neg_draws; it may be run on queries built
   by the caller.  stats is NULL or a device int64 [batch, 4] array that
   receives, per query, the bytes and the 64-byte lines of graph data the
   verification read: [0], [1] in the candidate kernel (forward-cached lists
   once per query, then every read made from a candidate's side), [2], [3]
   in the kernel that intersects long lists; lookups inside forward-cached
   lists are cache hits of the method and are not counted.  Counting makes
   the call slower and does not change any other output.  workspace /
   ws_bytes as for smore_sample (smore_sample_positives needs none). */
int smore_sample_positives(const smore_graph *g, const smore_query_dag *dag,
                           const smore_sample_args *args, const smore_sample_out *out,
                           void *hip_stream);
int smore_sample_negatives(const smore_graph *g, const smore_query_dag *dag,
                           const smore_sample_args *args, const smore_sample_out *out,
                           int64_t *stats, void *workspace, size_t ws_bytes, void *hip_stream);

/* smore_sample_negatives in three parts, for callers that schedule the
   first round's candidate kernel (the verification of the first batch of
   rejection-sampling draws, Sec. 3.2) apart from the rest, e.g. the
   candidate kernels of several calls back to back on one stream:
   part 0 the per-query preparation, part 1 the first round's candidate
   kernel, part 2 the rest (long lists, ordered selection, later rounds).
   Calling parts 0, 1 and 2 with the same arguments, outputs and workspace,
   each after the previous one has completed in stream order (on one stream,
   or ordered by the caller's events across streams), has exactly the effect
   of one smore_sample_negatives call; the outputs are final only after
   part 2.  The workspace carries state from part to part: it must not be
   used by any other call in between.  stats, the instrumentation hooks and
   errors as for smore_sample_negatives (smore_profile_kernel's candidate
   kernel and smore_wait_before_kernel act in part 1; any part disarms
   them).  SMORE_E_INVALID_ARG for another part. */
int smore_sample_negatives_part(const smore_graph *g, const smore_query_dag *dag,
                                const smore_sample_args *args, const smore_sample_out *out,
                                int64_t *stats, int32_t part, void *workspace, size_t ws_bytes,
                                void *hip_stream);

/* Caller-owned device outputs of smore_sample_shared, int32 unless noted.
   anchors [B,3], relations [B,3], positive [B], pos_attempts [B]
                     as in smore_sample_out
   shared   [n_neg]  the minibatch's candidate set N, in draw order, -1 padded
   n_shared [1]      |N|: n_neg, or fewer when neg_tries draws hold fewer
                     distinct entities
   mask     uint32 [B, (n_neg + 31) / 32]: bit k % 32 of word k / 32 of row i
                     is set iff N[k] is a verified non-answer of query i
   n_valid  [B]      set bits of row i; -1 for a query without a positive
                     (its row is zero)
   All pointers are required (shared and mask may be NULL when n_neg = 0). */
typedef struct {
    int32_t *anchors, *relations, *positive, *pos_attempts, *shared, *n_shared;
    uint32_t *mask;
    int32_t *n_valid;
} smore_shared_out;

/* A minibatch whose queries share one set of candidate negatives (Sec. 4.3,
   sharing negative samples): one candidate set N for all args->batch
   queries and a mask saying, per query, which members of N are negatives.
   The positives are exactly those of smore_sample with the same arguments.
   N holds the first n_neg distinct values of the draws
   pick(U(3, query_offset, 0, j), V), j < neg_tries (Philox counter
   (j, 0, low 32 bits of query_offset, 3)), so different minibatches
   (query_offset) draw different sets.  Every (query, member) pair is
   verified by the same bidirectional test as smore_sample.  Arguments,
   validation and workspace (smore_sample_workspace_bytes with the same
   args) as for smore_sample; asynchronous on hip_stream.  With n_neg = 0
   the set is empty (*n_shared = 0), no mask word exists, n_valid is 0 (or
   -1 without a positive) and no workspace is needed. */
int smore_sample_shared(const smore_graph *g, const smore_query_dag *dag,
                        const smore_sample_args *args, const smore_shared_out *out,
                        void *workspace, size_t ws_bytes, void *hip_stream);

/* Membership verification of caller-given candidates: for every query i
   (anchors / relations [B,3], device, as smore_sample writes them) and
   each of its n = args->n_neg candidates (device int32 [B, n]), is the
   candidate an entity outside the query's answer set?  This is the test
   behind rejection sampling (Sec. 3.2, bidirectional), run here on given
   pairs - for evaluation, where a query's answers differ between nested
   graphs G_train, G_valid, G_test (appendix on the task setup): verifying
   the positives of queries sampled on G_test against G_valid finds the
   answers missing from G_valid.
   mask  uint32 [B, (n + 31) / 32]: bit k % 32 of word k / 32 of row i set
         iff candidate k of query i is in [0, V) and not an answer
   n_valid [B]: set bits of row i; -1 when an anchor or relation the shape
         uses is out of range (row zero)
   Candidates outside [0, V) are never negatives and read no graph data.
   args: batch = B, n_neg = n, neg_tries >= n (workspace sizing as for
   smore_sample, see smore_sample_workspace_bytes); the other fields are
   checked as for smore_sample but unused.  With n = 0 only n_valid is
   written (0, or -1 as above) and candidates, mask and the workspace may
   be NULL.  Asynchronous on hip_stream. */
int smore_verify(const smore_graph *g, const smore_query_dag *dag, const smore_sample_args *args,
                 const int32_t *anchors, const int32_t *relations, const int32_t *candidates,
                 uint32_t *mask, int32_t *n_valid, void *workspace, size_t ws_bytes,
                 void *hip_stream);

/* Instrumentation: the next smore_sample or smore_sample_negatives call
   made by this thread records the caller's HIP events (hipEvent_t) on its
   stream immediately before and after one of its kernels in the first
   round of candidate draws: which = 0 the candidate kernel, 1 the kernels
   that intersect long lists (for 3p the batched long-list kernel and the
   kernel of its units, timed together), 2 the ordered selection.  Each `which` has
   its own arm, so one call can time several kernels.  One-shot: the
   next smore_sample, smore_sample_negatives or smore_sample_negatives_part
   call of this thread disarms all of them whether or not they recorded,
   also when that call fails validation.  Either event NULL disarms that
   `which`.  The events stay owned by the
   caller.  Returns SMORE_E_INVALID_ARG for another `which`. */
int smore_profile_kernel(void *start_event, void *stop_event, int32_t which);

/* Scheduling, for callers that run several sampling calls on different
   streams and want their candidate kernels one after another: the next
   smore_sample or smore_sample_negatives call made by this thread makes its
   stream wait on the caller's HIP event (hipEvent_t) right before its
   first candidate kernel (which = 0), after the per-query preparation, so
   the preparation does not wait.  One-shot: the next such call (or
   smore_sample_negatives_part) disarms it, also when it launches no
   candidate kernel (n_neg = 0) or fails validation.  NULL disarms.
   The event stays owned by the caller.  SMORE_E_INVALID_ARG for another
   `which`; SMORE_E_HIP if the wait cannot be enqueued (the call then
   launches nothing after the preparation). */
int smore_wait_before_kernel(void *event, int32_t which);

/* Instrumentation: n_reads random 4-byte reads from the device table of
   table_bytes (the first word of pseudo-randomly chosen 64-byte lines among
   the largest power-of-two number of lines that fits), eight independent
   reads in flight per lane, folded into sink (device uint32, at least
   (n_reads + 63) / 64 words, overwritten).  The rate of this kernel is the
   device's random-read ceiling that the sampler's gathers are compared
   with; it is not part of sampling.  Asynchronous on hip_stream.  Errors:
   SMORE_E_INVALID_ARG for null pointers, a table under 64 bytes, n_reads
   outside [1, 2^40] or a short sink. */
int smore_gather_probe(const void *table, int64_t table_bytes, int64_t n_reads, uint32_t *sink,
                       int64_t sink_words, void *hip_stream);

/* Release a graph (NULL is a no-op). */
void smore_free_graph(smore_graph *g);

/* Message of the last failed call on this thread ("" if none). */
const char *smore_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SMORE_H */
