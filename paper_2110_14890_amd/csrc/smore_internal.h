// smore_internal.h -- types shared by the host C ABI and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/smore.h"

namespace smore {

// Device-resident adjacency of one direction (forward: entity -> tails by
// relation; reverse: entity -> heads by relation).
//   node[v] .. node[v+1]   : groups (one per relation) of entity v, v in [0, V]
//   grp[g] = (relation, first edge); grp[S] = (INT32_MAX, E) is a sentinel so
//            that group g spans edges [grp[g].y, grp[g+1].y)
//   nbr[e]                 : neighbour entity of edge e, ascending in a group
struct DirView {
    const int32_t* node;
    const int2* grp;
    const int32_t* nbr;
};

struct GraphView {
    DirView fwd, rev;
    const int32_t* active_in;  // entities with an in-edge, ascending
    const uint32_t* has_in;    // bit v: entity v has an in-edge (V bits, cache-resident)
    const uint32_t* has_in4;   // bit i: one of entities 4i .. 4i + 3 has an in-edge (V / 4 bits)
    const uint8_t* sig;        // in-relation signature of entity v: bit sig_bit(r) set for
                               // each relation r of its in-edges (V bytes, 0 without in-edge)
    int32_t coarse;            // test has_in4, then sig (when has_in outgrows the L2)
    int32_t V;
    int32_t n_active;
};

// Positive-sampling program compiled from a plan on the host: the
// projection steps in grounding order (pre-order, an intersection's
// positive operands before its complemented one).  Register 0 holds the
// root; step k reads register src[k], grounds relation slot rel_slot[k]
// and writes register k + 1.  Anchor slot a takes register anchor_reg[a].
// Pairs of single-projection siblings under an intersection or union must
// differ in (anchor, relation).
//
// A complemented operand (neg_steps > 0): before step neg_first, register
// WALK_SIB takes the sibling entity w, one draw uniform over A_r(x) of
// step sib_step ((x, r) = its register sib_step + 1 and its relation);
// steps neg_first .. neg_first + neg_steps - 1 ground the operand from w;
// after the walk, register neg_target must lie outside the operand's set,
// the chain from anchor slot neg_anchor through relation slots neg_rel[0]
// (innermost) .. neg_rel[neg_steps - 1].  Draws are numbered in grounding
// order: 0 for the root, two per step, one for w.
constexpr int WALK_SIB = 4;
struct WalkProgram {
    int32_t n_steps;
    int32_t src[3];
    int32_t rel_slot[3];
    int32_t n_anchor;
    int32_t anchor_reg[3];
    int32_t n_pairs;
    int32_t pair_anchor[3][2];
    int32_t pair_rel[3][2];
    int32_t neg_steps, neg_first, sib_step, neg_target, neg_anchor;
    int32_t neg_rel[2];
    int32_t root_pairs;   // of the pairs, those whose siblings hang off the root entity
};

// Query shapes with a dedicated verification kernel: the nine without
// negation, then 2in 3in inp pin pni.
enum QType { Q1P = 0, Q2P, Q3P, Q2I, Q3I, QIP, QPI, Q2U, QUP, Q2IN, Q3IN, QINP, QPIN, QPNI, NQTYPE };

struct SampleParams {
    int32_t batch, n_neg, pos_tries, neg_tries, max_fanout;
    uint64_t seed, query_offset;
    // shared-candidate minibatches (shared_mode 1): the candidate set and its
    // size (device; the set is NULL when it is empty); per-query negatives
    // have shared_mode 0 and write per-query rows and draw counts instead
    int32_t shared_mode = 0;
    const int32_t* shared = nullptr;
    const int32_t* n_shared = nullptr;
    // candidates of query b start at shared + cand_stride * b (0: one set for
    // all queries); without n_shared every query has n_neg candidates, and
    // ids outside [0, V) are never negatives
    int32_t cand_stride = 0;
};

}  // namespace smore

// Bit of relation r in an entity's in-relation signature (eight classes,
// multiplicative hash of the relation id).
__host__ __device__ inline uint32_t sig_bit(int32_t r)
{
    return 1u << (((uint32_t)r * 0x9E3779B1u) >> 29);
}

struct smore_graph {
    int device;
    int32_t V, R;
    int64_t E, S_fwd, S_rev, n_active;
    int32_t *f_node, *f_nbr, *r_node, *r_nbr, *active_in;
    int2 *f_grp, *r_grp;
    uint32_t *has_in, *has_in4;
    uint8_t* sig;
    size_t bytes;
};

// Entry points implemented in the .hip files (host side, C++ linkage).
namespace smore {
int build_graph_device(const int32_t* triples_host, int64_t n, int32_t V, int32_t R,
                       bool add_inverse, smore_graph* g, const char** err);
int launch_positive(const smore_graph* g, const WalkProgram& wp, const SampleParams& p,
                    const smore_sample_out& out, hipStream_t stream, const char** err);
// Parts of the negative stage (bit masks for launch_negative).
constexpr int NEG_PREPARE = 1, NEG_CANDIDATES = 2, NEG_REST = 4, NEG_ALL = 7;
int launch_negative(const smore_graph* g, QType qt, const SampleParams& p,
                    const smore_sample_out& out, int64_t* stats, void* workspace, size_t ws_bytes,
                    int parts, hipStream_t stream, const char** err);
size_t negatives_workspace_bytes(const SampleParams& p);
int launch_shared(const smore_graph* g, QType qt, const SampleParams& p, const smore_sample_out& pos,
                  int32_t* shared, int32_t* n_shared, uint32_t* mask, void* workspace,
                  size_t ws_bytes, hipStream_t stream, const char** err);
int launch_verify(const smore_graph* g, QType qt, const SampleParams& p, const int32_t* anchors,
                  const int32_t* relations, const int32_t* candidates, uint32_t* mask,
                  int32_t* n_valid, void* workspace, size_t ws_bytes, hipStream_t stream,
                  const char** err);
// one-shot event pair recorded around one kernel of the next negatives call
void arm_profile(void* start_event, void* stop_event, int which);
// one-shot wait on an event before the first candidate kernel of the next negatives call
void arm_wait(void* event);
// clear both one-shot arms of the calling thread
void disarm();
// the current device's fixed scratch (SMORE_NOALLOC_SCRATCH_BYTES bytes)
int scratch_workspace(void** ptr, size_t* bytes, const char** err);
int64_t gather_probe_threads(int64_t n_reads);
int launch_gather_probe(const void* table, int64_t table_bytes, int64_t n_reads, uint32_t* sink,
                        hipStream_t st, const char** err);
}  // namespace smore
