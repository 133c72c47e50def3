// capi.cpp -- host side of the C ABI declared in include/smore.h: argument
// validation, the fourteen plan presets, the node-cut planner, compilation of a
// plan into the positive-sampling program, and graph handle management.
// Device work is in graph_build.hip and sample.hip.
#include <hip/hip_runtime.h>

#include <climits>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>

#include "smore_internal.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int ok()
{
    g_err.clear();
    return SMORE_OK;
}

// ----------------------------------------------------------- plan presets
// The fourteen query structures of the experiments (Sec. 5.1, the shapes
// of BetaE) as computation-plan trees, children listed before parents: nine
// without negation, then five whose intersection has one complemented
// operand (complement is a plan operator, appendix on the computation plan).
smore_dag_node anchor(int slot) { return {SMORE_OP_ANCHOR, 0, {-1, -1, -1}, slot}; }
smore_dag_node proj(int c, int slot) { return {SMORE_OP_PROJ, 1, {c, -1, -1}, slot}; }
smore_dag_node both(int op, int a, int b) { return {op, 2, {a, b, -1}, -1}; }
smore_dag_node neg(int c) { return {SMORE_OP_NOT, 1, {c, -1, -1}, -1}; }

struct Preset {
    const char* name;
    smore::QType qt;
    int n;
    smore_dag_node nd[8];
};

const Preset kPresets[smore::NQTYPE] = {
    {"1p", smore::Q1P, 2, {anchor(0), proj(0, 0)}},
    {"2p", smore::Q2P, 3, {anchor(0), proj(0, 0), proj(1, 1)}},
    {"3p", smore::Q3P, 4, {anchor(0), proj(0, 0), proj(1, 1), proj(2, 2)}},
    {"2i", smore::Q2I, 5, {anchor(0), proj(0, 0), anchor(1), proj(2, 1), both(SMORE_OP_AND, 1, 3)}},
    {"3i", smore::Q3I, 7,
     {anchor(0), proj(0, 0), anchor(1), proj(2, 1), anchor(2), proj(4, 2),
      {SMORE_OP_AND, 3, {1, 3, 5}, -1}}},
    {"ip", smore::QIP, 6,
     {anchor(0), proj(0, 0), anchor(1), proj(2, 1), both(SMORE_OP_AND, 1, 3), proj(4, 2)}},
    {"pi", smore::QPI, 6,
     {anchor(0), proj(0, 0), proj(1, 1), anchor(1), proj(3, 2), both(SMORE_OP_AND, 2, 4)}},
    {"2u", smore::Q2U, 5, {anchor(0), proj(0, 0), anchor(1), proj(2, 1), both(SMORE_OP_OR, 1, 3)}},
    {"up", smore::QUP, 6,
     {anchor(0), proj(0, 0), anchor(1), proj(2, 1), both(SMORE_OP_OR, 1, 3), proj(4, 2)}},
    {"2in", smore::Q2IN, 6,
     {anchor(0), proj(0, 0), anchor(1), proj(2, 1), neg(3), both(SMORE_OP_AND, 1, 4)}},
    {"3in", smore::Q3IN, 8,
     {anchor(0), proj(0, 0), anchor(1), proj(2, 1), anchor(2), proj(4, 2), neg(5),
      {SMORE_OP_AND, 3, {1, 3, 6}, -1}}},
    {"inp", smore::QINP, 7,
     {anchor(0), proj(0, 0), anchor(1), proj(2, 1), neg(3), both(SMORE_OP_AND, 1, 4), proj(5, 2)}},
    {"pin", smore::QPIN, 7,
     {anchor(0), proj(0, 0), proj(1, 1), anchor(1), proj(3, 2), neg(4), both(SMORE_OP_AND, 2, 5)}},
    {"pni", smore::QPNI, 7,
     {anchor(0), proj(0, 0), proj(1, 1), neg(2), anchor(1), proj(4, 2), both(SMORE_OP_AND, 3, 5)}},
};

// Node cut the verification kernel of each shape is written for: the cut the
// planner returns with tie_break 0 on the preset (node indices).
const int kKernelCut[smore::NQTYPE][4] = {
    {1, 0}, {1, 1}, {1, 1}, {2, 0, 2}, {3, 0, 2, 4}, {2, 1, 3}, {2, 1, 3}, {2, 0, 2}, {2, 1, 3},
    {2, 0, 2}, {3, 0, 2, 4}, {2, 1, 3}, {2, 1, 3}, {2, 1, 4},
};

// Structural validation: a tree whose children precede their parent, with
// arities and slots that fit the operators.
int check_dag(const smore_query_dag* d)
{
    if (!d) return fail(SMORE_E_INVALID_ARG, "query plan is NULL");
    if (d->n_nodes < 1 || d->n_nodes > 16)
        return fail(SMORE_E_INVALID_ARG, "plan has %d nodes (1..16 allowed)", d->n_nodes);
    if (d->root < 0 || d->root >= d->n_nodes)
        return fail(SMORE_E_INVALID_ARG, "plan root %d out of range", d->root);
    int parents[16] = {0};
    for (int k = 0; k < d->n_nodes; ++k) {
        const smore_dag_node& nd = d->node[k];
        int need_lo, need_hi;
        switch (nd.op) {
            case SMORE_OP_ANCHOR: need_lo = need_hi = 0; break;
            case SMORE_OP_PROJ:
            case SMORE_OP_NOT: need_lo = need_hi = 1; break;
            case SMORE_OP_AND:
            case SMORE_OP_OR: need_lo = 2; need_hi = 3; break;
            default: return fail(SMORE_E_INVALID_ARG, "node %d has unknown operator %d", k, nd.op);
        }
        if (nd.n_child < need_lo || nd.n_child > need_hi)
            return fail(SMORE_E_INVALID_ARG, "node %d: operator %d with %d children", k, nd.op,
                        nd.n_child);
        for (int c = 0; c < nd.n_child; ++c) {
            if (nd.child[c] < 0 || nd.child[c] >= k)
                return fail(SMORE_E_INVALID_ARG, "node %d: child %d must index an earlier node", k,
                            nd.child[c]);
            parents[nd.child[c]]++;
        }
        if ((nd.op == SMORE_OP_ANCHOR || nd.op == SMORE_OP_PROJ) && (nd.slot < 0 || nd.slot > 2))
            return fail(SMORE_E_INVALID_ARG, "node %d: slot %d outside 0..2", k, nd.slot);
    }
    for (int k = 0; k < d->n_nodes; ++k) {
        const int want = k == d->root ? 0 : 1;
        if (parents[k] != want)
            return fail(SMORE_E_INVALID_ARG, "node %d has %d parents; a plan must be a tree", k,
                        parents[k]);
    }
    return SMORE_OK;
}

bool same_dag(const smore_query_dag* d, const Preset& p)
{
    if (d->n_nodes != p.n || d->root != p.n - 1) return false;
    for (int k = 0; k < p.n; ++k) {
        const smore_dag_node &a = d->node[k], &b = p.nd[k];
        if (a.op != b.op || a.n_child != b.n_child) return false;
        for (int c = 0; c < a.n_child; ++c)
            if (a.child[c] != b.child[c]) return false;
        if ((a.op == SMORE_OP_ANCHOR || a.op == SMORE_OP_PROJ) && a.slot != b.slot) return false;
    }
    return true;
}

// ------------------------------------------------------------------ planner
// Dynamic program of the appendix on the optimal node cut.
//   u(v): relation projections between v and the root
//         (u(root) = 0; u(v) = u(p(v)) + IsRel(v -> p(v))),
//   s(v): longest projection count from v down to an anchor
//         (0 at anchors; max over children across AND/OR; s(child) + 1
//         across a projection, + 0 across a negation),
//   o(v): best cost of the paths through v (u(v) at an anchor, else
//         min(max over children o(z), max(u(v), s(v)))).
// The cut is built top-down: v joins the cut when the children's best
// cost exceeds max(u(v), s(v)) (tie_break 1: or equals it); otherwise the
// children are examined; an anchor reached by the descent joins the cut.
struct Planner {
    const smore_query_dag* d;
    int parent[16], u[16], s[16], o[16];
    int tie;
    int cut[16], n_cut;

    int best_child(int v) const
    {
        int m = INT_MIN;
        for (int c = 0; c < d->node[v].n_child; ++c) m = o[d->node[v].child[c]] > m ? o[d->node[v].child[c]] : m;
        return m;
    }

    void run()
    {
        const int n = d->n_nodes;
        for (int k = 0; k < n; ++k) parent[k] = -1;
        for (int k = 0; k < n; ++k)
            for (int c = 0; c < d->node[k].n_child; ++c) parent[d->node[k].child[c]] = k;
        // u top-down: parents have larger indices than children
        for (int k = n - 1; k >= 0; --k)
            u[k] = parent[k] < 0 ? 0 : u[parent[k]] + (d->node[parent[k]].op == SMORE_OP_PROJ ? 1 : 0);
        // s and o bottom-up
        for (int k = 0; k < n; ++k) {
            const smore_dag_node& nd = d->node[k];
            if (nd.op == SMORE_OP_ANCHOR) {
                s[k] = 0;
                o[k] = u[k];
                continue;
            }
            if (nd.op == SMORE_OP_AND || nd.op == SMORE_OP_OR) {
                int m = 0;
                for (int c = 0; c < nd.n_child; ++c) m = s[nd.child[c]] > m ? s[nd.child[c]] : m;
                s[k] = m;
            } else {
                s[k] = s[nd.child[0]] + (nd.op == SMORE_OP_NOT ? 0 : 1);
            }
            const int own = u[k] > s[k] ? u[k] : s[k];
            const int bc = best_child(k);
            o[k] = bc < own ? bc : own;
        }
        n_cut = 0;
        descend(d->root);
    }

    void descend(int v)
    {
        const smore_dag_node& nd = d->node[v];
        if (nd.op == SMORE_OP_ANCHOR) {
            cut[n_cut++] = v;
            return;
        }
        const int own = u[v] > s[v] ? u[v] : s[v];
        const int bc = best_child(v);
        if (bc > own || (tie && bc == own)) {
            cut[n_cut++] = v;
            return;
        }
        for (int c = 0; c < nd.n_child; ++c) descend(nd.child[c]);
    }
};

// Walk program of reverse directional sampling (Sec. 3.1): pre-order, an
// intersection's positive operands first; its complemented operand (the
// presets have at most one, a chain of projections down to an anchor) is
// grounded from the sibling entity drawn from the first positive operand's
// step (the oracle's reading of how a negated operand is grounded).
void compile_walk(const smore_query_dag* d, int v, int reg, smore::WalkProgram* w)
{
    const smore_dag_node& nd = d->node[v];
    if (nd.op == SMORE_OP_ANCHOR) {
        w->anchor_reg[nd.slot] = reg;
        if (nd.slot + 1 > w->n_anchor) w->n_anchor = nd.slot + 1;
        return;
    }
    if (nd.op == SMORE_OP_PROJ) {
        const int k = w->n_steps++;
        w->src[k] = reg;
        w->rel_slot[k] = nd.slot;
        compile_walk(d, nd.child[0], k + 1, w);
        return;
    }
    if (nd.op == SMORE_OP_NOT) {
        compile_walk(d, nd.child[0], reg, w);
        return;
    }
    int first_pos = -1;
    for (int c = 0; c < nd.n_child; ++c) {
        if (d->node[nd.child[c]].op == SMORE_OP_NOT) continue;
        if (first_pos < 0) first_pos = w->n_steps;
        compile_walk(d, nd.child[c], reg, w);
    }
    for (int c = 0; c < nd.n_child; ++c) {
        const int n = nd.child[c];
        if (d->node[n].op != SMORE_OP_NOT) continue;
        w->neg_first = w->n_steps;
        w->sib_step = first_pos;
        w->neg_target = reg;
        compile_walk(d, n, smore::WALK_SIB, w);
        w->neg_steps = w->n_steps - w->neg_first;
        // the operand's chain: relations outermost first, then its anchor
        int x = d->node[n].child[0], depth = 0, rels[2] = {-1, -1};
        while (d->node[x].op == SMORE_OP_PROJ && depth < 2) {
            rels[depth++] = d->node[x].slot;
            x = d->node[x].child[0];
        }
        w->neg_anchor = d->node[x].slot;
        for (int k = 0; k < depth; ++k) w->neg_rel[k] = rels[depth - 1 - k];
    }
    for (int a = 0; a < nd.n_child; ++a)
        for (int b = a + 1; b < nd.n_child; ++b) {
            const smore_dag_node &x = d->node[nd.child[a]], &y = d->node[nd.child[b]];
            if (x.op != SMORE_OP_PROJ || y.op != SMORE_OP_PROJ) continue;
            const smore_dag_node &xa = d->node[x.child[0]], &ya = d->node[y.child[0]];
            if (xa.op != SMORE_OP_ANCHOR || ya.op != SMORE_OP_ANCHOR) continue;
            const int p = w->n_pairs++;
            if (reg == 0) ++w->root_pairs;
            w->pair_anchor[p][0] = xa.slot;
            w->pair_anchor[p][1] = ya.slot;
            w->pair_rel[p][0] = x.slot;
            w->pair_rel[p][1] = y.slot;
        }
}

}  // namespace

extern "C" {

const char* smore_last_error(void) { return g_err.c_str(); }

int smore_query_preset(const char* name, smore_query_dag* out)
{
    if (!name || !out) return fail(SMORE_E_INVALID_ARG, "NULL argument");
    for (const Preset& p : kPresets)
        if (std::strcmp(p.name, name) == 0) {
            std::memset(out, 0, sizeof(*out));
            out->n_nodes = p.n;
            out->root = p.n - 1;
            for (int k = 0; k < p.n; ++k) out->node[k] = p.nd[k];
            return ok();
        }
    return fail(SMORE_E_UNSUPPORTED,
                "unknown query shape '%s' (1p 2p 3p 2i 3i ip pi 2u up 2in 3in inp pin pni)", name);
}

int smore_plan(const smore_query_dag* dag, int32_t tie_break, int32_t* cut_nodes, int32_t* n_cut)
{
    if (!cut_nodes || !n_cut) return fail(SMORE_E_INVALID_ARG, "NULL output");
    if (tie_break != 0 && tie_break != 1) return fail(SMORE_E_INVALID_ARG, "tie_break must be 0 or 1");
    int rc = check_dag(dag);
    if (rc) return rc;
    Planner P;
    P.d = dag;
    P.tie = tie_break;
    P.run();
    for (int k = 0; k < P.n_cut; ++k) cut_nodes[k] = P.cut[k];
    *n_cut = P.n_cut;
    return ok();
}

int smore_build_graph(const int32_t* triples_host, int64_t n_triples, int32_t n_entities,
                      int32_t n_relations, uint32_t flags, smore_graph** out)
{
    if (!out) return fail(SMORE_E_INVALID_ARG, "out is NULL");
    *out = nullptr;
    if (n_triples < 0) return fail(SMORE_E_INVALID_ARG, "n_triples < 0");
    if (n_triples > 0 && !triples_host) return fail(SMORE_E_INVALID_ARG, "triples_host is NULL");
    if (n_entities < 1 || n_relations < 1)
        return fail(SMORE_E_INVALID_ARG, "need n_entities >= 1 and n_relations >= 1");
    if (flags & ~SMORE_ADD_INVERSE) return fail(SMORE_E_INVALID_ARG, "unknown flags 0x%x", flags);
    const bool inv = (flags & SMORE_ADD_INVERSE) != 0;
    if (inv && (int64_t)n_relations * 2 > INT32_MAX - 1)
        return fail(SMORE_E_OVERFLOW, "2 * n_relations overflows int32");
    if ((inv ? 2 * n_triples : n_triples) >= (int64_t)INT32_MAX)
        return fail(SMORE_E_OVERFLOW, "edge count must stay below 2^31");
    if (n_entities == INT32_MAX) return fail(SMORE_E_OVERFLOW, "n_entities must be < 2^31 - 1");
    smore_graph* g = new (std::nothrow) smore_graph();
    if (!g) return fail(SMORE_E_NOMEM, "host allocation failed");
    const char* err = "";
    int rc = smore::build_graph_device(triples_host, n_triples, n_entities, n_relations, inv, g, &err);
    if (rc) {
        smore_free_graph(g);
        return fail(rc, "smore_build_graph: %s", err);
    }
    *out = g;
    return ok();
}

int smore_graph_info(const smore_graph* g, int64_t* v, int64_t* r, int64_t* e, int64_t* sf,
                     int64_t* sr, int64_t* bytes)
{
    if (!g) return fail(SMORE_E_INVALID_ARG, "graph is NULL");
    if (v) *v = g->V;
    if (r) *r = g->R;
    if (e) *e = g->E;
    if (sf) *sf = g->S_fwd;
    if (sr) *sr = g->S_rev;
    if (bytes) *bytes = (int64_t)g->bytes;
    return ok();
}

int smore_graph_copy(const smore_graph* g, int32_t which, int32_t* host_dst, int64_t count)
{
    if (!g || !host_dst) return fail(SMORE_E_INVALID_ARG, "NULL argument");
    const void* src = nullptr;
    int64_t n = 0;
    switch (which) {
        case 0: src = g->f_node; n = (int64_t)g->V + 1; break;
        case 1: src = g->f_grp; n = 2 * (g->S_fwd + 1); break;
        case 2: src = g->f_nbr; n = g->E; break;
        case 3: src = g->r_node; n = (int64_t)g->V + 1; break;
        case 4: src = g->r_grp; n = 2 * (g->S_rev + 1); break;
        case 5: src = g->r_nbr; n = g->E; break;
        case 6: src = g->active_in; n = g->n_active; break;
        case 7: src = g->has_in; n = ((int64_t)g->V + 31) / 32; break;
        case 8: src = g->has_in4; n = ((int64_t)g->V + 127) / 128; break;
        case 9: src = g->sig; n = ((int64_t)g->V + 3) / 4; break;
        default: return fail(SMORE_E_INVALID_ARG, "unknown array %d", which);
    }
    if (count != n) return fail(SMORE_E_INVALID_ARG, "array %d has %lld entries, not %lld", which,
                                (long long)n, (long long)count);
    if (n == 0) return ok();
    hipError_t e = hipMemcpy(host_dst, src, (size_t)n * 4, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail(SMORE_E_HIP, "hipMemcpy: %s", hipGetErrorString(e));
    return ok();
}

int smore_profile_kernel(void* start_event, void* stop_event, int32_t which)
{
    if (which < 0 || which > 2) return fail(SMORE_E_INVALID_ARG, "which must be 0, 1 or 2");
    smore::arm_profile(start_event, stop_event, which);
    return ok();
}

int smore_wait_before_kernel(void* event, int32_t which)
{
    if (which != 0) return fail(SMORE_E_INVALID_ARG, "only the candidate kernel (which = 0) can wait");
    smore::arm_wait(event);
    return ok();
}

int smore_gather_probe(const void* table, int64_t table_bytes, int64_t n_reads, uint32_t* sink,
                       int64_t sink_words, void* hip_stream)
{
    if (!table || !sink) return fail(SMORE_E_INVALID_ARG, "table and sink are required");
    if (table_bytes < 64) return fail(SMORE_E_INVALID_ARG, "table_bytes must be at least 64");
    if (n_reads < 1 || n_reads > ((int64_t)1 << 40)) return fail(SMORE_E_INVALID_ARG, "n_reads out of range");
    if (sink_words < smore::gather_probe_threads(n_reads))
        return fail(SMORE_E_INVALID_ARG, "sink needs %lld words", (long long)smore::gather_probe_threads(n_reads));
    const char* err = nullptr;
    const int rc = smore::launch_gather_probe(table, table_bytes, n_reads, sink, (hipStream_t)hip_stream, &err);
    if (rc) return fail(rc, "%s", err ? err : "launch failed");
    return ok();
}

void smore_free_graph(smore_graph* g)
{
    if (!g) return;
    int cur = -1;
    (void)hipGetDevice(&cur);
    if (cur != g->device) (void)hipSetDevice(g->device);
    void* bufs[] = {g->f_node, g->f_grp, g->f_nbr, g->r_node, g->r_grp, g->r_nbr, g->active_in,
                    g->has_in, g->has_in4, g->sig};
    for (void* b : bufs)
        if (b) (void)hipFree(b);
    if (cur >= 0 && cur != g->device) (void)hipSetDevice(cur);
    delete g;
}

int smore_sample_workspace_bytes(const smore_graph* g, const smore_query_dag* dag,
                                 const smore_sample_args* args, size_t* bytes)
{
    (void)g;
    if (!dag || !args || !bytes) return fail(SMORE_E_INVALID_ARG, "NULL argument");
    if (args->batch < 1 || args->n_neg < 0 || args->neg_tries < args->n_neg ||
        args->neg_tries > SMORE_MAX_NEG_TRIES)
        return fail(SMORE_E_INVALID_ARG, "batch, n_neg or neg_tries out of range");
    smore::SampleParams p{};
    p.batch = args->batch;
    p.n_neg = args->n_neg;
    p.neg_tries = args->neg_tries;
    *bytes = smore::negatives_workspace_bytes(p);
    return ok();
}

}  // extern "C"

namespace {

enum Stage { POS = 1, NEG = 2 };

// Checks of the plan and the arguments common to the sampling entry points
// (host only); *qt receives the shape.
int check_args(const smore_query_dag* dag, const smore_sample_args* a, int* qt_out)
{
    int rc = check_dag(dag);
    if (rc) return rc;
    int qt = -1;
    for (const Preset& p : kPresets)
        if (same_dag(dag, p)) qt = p.qt;
    if (qt < 0)
        return fail(SMORE_E_UNSUPPORTED, "plan is not one of the fourteen presets (use smore_query_preset)");
    if (a->batch < 1) return fail(SMORE_E_INVALID_ARG, "batch must be >= 1");
    if (a->n_neg < 0) return fail(SMORE_E_INVALID_ARG, "n_neg must be >= 0");
    if (a->pos_tries < 1) return fail(SMORE_E_INVALID_ARG, "pos_tries must be >= 1");
    if (a->neg_tries < a->n_neg) return fail(SMORE_E_INVALID_ARG, "neg_tries must be >= n_neg");
    if (a->neg_tries > SMORE_MAX_NEG_TRIES)
        return fail(SMORE_E_UNSUPPORTED, "neg_tries %d exceeds SMORE_MAX_NEG_TRIES (%d)", a->neg_tries,
                    SMORE_MAX_NEG_TRIES);
    if (a->max_fanout < 0) return fail(SMORE_E_INVALID_ARG, "max_fanout must be >= 0");
    if (a->flags != 0) return fail(SMORE_E_INVALID_ARG, "flags must be 0");
    if (a->query_offset > (1ull << 32) || a->query_offset + (uint64_t)a->batch > (1ull << 32))
        return fail(SMORE_E_OVERFLOW, "query ids must stay below 2^32");
    // the long-list queue is indexed by a 32-bit counter over batch x round length
    if ((int64_t)a->batch * a->neg_tries >= ((int64_t)1 << 31))
        return fail(SMORE_E_OVERFLOW, "batch x neg_tries must stay below 2^31");
    *qt_out = qt;
    return SMORE_OK;
}

// The graph's device is the current one, and the planner's cut for the
// shape is the one the kernels implement.
int check_graph_and_cut(const smore_graph* g, const smore_query_dag* dag, int qt)
{
    if (!g) return fail(SMORE_E_INVALID_ARG, "graph is NULL");
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return fail(SMORE_E_HIP, "hipGetDevice failed");
    if (dev != g->device)
        return fail(SMORE_E_INVALID_ARG, "graph lives on device %d, current device is %d", g->device, dev);
    Planner P;
    P.d = dag;
    P.tie = 0;
    P.run();
    bool match = P.n_cut == kKernelCut[qt][0];
    for (int k = 0; match && k < P.n_cut; ++k) match = P.cut[k] == kKernelCut[qt][k + 1];
    if (!match) return fail(SMORE_E_UNSUPPORTED, "internal: planner cut differs from the kernel's");
    return SMORE_OK;
}

smore::SampleParams params_of(const smore_sample_args* a)
{
    smore::SampleParams p;
    p.batch = a->batch;
    p.n_neg = a->n_neg;
    p.pos_tries = a->pos_tries;
    p.neg_tries = a->neg_tries;
    p.max_fanout = a->max_fanout;
    p.seed = a->seed;
    p.query_offset = a->query_offset;
    return p;
}

// Validation shared by the sampling entry points, then the launch(es).
int run_sample(const smore_graph* g, const smore_query_dag* dag, const smore_sample_args* a,
               const smore_sample_out* out, int64_t* stats, void* workspace, size_t ws_bytes,
               void* hip_stream, int stages, int parts = smore::NEG_ALL)
{
    // the one-shot instrumentation arms belong to this call whatever its
    // outcome: a call that fails validation disarms them too
    struct Disarm {
        bool on;
        ~Disarm()
        {
            if (on) smore::disarm();
        }
    } disarm_on_return{(stages & NEG) != 0};
    // host-side checks first (they need no device), the graph last
    if (!a || !out) return fail(SMORE_E_INVALID_ARG, "args or out is NULL");
    int qt = -1;
    int rc = check_args(dag, a, &qt);
    if (rc) return rc;
    if (!out->anchors || !out->relations || !out->positive || !out->n_valid ||
        ((stages & POS) && !out->pos_attempts) || ((stages & NEG) && !out->neg_draws) ||
        ((stages & NEG) && a->n_neg > 0 && !out->negatives))
        return fail(SMORE_E_INVALID_ARG, "an output pointer is NULL");
    if ((rc = check_graph_and_cut(g, dag, qt))) return rc;
    const smore::SampleParams p = params_of(a);
    const char* err = "";
    if (stages & POS) {
        smore::WalkProgram w;
        std::memset(&w, 0, sizeof(w));
        compile_walk(dag, dag->root, 0, &w);
        rc = smore::launch_positive(g, w, p, *out, (hipStream_t)hip_stream, &err);
        if (rc) return fail(rc, "positive sampling: %s", err);
    }
    if (stages & NEG) {
        if (a->n_neg > 0 && (!workspace || ws_bytes < smore::negatives_workspace_bytes(p)))
            return fail(SMORE_E_INVALID_ARG, "workspace missing or smaller than %zu bytes",
                        smore::negatives_workspace_bytes(p));
        rc = smore::launch_negative(g, (smore::QType)qt, p, *out, stats, workspace, ws_bytes, parts,
                                    (hipStream_t)hip_stream, &err);
        if (rc) return fail(rc, "negative sampling: %s", err);
    }
    return ok();
}

}  // namespace

extern "C" {

int smore_sample(const smore_graph* g, const smore_query_dag* dag, const smore_sample_args* a,
                 const smore_sample_out* out, void* workspace, size_t ws_bytes, void* hip_stream)
{
    return run_sample(g, dag, a, out, nullptr, workspace, ws_bytes, hip_stream, POS | NEG);
}

int smore_verify(const smore_graph* g, const smore_query_dag* dag, const smore_sample_args* a,
                 const int32_t* anchors, const int32_t* relations, const int32_t* candidates,
                 uint32_t* mask, int32_t* n_valid, void* workspace, size_t ws_bytes, void* hip_stream)
{
    if (!a) return fail(SMORE_E_INVALID_ARG, "args is NULL");
    int qt = -1;
    int rc = check_args(dag, a, &qt);
    if (rc) return rc;
    if (!anchors || !relations || !n_valid || (a->n_neg > 0 && (!candidates || !mask)))
        return fail(SMORE_E_INVALID_ARG, "an input or output pointer is NULL");
    if ((rc = check_graph_and_cut(g, dag, qt))) return rc;
    const smore::SampleParams p = params_of(a);
    if (a->n_neg > 0 && (!workspace || ws_bytes < smore::negatives_workspace_bytes(p)))
        return fail(SMORE_E_INVALID_ARG, "workspace missing or smaller than %zu bytes",
                    smore::negatives_workspace_bytes(p));
    const char* err = "";
    rc = smore::launch_verify(g, (smore::QType)qt, p, anchors, relations, candidates, mask, n_valid,
                              workspace, ws_bytes, (hipStream_t)hip_stream, &err);
    if (rc) return fail(rc, "verification: %s", err);
    return ok();
}

int smore_sample_shared(const smore_graph* g, const smore_query_dag* dag, const smore_sample_args* a,
                        const smore_shared_out* out, void* workspace, size_t ws_bytes,
                        void* hip_stream)
{
    if (!a || !out) return fail(SMORE_E_INVALID_ARG, "args or out is NULL");
    int qt = -1;
    int rc = check_args(dag, a, &qt);
    if (rc) return rc;
    if (!out->anchors || !out->relations || !out->positive || !out->pos_attempts ||
        !out->n_shared || !out->n_valid || (a->n_neg > 0 && (!out->mask || !out->shared)))
        return fail(SMORE_E_INVALID_ARG, "an output pointer is NULL");
    if ((rc = check_graph_and_cut(g, dag, qt))) return rc;
    const smore::SampleParams p = params_of(a);
    if (a->n_neg > 0 && (!workspace || ws_bytes < smore::negatives_workspace_bytes(p)))
        return fail(SMORE_E_INVALID_ARG, "workspace missing or smaller than %zu bytes",
                    smore::negatives_workspace_bytes(p));
    // positives exactly as smore_sample (same draws), into the shared outputs
    smore_sample_out pos;
    std::memset(&pos, 0, sizeof(pos));
    pos.anchors = out->anchors;
    pos.relations = out->relations;
    pos.positive = out->positive;
    pos.pos_attempts = out->pos_attempts;
    pos.n_valid = out->n_valid;
    smore::WalkProgram w;
    std::memset(&w, 0, sizeof(w));
    compile_walk(dag, dag->root, 0, &w);
    const char* err = "";
    rc = smore::launch_positive(g, w, p, pos, (hipStream_t)hip_stream, &err);
    if (rc) return fail(rc, "positive sampling: %s", err);
    rc = smore::launch_shared(g, (smore::QType)qt, p, pos, out->shared, out->n_shared, out->mask,
                              workspace, ws_bytes, (hipStream_t)hip_stream, &err);
    if (rc) return fail(rc, "shared negatives: %s", err);
    return ok();
}

int smore_sample_noalloc(const smore_graph* g, const smore_query_dag* dag, const smore_sample_args* a,
                         const smore_sample_out* out, void* hip_stream)
{
    if (!a || !out) return fail(SMORE_E_INVALID_ARG, "args or out is NULL");
    int qt = -1;
    int rc = check_args(dag, a, &qt);
    if (rc) return rc;
    const smore::SampleParams p = params_of(a);
    const size_t need = a->n_neg > 0 ? smore::negatives_workspace_bytes(p) : 0;
    if (need > (size_t)SMORE_NOALLOC_SCRATCH_BYTES)
        return fail(SMORE_E_UNSUPPORTED,
                    "smore_sample_noalloc: these arguments need %zu bytes of scratch, more than its "
                    "fixed %zu; use smore_sample with a caller workspace",
                    need, (size_t)SMORE_NOALLOC_SCRATCH_BYTES);
    // the graph's device must be current: the scratch taken is that device's
    if ((rc = check_graph_and_cut(g, dag, qt))) return rc;
    void* ws = nullptr;
    size_t ws_bytes = 0;
    if (need) {
        const char* err = "";
        if ((rc = smore::scratch_workspace(&ws, &ws_bytes, &err)))
            return fail(rc, "smore_sample_noalloc: %s", err);
    }
    return run_sample(g, dag, a, out, nullptr, ws, ws_bytes, hip_stream, POS | NEG);
}

int smore_sample_positives(const smore_graph* g, const smore_query_dag* dag,
                           const smore_sample_args* a, const smore_sample_out* out, void* hip_stream)
{
    return run_sample(g, dag, a, out, nullptr, nullptr, 0, hip_stream, POS);
}

int smore_sample_negatives(const smore_graph* g, const smore_query_dag* dag,
                           const smore_sample_args* a, const smore_sample_out* out, int64_t* stats,
                           void* workspace, size_t ws_bytes, void* hip_stream)
{
    return run_sample(g, dag, a, out, stats, workspace, ws_bytes, hip_stream, NEG);
}

int smore_sample_negatives_part(const smore_graph* g, const smore_query_dag* dag,
                                const smore_sample_args* a, const smore_sample_out* out,
                                int64_t* stats, int32_t part, void* workspace, size_t ws_bytes,
                                void* hip_stream)
{
    if (part < 0 || part > 2) return fail(SMORE_E_INVALID_ARG, "part must be 0, 1 or 2");
    return run_sample(g, dag, a, out, stats, workspace, ws_bytes, hip_stream, NEG, 1 << part);
}

}  // extern "C"
