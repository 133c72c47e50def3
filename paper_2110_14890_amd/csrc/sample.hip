// sample.hip -- query sampling with verified negatives on gfx950.
//
// Positives (smore_sample_positives), one kernel:
//
//  k_positive: PA lanes per query (two; four or eight for plans that
//    accept less often per attempt), lane l running attempts l, l + PA, ...;
//    the lowest successful attempt wins.
//    Reverse directional sampling
//    (Sec. 3.1; appendix on reverse directional sampling): attempt t grounds
//    the root among entities with an in-edge, then runs the pre-order walk
//    program compiled from the plan, each projection picking an in-relation
//    of the current entity and an in-neighbour under it.  The first attempt
//    that reaches every anchor, keeps single-projection siblings apart and
//    respects max_fanout wins.
//
// Negatives (smore_sample_negatives): bidirectional rejection sampling
// (Sec. 3.2) at the node cut the planner picks for the shape, in rounds of
// candidate draws; k_prepare once, then per round k_candidates, k_heavy
// and the selection (k_compact_reg, or k_compact for long rounds), all on
// the caller's stream with no host synchronisation in between (the kernels
// themselves are described where they are defined).  The three steps can
// also be launched apart (smore_sample_negatives_part): the preparation,
// the first round's candidate kernel, the rest.  Forward caching turns
// the anchors into their neighbour lists A_r(a) (sorted CSR groups, staged
// in LDS when small, used in place when not); a draw without an in-edge is
// settled by the in-edge mask (on large graphs a coarse mask, then the
// entity's in-relation signature, which also settles draws with in-edges
// under none of the root's relations); the others are verified backward
// from the candidate; the first occurrences of the non-answers, in draw
// order, are the negatives, so the output is a function of the draw
// indices alone.
//
// Shared-candidate minibatches (smore_sample_shared) and verification of
// caller candidates (smore_verify) run the same candidate and long-list
// kernels on given candidates, then pack the states into mask rows
// (k_shared_set, k_pack).
#include <hip/hip_runtime.h>

#include <climits>
#include <cstring>
#include <mutex>

#include "philox.h"
#include "rows.h"
#include "smore_internal.h"

namespace smore {
namespace {

constexpr int STAGE = 1024;   // LDS entries per wavefront for staged forward lists
constexpr int LANE_SEG = 8;   // backward lists up to this length stay on one lane

// Draw states.  ST_DEEP exists only inside the candidate kernel: the
// candidate's backward list is short and it is tested after the shallow
// pass over all survivors of the window.
enum : int32_t { ST_NON = 0, ST_ANS = 1, ST_DUP = 2, ST_PEND = 3, ST_DEEP = 4 };

// Accounting of graph reads (bytes, and the 64-byte lines they span).  The
// verification kernel is instantiated with Tally when the caller asks for
// the figures and with NoTally otherwise; NoTally compiles to nothing.
struct NoTally {
    static constexpr bool on = false;
    __device__ __forceinline__ void read(const void*, int32_t) {}
    __device__ __forceinline__ void bytes_only(int64_t) {}
};
struct Tally {
    static constexpr bool on = true;
    uint64_t b = 0, l = 0;
    __device__ __forceinline__ void read(const void* p, int32_t nbytes)
    {
        if (nbytes <= 0) return;
        const uint64_t a = (uint64_t)p;
        b += (uint64_t)nbytes;
        l += ((a + nbytes - 1) >> 6) - (a >> 6) + 1;
    }
    __device__ __forceinline__ void bytes_only(int64_t n) { b += (uint64_t)n; }
};

// Edges [x, y) of v under r when v's node-pointer pair (n0, n1) is known.
template <class T>
__device__ __forceinline__ int2 group_from(const DirView& d, int32_t n0, int32_t n1, int32_t r, T& tl)
{
    int32_t lo = n0, hi = n1;
    while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        tl.read(&d.grp[mid].x, 4);
        if (d.grp[mid].x < r) lo = mid + 1; else hi = mid;
    }
    if (lo < n1 && d.grp[lo].x == r) {
        tl.read(&d.grp[lo].y, 4);
        tl.read(&d.grp[lo + 1].y, 4);
        return make_int2(d.grp[lo].y, d.grp[lo + 1].y);
    }
    return make_int2(0, 0);
}

// group_from for an entity with at most SCAN groups: all of its group
// entries (and the next one, for the end bound) are loaded at once, so the
// lookup is one dependent step instead of a chain of binary-search probes.
constexpr int SCAN = 8;

template <class T>
__device__ __forceinline__ int2 group_find(const DirView& d, int32_t n0, int32_t n1, int32_t r, T& tl)
{
    const int32_t n = n1 - n0;
    if (n > SCAN) return group_from(d, n0, n1, r, tl);
    if (n <= 0) return make_int2(0, 0);
    int2 e[SCAN + 1];
#pragma unroll
    for (int k = 0; k <= SCAN; ++k) e[k] = k <= n ? d.grp[n0 + k] : make_int2(INT_MAX, 0);
    tl.read(d.grp + n0, 8 * (n + 1));
    int2 res = make_int2(0, 0);
#pragma unroll
    for (int k = 0; k < SCAN; ++k)
        if (k < n && e[k].x == r) res = make_int2(e[k].y, e[k + 1].y);
    return res;
}

// group_find of two entities at once (the loads of both scans in flight
// together); inactive entries return (0, 0).
template <class T>
__device__ __forceinline__ void group_find2(const DirView& d, const int32_t* n0, const int32_t* n1,
                                            const bool* act, int32_t r, int2* res, T& tl)
{
    int2 e[2][SCAN + 1];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int32_t n = act[u] ? n1[u] - n0[u] : 0;
#pragma unroll
        for (int k = 0; k <= SCAN; ++k)
            e[u][k] = (n > 0 && n <= SCAN && k <= n) ? d.grp[n0[u] + k] : make_int2(INT_MAX, 0);
        if (n > 0 && n <= SCAN) tl.read(d.grp + n0[u], 8 * (n + 1));
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int32_t n = act[u] ? n1[u] - n0[u] : 0;
        res[u] = make_int2(0, 0);
        if (n > SCAN) {
            res[u] = group_from(d, n0[u], n1[u], r, tl);
        } else {
#pragma unroll
            for (int k = 0; k < SCAN; ++k)
                if (k < n && e[u][k].x == r) res[u] = make_int2(e[u][k].y, e[u][k + 1].y);
        }
    }
}

// Edges [x, y) of entity v under relation r in one direction ((0, 0) if
// none): the node-pointer pair, then the group lookup.
template <class T>
__device__ __forceinline__ int2 group_range(const DirView& d, int32_t v, int32_t r, T& tl)
{
    const int32_t n0 = d.node[v], n1 = d.node[v + 1];
    tl.read(d.node + v, 8);
    return group_find(d, n0, n1, r, tl);
}

__device__ __forceinline__ int2 group_range(const DirView& d, int32_t v, int32_t r)
{
    NoTally t;
    return group_range(d, v, r, t);
}

// A sorted entity list, staged in LDS (lds = true) or read in place.
struct FSet {
    const int32_t* p;
    int32_t n;
    bool lds;
};

template <class T>
__device__ __forceinline__ bool has(const int32_t* p, int32_t n, int32_t x, bool count, T& tl)
{
    int32_t lo = 0, hi = n;
    while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        if (count) tl.read(p + mid, 4);
        if (p[mid] < x) lo = mid + 1; else hi = mid;
    }
    if (lo < n && count) tl.read(p + lo, 4);
    return lo < n && p[lo] == x;
}

// Membership in a forward-cached list.  The list itself is accounted once
// per query when it is cached; lookups in it are not graph traffic of the
// method, wherever the list lives.
template <class T>
__device__ __forceinline__ bool has(const FSet& s, int32_t x, T&)
{
    NoTally none;
    return has(s.p, s.n, x, false, none);
}

// Wave-uniform copy of a value every lane holds (the compiler then keeps
// loops and exits that depend on it converged).
__device__ __forceinline__ int32_t uni(int32_t x) { return __builtin_amdgcn_readfirstlane(x); }

// Lane k's copy of a value (k wave-uniform).
__device__ __forceinline__ int32_t readlane(int32_t x, int k) { return __builtin_amdgcn_readlane(x, k); }
__device__ __forceinline__ int64_t readlane64(int64_t x, int k)
{
    return (int64_t)(uint32_t)readlane((int32_t)x, k) | ((int64_t)readlane((int32_t)(x >> 32), k) << 32);
}

__device__ __forceinline__ uint64_t lanes_below(int lane)
{
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Four independent membership searches of x[0..3] in the sorted list
// B[0..nb) (nb wave-uniform): branchless, the same number of steps in every
// lane, and the four loads of a step independent of each other, so a lane
// keeps four dependent chains in flight.  A key of -1 never matches.
template <class T>
__device__ __forceinline__ void search4(const int32_t* B, int32_t nb, const int32_t* x, bool* found,
                                        bool count, T& tl)
{
    int32_t base[4] = {0, 0, 0, 0};
    if (nb <= 0) {
        found[0] = found[1] = found[2] = found[3] = false;
        return;
    }
    for (int32_t n = nb; n > 1;) {
        const int32_t half = n >> 1;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (count) tl.read(B + base[k] + half, 4);
            base[k] = B[base[k] + half] <= x[k] ? base[k] + half : base[k];
        }
        n -= half;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if (count) tl.read(B + base[k], 4);
        found[k] = B[base[k]] == x[k];
    }
}

// search4 with a target list per key (lists of different lengths; the loop
// runs until every key of the lane is settled).
template <class T>
__device__ __forceinline__ void search4v(const int32_t* const* B, const int32_t* nb, const int32_t* x,
                                         const bool* count, bool* found, T& tl)
{
    int32_t base[4] = {0, 0, 0, 0}, n[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) n[k] = nb[k];
    for (;;) {
        bool more = false;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (n[k] > 1) {
                const int32_t half = n[k] >> 1;
                if (count[k]) tl.read(B[k] + base[k] + half, 4);
                base[k] = B[k][base[k] + half] <= x[k] ? base[k] + half : base[k];
                n[k] -= half;
                more |= n[k] > 1;
            }
        }
        if (!more) break;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        found[k] = false;
        if (nb[k] > 0) {
            if (count[k]) tl.read(B[k] + base[k], 4);
            found[k] = B[k][base[k]] == x[k];
        }
    }
}

// search4v with three probes per step where four or more entries remain
// (a quaternary search: fewer dependent reads, more reads in all).
template <class T>
__device__ __forceinline__ void search4q(const int32_t* const* B, const int32_t* nb, const int32_t* x,
                                         const bool* count, bool* found, T& tl)
{
    int32_t base[4] = {0, 0, 0, 0}, n[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) n[k] = nb[k];
    for (;;) {
        bool more = false;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (n[k] >= 4) {
                const int32_t q = n[k] >> 2;
                const int32_t* b = B[k] + base[k];
                if (count[k]) { tl.read(b + q, 4); tl.read(b + 2 * q, 4); tl.read(b + 3 * q, 4); }
                const int32_t v1 = b[q], v2 = b[2 * q], v3 = b[3 * q];
                base[k] += q * ((v1 <= x[k]) + (v2 <= x[k]) + (v3 <= x[k]));
                n[k] -= 3 * q;
            } else if (n[k] > 1) {
                const int32_t half = n[k] >> 1;
                if (count[k]) tl.read(B[k] + base[k] + half, 4);
                base[k] = B[k][base[k] + half] <= x[k] ? base[k] + half : base[k];
                n[k] -= half;
            }
            more |= n[k] > 1;
        }
        if (!more) break;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        found[k] = false;
        if (nb[k] > 0) {
            if (count[k]) tl.read(B[k] + base[k], 4);
            found[k] = B[k][base[k]] == x[k];
        }
    }
}

// Does some element of K[0..nk) occur in L[0..nl)?  Whole wavefront, 256
// keys per step (four per lane).  k_glob / l_glob: whether reads of the
// list count as graph traffic.
template <class T>
__device__ bool wave_any(const int32_t* K, int32_t nk, bool k_glob, const int32_t* L, int32_t nl,
                         bool l_glob, int lane, T& tl)
{
    for (int32_t k0 = 0; k0 < nk; k0 += 256) {
        int32_t x[4];
        bool f[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int32_t i = k0 + 64 * k + lane;
            x[k] = i < nk ? K[i] : -1;
        }
        if (k_glob && lane == 0) tl.read(K + k0, 4 * min(256, nk - k0));
        search4(L, nl, x, f, l_glob, tl);
        if (__ballot(f[0] || f[1] || f[2] || f[3])) return true;
    }
    return false;
}

// Do the sorted lists A and B share an element?  The shorter is the key
// list, searched in the longer.
template <class T>
__device__ bool wave_meet(const int32_t* A, int32_t na, bool a_glob, const int32_t* B, int32_t nb,
                          bool b_glob, int lane, T& tl)
{
    if (na <= nb) return wave_any(A, na, a_glob, B, nb, b_glob, lane, tl);
    return wave_any(B, nb, b_glob, A, na, a_glob, lane, tl);
}

// Does the sorted graph list S share one element with both A and B?  The
// shortest of the three is the key list, searched in the other two.
template <class T>
__device__ bool wave_meet3(const int32_t* S, int32_t ns, FSet A, FSet B, int lane, T& tl)
{
    const int32_t *K = S, *L1 = A.p, *L2 = B.p;
    int32_t nk = ns, n1 = A.n, n2 = B.n;
    bool kg = true, g1 = false, g2 = false;   // lookups inside forward lists are not counted
    if (A.n < nk && A.n <= B.n) {
        K = A.p; nk = A.n; kg = false;
        L1 = S; n1 = ns; g1 = true;
    } else if (B.n < nk) {
        K = B.p; nk = B.n; kg = false;
        L2 = S; n2 = ns; g2 = true;
    }
    for (int32_t k0 = 0; k0 < nk; k0 += 256) {
        int32_t x[4];
        bool f1[4], f2[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int32_t i = k0 + 64 * k + lane;
            x[k] = i < nk ? K[i] : -1;
        }
        if (kg && lane == 0) tl.read(K + k0, 4 * min(256, nk - k0));
        search4(L1, n1, x, f1, g1, tl);
        search4(L2, n2, x, f2, g2, tl);
        const bool hit = (f1[0] && f2[0]) || (f1[1] && f2[1]) || (f1[2] && f2[2]) || (f1[3] && f2[3]);
        if (__ballot(hit)) return true;
    }
    return false;
}

// Does the sorted graph list S share an element with A that is not in B
// (the set difference of an intersection with a complemented operand)?
// The shorter of S and A is the key list, searched in the other and in B.
template <class T>
__device__ bool wave_meet_minus(const int32_t* S, int32_t ns, FSet A, FSet B, int lane, T& tl)
{
    const int32_t *K = S, *L = A.p;
    int32_t nk = ns, nl = A.n;
    bool kg = true, lg = false;   // lookups inside forward lists are not counted
    if (A.n < ns) {
        K = A.p; nk = A.n; kg = false;
        L = S; nl = ns; lg = true;
    }
    for (int32_t k0 = 0; k0 < nk; k0 += 256) {
        int32_t x[4];
        bool f1[4], f2[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int32_t i = k0 + 64 * k + lane;
            x[k] = i < nk ? K[i] : -1;
        }
        if (kg && lane == 0) tl.read(K + k0, 4 * min(256, nk - k0));
        search4(L, nl, x, f1, lg, tl);
        search4(B.p, B.n, x, f2, false, tl);
        const bool hit = (f1[0] && !f2[0]) || (f1[1] && !f2[1]) || (f1[2] && !f2[2]) || (f1[3] && !f2[3]);
        if (__ballot(hit)) return true;
    }
    return false;
}

// ------------------------------------------------------------- positive
__device__ __forceinline__ int32_t sel4(int i, int32_t a, int32_t b, int32_t c, int32_t d)
{
    return i == 0 ? a : i == 1 ? b : i == 2 ? c : d;
}

__device__ __forceinline__ int32_t reg5(int i, const int32_t* e)
{
    return i == 0 ? e[0] : i == 1 ? e[1] : i == 2 ? e[2] : i == 3 ? e[3] : e[4];
}

// Relation grounded for relation slot sl (-1 if no step has it).
__device__ __forceinline__ int32_t slot_rel(const WalkProgram& wp, const int32_t* qr, int sl)
{
    int32_t v = -1;
    for (int k = 0; k < wp.n_steps; ++k)
        if (wp.rel_slot[k] == sl) v = sel4(k, qr[0], qr[1], qr[2], -1);
    return v;
}

// Is t in the complemented operand's set: A_r0(a) for one step, or the
// entities reached from A_r0(a) under r1 for two (some y of A_r0(a) with
// (y, r1, t) an edge)?  At lane level: the shorter of A_r0(a) and t's
// in-list under r1 is walked and each entry searched in the longer.
__device__ bool neg_member(const GraphView& g, int steps, int32_t a, int32_t r0, int32_t r1, int32_t t)
{
    NoTally none;
    const int2 f = group_range(g.fwd, a, r0);
    const int32_t nf = f.y - f.x;
    if (steps == 1) return nf > 0 && has(g.fwd.nbr + f.x, nf, t, false, none);
    const int2 b = group_range(g.rev, t, r1);
    const int32_t nb = b.y - b.x;
    if (nf == 0 || nb == 0) return false;
    const bool fk = nf <= nb;
    const int32_t* K = fk ? g.fwd.nbr + f.x : g.rev.nbr + b.x;
    const int32_t* L = fk ? g.rev.nbr + b.x : g.fwd.nbr + f.x;
    const int32_t nk = fk ? nf : nb, nl = fk ? nb : nf;
    for (int32_t i = 0; i < nk; ++i)
        if (has(L, nl, K[i], false, none)) return true;
    return false;
}

// Attempts of one query run PA at a time, on PA neighbouring lanes (lane l
// of the group takes attempts l, l + PA, ...): the lowest successful
// attempt of a group step is the first successful attempt overall, so the
// result is that of trying them one after the other.  Four lanes per query,
// eight for plans with a complemented operand, whose attempts are rejected
// more often.

// One attempt t of query q: true and the grounded registers when accepted.
__device__ __forceinline__ bool pos_attempt(const GraphView& g, const WalkProgram& wp,
                                            const SampleParams& p, uint32_t q, int t, int32_t* e,
                                            int32_t* qr)
{
    e[0] = e[1] = e[2] = e[3] = e[4] = -1;
    qr[0] = qr[1] = qr[2] = -1;
    if (g.n_active == 0) return false;
    e[0] = g.active_in[reduce_range(draw64(p.seed, TAG_POS, q, t, 0), (uint32_t)g.n_active)];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        if (k >= wp.n_steps) break;
        const bool sib = wp.neg_steps > 0 && k == wp.neg_first;
        const int after = wp.neg_steps > 0 && k >= wp.neg_first ? 1 : 0;
        if (sib) {
            // sibling entity of the complemented operand: uniform over
            // A_r(x) of step sib_step, a list that holds that step's entity
            const int32_t x = reg5(wp.sib_step + 1, e);
            const int32_t r = sel4(wp.sib_step, qr[0], qr[1], qr[2], -1);
            const int2 fr = group_range(g.fwd, x, r);
            if (fr.y == fr.x) return false;
            const uint64_t u = draw64(p.seed, TAG_POS, q, t, 1 + 2 * k);
            e[WALK_SIB] = g.fwd.nbr[fr.x + (int32_t)reduce_range(u, (uint32_t)(fr.y - fr.x))];
        }
        const int32_t v = reg5(wp.src[k], e);
        const uint64_t u0 = draw64(p.seed, TAG_POS, q, t, 1 + 2 * k + after);
        const uint64_t u1 = draw64(p.seed, TAG_POS, q, t, 2 + 2 * k + after);
        const int32_t s0 = g.rev.node[v], s1 = g.rev.node[v + 1];
        if (s0 == s1) return false;                       // no in-edge: dead end
        const int32_t s = s0 + (int32_t)reduce_range(u0, (uint32_t)(s1 - s0));
        const int2 gr = g.rev.grp[s];
        const int32_t len = g.rev.grp[s + 1].y - gr.y;
        const int32_t x = g.rev.nbr[gr.y + (int32_t)reduce_range(u1, (uint32_t)len)];
        if (p.max_fanout > 0) {
            const int2 fr = group_range(g.fwd, x, gr.x);
            if (fr.y - fr.x > p.max_fanout) return false;
        }
        e[k + 1] = x;
        qr[k] = gr.x;
    }
    for (int pr = 0; pr < wp.n_pairs; ++pr) {
        const int32_t xa = reg5(wp.anchor_reg[wp.pair_anchor[pr][0]], e);
        const int32_t xb = reg5(wp.anchor_reg[wp.pair_anchor[pr][1]], e);
        const int32_t ra = slot_rel(wp, qr, wp.pair_rel[pr][0]);
        const int32_t rb = slot_rel(wp, qr, wp.pair_rel[pr][1]);
        if (xa == xb && ra == rb) return false;           // degenerate sibling branches
    }
    if (wp.neg_steps > 0) {   // the intersection's entity must stay outside the complemented set
        const int32_t a = reg5(wp.anchor_reg[wp.neg_anchor], e);
        const int32_t r0 = slot_rel(wp, qr, wp.neg_rel[0]);
        const int32_t r1 = wp.neg_steps > 1 ? slot_rel(wp, qr, wp.neg_rel[1]) : -1;
        if (neg_member(g, wp.neg_steps, a, r0, r1, reg5(wp.neg_target, e))) return false;
    }
    return true;
}

template <int PA>
__global__ __launch_bounds__(256) void k_positive(GraphView g, WalkProgram wp, SampleParams p,
                                                  smore_sample_out out)
{
    const int32_t gid = blockIdx.x * blockDim.x + threadIdx.x;
    const int32_t b = gid / PA;
    const int l = gid % PA;
    if (b >= p.batch) return;   // whole groups: PA divides the workgroup size
    const uint32_t q = (uint32_t)(p.query_offset + (uint64_t)b);
    const int gbase = (threadIdx.x & 63) & ~(PA - 1);
    int32_t e[5], qr[3];
    int win = -1;
    for (int t0 = 0; t0 < p.pos_tries; t0 += PA) {
        const int t = t0 + l;
        const bool ok = t < p.pos_tries && pos_attempt(g, wp, p, q, t, e, qr);
        const uint32_t m = (uint32_t)(__ballot(ok) >> gbase) & ((1u << PA) - 1);
        if (m) {
            win = t0 + __ffs(m) - 1;
            break;
        }
    }
    if (win < 0) {
        if (l == 0) {
            int32_t* A = out.anchors + 3 * (int64_t)b;
            int32_t* R = out.relations + 3 * (int64_t)b;
            for (int k = 0; k < 3; ++k) { A[k] = -1; R[k] = -1; }
            out.positive[b] = -1;
            out.n_valid[b] = -1;
            out.pos_attempts[b] = p.pos_tries;
        }
        return;
    }
    if (l != win % PA) return;  // the lane that ran the winning attempt writes the row
    int32_t* A = out.anchors + 3 * (int64_t)b;
    int32_t* R = out.relations + 3 * (int64_t)b;
    for (int a = 0; a < 3; ++a) A[a] = a < wp.n_anchor ? reg5(wp.anchor_reg[a], e) : -1;
    for (int sl = 0; sl < 3; ++sl) R[sl] = slot_rel(wp, qr, sl);
    out.positive[b] = e[0];
    out.n_valid[b] = 0;
    out.pos_attempts[b] = win + 1;
}


// --------------------------------------------------------------- negatives
// Bidirectional rejection sampling of the negatives, in rounds of candidate
// draws.  Per round:
//   k_candidates  one wavefront per query (one-wave workgroups): the round's
//                 draws, the in-edge mask / signature test, and for the
//                 survivors either a decision at lane level or a push to the
//                 heavy queue;
//   k_heavy       one wavefront per queued (query, draw), persistent
//                 wavefronts: intersection of a long backward list with the
//                 forward-cached list(s);
//   k_compact_reg one wavefront per query (k_compact for rounds of more
//                 than 1,024 draws): first-occurrence test of every draw so
//                 far, ordered selection of the first n_neg kept.
// Queries still short of n_neg after a round go to the next round through a
// device-side list, each with the draw range the selection sets for it, so
// rounds need no host synchronisation.

// Lists per shape (anchor slot, relation slot) at the cut the planner picks:
//   1p {a0}, 2p/3p {V1}, 2i/3i/2u/2in/3in {anchors}, ip/up/inp {Y0, Y1},
//   pi/pin {V1, a1}, pni {V1 of the complemented chain, a1}.
// cached = forward caching to the cut (A_r(a) at a cut node one projection
// above the anchor); otherwise the list is the anchor's neighbour list used
// for an edge test at a cut placed on the anchor, which may be decided from
// either end of the edge.  n_anc / n_rel: slots the shape uses.
template <int QT> struct Shape;
#define SHAPE(Q, NF, NA, NR, A0, A1, A2, R0, R1, R2, C0, C1, C2)                                 \
    template <> struct Shape<Q> {                                                              \
        static constexpr int nf = NF, n_anc = NA, n_rel = NR;                                  \
        static constexpr int fa[3] = {A0, A1, A2}, fr[3] = {R0, R1, R2}, cached[3] = {C0, C1, C2}; \
    };
SHAPE(Q1P, 1, 1, 1, 0, 0, 0, 0, 0, 0, 0, 0, 0)
SHAPE(Q2P, 1, 1, 2, 0, 0, 0, 0, 0, 0, 1, 0, 0)
SHAPE(Q3P, 1, 1, 3, 0, 0, 0, 0, 0, 0, 1, 0, 0)
SHAPE(Q2I, 2, 2, 2, 0, 1, 0, 0, 1, 0, 0, 0, 0)
SHAPE(Q3I, 3, 3, 3, 0, 1, 2, 0, 1, 2, 0, 0, 0)
SHAPE(QIP, 2, 2, 3, 0, 1, 0, 0, 1, 0, 1, 1, 0)
SHAPE(QPI, 2, 2, 3, 0, 1, 0, 0, 2, 0, 1, 0, 0)
SHAPE(Q2U, 2, 2, 2, 0, 1, 0, 0, 1, 0, 0, 0, 0)
SHAPE(QUP, 2, 2, 3, 0, 1, 0, 0, 1, 0, 1, 1, 0)
SHAPE(Q2IN, 2, 2, 2, 0, 1, 0, 0, 1, 0, 0, 0, 0)
SHAPE(Q3IN, 3, 3, 3, 0, 1, 2, 0, 1, 2, 0, 0, 0)
SHAPE(QINP, 2, 2, 3, 0, 1, 0, 0, 1, 0, 1, 1, 0)
SHAPE(QPIN, 2, 2, 3, 0, 1, 0, 0, 2, 0, 1, 0, 0)
SHAPE(QPNI, 2, 2, 3, 0, 1, 0, 0, 2, 0, 1, 0, 0)
#undef SHAPE

// Shapes whose last step into the root is the backward step of a two-hop
// chain under relation slot 1 (else slot 2), and shapes whose second list
// is a forward-cached set the deep test needs staged.
template <int QT> constexpr bool chain_r1 = QT == Q2P || QT == QPI || QT == QPIN || QT == QPNI;
template <int QT> constexpr bool two_cached = QT == QIP || QT == QUP || QT == QINP;

// Lists that test a candidate by one edge into the root: c is an answer
// only if c is in list f for every f of `mask` (any f when `any`).  When
// these lists are staged in LDS they decide the draws without a single
// graph read; otherwise the in-edge mask does.
// Relation slots of the projections that end at the root (bit s: slot s),
// positive operands only: an answer has an in-edge under each of them (any
// one of them for a union).
template <int QT> struct RootRels { static constexpr int mask = 0, any = 0; };
template <> struct RootRels<Q1P> { static constexpr int mask = 1, any = 0; };
template <> struct RootRels<Q2P> { static constexpr int mask = 2, any = 0; };
template <> struct RootRels<Q3P> { static constexpr int mask = 4, any = 0; };
template <> struct RootRels<Q2I> { static constexpr int mask = 3, any = 0; };
template <> struct RootRels<Q3I> { static constexpr int mask = 7, any = 0; };
template <> struct RootRels<QIP> { static constexpr int mask = 4, any = 0; };
template <> struct RootRels<QPI> { static constexpr int mask = 6, any = 0; };
template <> struct RootRels<Q2U> { static constexpr int mask = 3, any = 1; };
template <> struct RootRels<QUP> { static constexpr int mask = 4, any = 0; };
template <> struct RootRels<Q2IN> { static constexpr int mask = 1, any = 0; };
template <> struct RootRels<Q3IN> { static constexpr int mask = 3, any = 0; };
template <> struct RootRels<QINP> { static constexpr int mask = 4, any = 0; };
template <> struct RootRels<QPIN> { static constexpr int mask = 2, any = 0; };
template <> struct RootRels<QPNI> { static constexpr int mask = 4, any = 0; };

template <int QT> struct RootLists { static constexpr int mask = 0, any = 0; };
template <> struct RootLists<Q1P> { static constexpr int mask = 1, any = 0; };
template <> struct RootLists<Q2I> { static constexpr int mask = 3, any = 0; };
template <> struct RootLists<Q3I> { static constexpr int mask = 7, any = 0; };
template <> struct RootLists<QPI> { static constexpr int mask = 2, any = 0; };
template <> struct RootLists<Q2U> { static constexpr int mask = 3, any = 1; };
// with negation, only the positive operands' lists are necessary conditions
template <> struct RootLists<Q2IN> { static constexpr int mask = 1, any = 0; };
template <> struct RootLists<Q3IN> { static constexpr int mask = 3, any = 0; };
template <> struct RootLists<QPNI> { static constexpr int mask = 2, any = 0; };

// The candidate kernel runs one wavefront per workgroup, and its first pass
// one query per workgroup: queries differ widely in cost, and the hardware
// dispatcher hands each freed slot the next query, where a fixed share per
// wavefront leaves the kernel waiting on its slowest shares.
constexpr int CWG = 64;
constexpr int HEAVY_WG = 256;    // threads of the heavy-queue workgroups
constexpr int QF = 8;            // int32 per query in the per-query block
constexpr int PERSIST_BLOCKS = 2048;
// 3p long-list work in bounded units: the long-list kernel expands at most
// UNIT_Y entities y of an item and searches at most UNIT_PAIRS pairs of one
// y itself; the rest become units of the unit queue (UNITS_PER_QUERY slots
// per query), which the unit kernel then takes, so one huge item is spread
// over many wavefronts instead of setting the kernel's length alone.
constexpr int UNIT_Y = 256;
constexpr int UNIT_PAIRS = 1024;
constexpr int UNITS_PER_QUERY = 64;

// Workspace carved out of the caller's buffer.
struct Ws {
    int32_t* ctrl;    // [0] queue pushes [1] queue pops [2 + k] size of active list k
                      // [5] 3p units pushed
    int32_t* qf;      // [B][QF]: list k at [2k, 2k+1) edge range; [6] bit k: list k staged
    uint8_t* status;  // [B][neg_tries] ST_*
    int32_t* act[2];  // active query lists
    int2* queue;      // (query, draw) items
    int64_t qcap;
    int4* units;      // 3p long-list units: (item, a, b, kind), counted by ctrl[5]
    int64_t ucap;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Candidate j of query b: draw j of the query's own stream, pick(U(NEG, q,
// 0, j), V) with q = query_offset + b (Sec. 3.2: candidates uniform over the
// entities), or entry j of the caller's list or the shared set, -1 when it
// is not an entity.  Every kernel that needs a candidate takes it from here,
// so the draws are recomputed where they are used instead of being stored
// and read back.
__device__ __forceinline__ int32_t candidate(const SampleParams& p, int32_t V, int32_t b, int32_t j)
{
    if (p.shared_mode != 0) {
        const int32_t c = p.shared[(int64_t)p.cand_stride * b + j];
        return (uint32_t)c >= (uint32_t)V ? -1 : c;
    }
    const uint32_t q = (uint32_t)(p.query_offset + (uint64_t)b);
    return (int32_t)reduce_range(draw64(p.seed, TAG_NEG, q, 0, (uint32_t)j), (uint32_t)V);
}

// Rounds of candidate draws.  Round 0 takes draws [0, first_round(p)) of
// every query: n_neg plus a small margin (a query rarely rejects more than
// a few percent of its draws).  A query still short of n_neg after a round
// takes its own next range: the draws its deficit needs at the acceptance
// rate it has had so far, with a margin (next_round_end); the last round
// takes every query still short to neg_tries.  Rounds are a scheduling
// detail: a query's negatives are its first n_neg accepted draws in draw
// order whatever the rounds were.
inline int32_t first_round(const SampleParams& p)
{
    const int64_t e = (int64_t)p.n_neg + p.n_neg / 32 + 8;
    return (int32_t)(e < p.neg_tries ? e : p.neg_tries);
}

// Three rounds (first, own ranges, the rest); a batch under 4,096 queries
// is bound by launches rather than draws, and its second round takes the
// rest of the budget at once.
inline int n_rounds(const SampleParams& p)
{
    if (first_round(p) >= p.neg_tries) return 1;
    return p.batch >= 4096 ? 3 : 2;
}

// Longest range one query takes in one round.
inline int32_t max_round_len(const SampleParams& p)
{
    const int32_t e0 = first_round(p);
    return e0 > p.neg_tries - e0 ? e0 : p.neg_tries - e0;
}

// End of the next range of a query that has `kept` accepted draws among its
// first `end`: the deficit over that acceptance rate, a quarter more, and
// 16 draws; everything up to neg_tries when nothing was accepted yet or the
// next round is the last.
__device__ __forceinline__ int32_t next_round_end(const SampleParams& p, int32_t end, int32_t kept,
                                                  bool to_last)
{
    if (to_last || kept <= 0) return p.neg_tries;
    const int64_t need = (int64_t)(p.n_neg - kept) * end;
    const int64_t more = (need * 5 + 4 * (int64_t)kept - 1) / (4 * (int64_t)kept) + 16;
    return (int32_t)(end + more < p.neg_tries ? end + more : p.neg_tries);
}

// A query's draw range of a later round, kept in its per-query block (two
// 16-bit draw indices).
static_assert(SMORE_MAX_NEG_TRIES < 65536, "draw indices must fit 16 bits");
__host__ __device__ __forceinline__ int32_t pack_range(int32_t a, int32_t b) { return a | (b << 16); }
__host__ __device__ __forceinline__ int32_t range_lo(int32_t r) { return r & 0xFFFF; }
__host__ __device__ __forceinline__ int32_t range_hi(int32_t r) { return (int32_t)((uint32_t)r >> 16); }

size_t ws_layout(const SampleParams& p, Ws* w, char* base)
{
    const int64_t B = p.batch, T = p.neg_tries > 0 ? p.neg_tries : 1;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char* ptr = base ? base + off : nullptr;
        off += align256(bytes);
        return ptr;
    };
    Ws x;
    x.ctrl = (int32_t*)take(64 * sizeof(int32_t));
    x.qf = (int32_t*)take((size_t)B * QF * sizeof(int32_t));
    x.status = (uint8_t*)take((size_t)B * T);
    x.act[0] = (int32_t*)take((size_t)B * sizeof(int32_t));
    x.act[1] = (int32_t*)take((size_t)B * sizeof(int32_t));
    x.qcap = B * (int64_t)max_round_len(p);
    x.queue = (int2*)take((size_t)x.qcap * sizeof(int2));
    x.ucap = B * (int64_t)UNITS_PER_QUERY;
    x.units = (int4*)take((size_t)x.ucap * sizeof(int4));
    if (w) *w = x;
    return off;
}

// Tally of one lane summed over its wavefront and added to the query's
// counters (the wavefront must be converged).
template <class T>
__device__ __forceinline__ void flush_tally(T& tl, int64_t* stats, int32_t b, int lane, int slot = 0)
{
    if constexpr (T::on) {
        uint64_t x = tl.b, y = tl.l;
        for (int s = 32; s > 0; s >>= 1) {
            x += __shfl_xor(x, s);
            y += __shfl_xor(y, s);
        }
        if (lane == 0 && (x | y)) {
            atomicAdd((unsigned long long*)&stats[4 * (int64_t)b + slot], (unsigned long long)x);
            atomicAdd((unsigned long long*)&stats[4 * (int64_t)b + slot + 1], (unsigned long long)y);
        }
        tl.b = tl.l = 0;
    }
}

// Is (a, r, c) an edge?  From the anchor's list when it is staged in LDS,
// otherwise from c's reverse list under r (c's node pair already loaded).
template <class T>
__device__ __forceinline__ bool edge_test(const GraphView& g, const FSet& Fa, int32_t a, int32_t r,
                                          int32_t c, int32_t n0, int32_t n1, T& tl)
{
    if (Fa.lds) return has(Fa, c, tl);
    const int2 s = group_find(g.rev, n0, n1, r, tl);
    return s.y > s.x && has(g.rev.nbr + s.x, s.y - s.x, a, true, tl);
}

// First, shallow decision for candidate c at lane level: ST_NON or ST_ANS
// when it is settled by the cached lists and c's own groups, ST_PEND when a
// wavefront must intersect a long list, ST_DEEP with c's backward list
// [lst.x, lst.y) when that list is short and is to be tested next.
template <int QT, class T>
__device__ __forceinline__ int32_t shallow_test(const GraphView& g, const FSet* F, const int32_t* anc,
                                                const int32_t* rel, int32_t c, int32_t n0, int32_t n1,
                                                int2& lst, T& tl)
{
    if (QT == Q1P) return edge_test(g, F[0], anc[0], rel[0], c, n0, n1, tl) ? ST_ANS : ST_NON;
    if (QT == Q2I)
        return (edge_test(g, F[0], anc[0], rel[0], c, n0, n1, tl) &&
                edge_test(g, F[1], anc[1], rel[1], c, n0, n1, tl)) ? ST_ANS : ST_NON;
    if (QT == Q3I)
        return (edge_test(g, F[0], anc[0], rel[0], c, n0, n1, tl) &&
                edge_test(g, F[1], anc[1], rel[1], c, n0, n1, tl) &&
                edge_test(g, F[2], anc[2], rel[2], c, n0, n1, tl)) ? ST_ANS : ST_NON;
    if (QT == Q2U)
        return (edge_test(g, F[0], anc[0], rel[0], c, n0, n1, tl) ||
                edge_test(g, F[1], anc[1], rel[1], c, n0, n1, tl)) ? ST_ANS : ST_NON;
    if (QT == Q2IN)
        return (edge_test(g, F[0], anc[0], rel[0], c, n0, n1, tl) &&
                !edge_test(g, F[1], anc[1], rel[1], c, n0, n1, tl)) ? ST_ANS : ST_NON;
    if (QT == Q3IN)
        return (edge_test(g, F[0], anc[0], rel[0], c, n0, n1, tl) &&
                edge_test(g, F[1], anc[1], rel[1], c, n0, n1, tl) &&
                !edge_test(g, F[2], anc[2], rel[2], c, n0, n1, tl)) ? ST_ANS : ST_NON;
    if ((QT == QPI || QT == QPNI) && !edge_test(g, F[1], anc[1], rel[2], c, n0, n1, tl)) return ST_NON;
    if (QT == QPIN && edge_test(g, F[1], anc[1], rel[2], c, n0, n1, tl)) return ST_NON;
    // backward step from c under the relation entering the root; for pni a
    // meeting chain puts c in the complemented set
    const int32_t rb = chain_r1<QT> ? rel[1] : rel[2];
    const int2 s = group_find(g.rev, n0, n1, rb, tl);
    if (s.y == s.x) return QT == QPNI ? ST_ANS : ST_NON;
    if (s.y - s.x > LANE_SEG || !F[0].lds || (two_cached<QT> && !F[1].lds)) return ST_PEND;
    lst = s;
    return ST_DEEP;
}

// shallow_test of two candidates c[0], c[1] (act[u]: slot in use) with the
// dependent steps of both interleaved.
template <int QT, class T>
__device__ __forceinline__ void shallow_test2(const GraphView& g, const FSet* F, const int32_t* anc,
                                              const int32_t* rel, const int32_t* c, const bool* act,
                                              int32_t* st, int2* lst, T& tl)
{
    int32_t n0[2], n1[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        n0[u] = n1[u] = 0;
        if (act[u]) {
            n0[u] = g.rev.node[c[u]];
            n1[u] = g.rev.node[c[u] + 1];
            tl.read(g.rev.node + c[u], 8);
        }
    }
    if (QT == Q1P || QT == Q2I || QT == Q3I || QT == Q2U || QT == Q2IN || QT == Q3IN) {
#pragma unroll
        for (int u = 0; u < 2; ++u)
            st[u] = act[u] ? shallow_test<QT>(g, F, anc, rel, c[u], n0[u], n1[u], lst[u], tl) : ST_NON;
        return;
    }
    bool live[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        live[u] = act[u];
        if (QT == QPI || QT == QPNI || QT == QPIN) {
            const bool e = act[u] && edge_test(g, F[1], anc[1], rel[2], c[u], n0[u], n1[u], tl);
            live[u] = act[u] && (QT == QPIN ? !e : e);
        }
    }
    const int32_t rb = chain_r1<QT> ? rel[1] : rel[2];
    int2 sr[2];
    group_find2(g.rev, n0, n1, live, rb, sr, tl);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        st[u] = ST_NON;
        if (!live[u]) continue;
        if (sr[u].y == sr[u].x) {
            if (QT == QPNI) st[u] = ST_ANS;   // nothing reaches c through the complemented chain
            continue;
        }
        if (sr[u].y - sr[u].x > LANE_SEG || !F[0].lds || (two_cached<QT> && !F[1].lds)) {
            st[u] = ST_PEND;
        } else {
            lst[u] = sr[u];
            st[u] = ST_DEEP;
        }
    }
}

// Then the deep decision: the backward list y[0..len) of c (len <= LANE_SEG)
// against the staged forward list(s); for 3p one more backward step from
// every y.
template <int QT, class T>
__device__ __forceinline__ int32_t deep_test(const GraphView& g, const FSet* F, const int32_t* rel,
                                             int32_t start, int32_t len, T& tl)
{
    int32_t y[LANE_SEG];
#pragma unroll
    for (int k = 0; k < LANE_SEG; ++k) y[k] = k < len ? g.rev.nbr[start + k] : -1;
    tl.read(g.rev.nbr + start, 4 * len);
    if (QT != Q3P) {
        bool hit = false;
#pragma unroll
        for (int k = 0; k < LANE_SEG; ++k) {
            if (k >= len) break;
            if (chain_r1<QT>) hit = hit || has(F[0], y[k], tl);
            else if (QT == QIP) hit = hit || (has(F[0], y[k], tl) && has(F[1], y[k], tl));
            else if (QT == QINP) hit = hit || (has(F[0], y[k], tl) && !has(F[1], y[k], tl));
            else hit = hit || has(F[0], y[k], tl) || has(F[1], y[k], tl);
        }
        // pni: a meeting chain means c is in the complemented set
        return (QT == QPNI ? !hit : hit) ? ST_ANS : ST_NON;
    }
    // 3p: node pairs and signatures of every y at once, then each y's
    // group under r1 (skipped when y's signature lacks r1's class: y then
    // has no in-edge under r1)
    int32_t a0[LANE_SEG], a1[LANE_SEG];
    uint32_t sg[LANE_SEG];
    const uint32_t b1 = sig_bit(rel[1]);
#pragma unroll
    for (int k = 0; k < LANE_SEG; ++k) {
        a0[k] = 0;
        a1[k] = 0;
        sg[k] = 0;
        if (k < len) {
            a0[k] = g.rev.node[y[k]];
            a1[k] = g.rev.node[y[k] + 1];
            sg[k] = g.sig[y[k]];
            tl.read(g.rev.node + y[k], 8);
            tl.read(g.sig + y[k], 1);
        }
    }
    for (int k = 0; k < len; ++k) {
        if (!(sg[k] & b1)) continue;
        const int2 s2 = group_find(g.rev, a0[k], a1[k], rel[1], tl);
        const int32_t n2 = s2.y - s2.x;
        if (n2 > LANE_SEG) return ST_PEND;
        int32_t x[LANE_SEG];
#pragma unroll
        for (int m = 0; m < LANE_SEG; ++m) x[m] = m < n2 ? g.rev.nbr[s2.x + m] : -1;
        tl.read(g.rev.nbr + s2.x, 4 * n2);
        bool hit = false;
#pragma unroll
        for (int m = 0; m < LANE_SEG; ++m)
            if (m < n2) hit = hit || has(F[0], x[m], tl);
        if (hit) return ST_ANS;
    }
    return ST_NON;
}

// Wavefront decision for a queued candidate (the one-hop operand of
// pi / pin / pni has already been tested at lane level).
// s is the candidate's backward list under the last relation (wave-uniform).
template <int QT, class T>
__device__ bool heavy_test(const GraphView& g, const FSet* F, const int32_t* rel, int2 s, int lane,
                           T& tl)
{
    const int32_t* S = g.rev.nbr + s.x;
    const int32_t ns = s.y - s.x;
    if (QT == Q2P || QT == QPI || QT == QPIN) return wave_meet(S, ns, true, F[0].p, F[0].n, false, lane, tl);
    if (QT == QPNI) return !wave_meet(S, ns, true, F[0].p, F[0].n, false, lane, tl);
    if (QT == QIP) return wave_meet3(S, ns, F[0], F[1], lane, tl);
    if (QT == QINP) return wave_meet_minus(S, ns, F[0], F[1], lane, tl);
    if (QT == QUP)
        return wave_meet(S, ns, true, F[0].p, F[0].n, false, lane, tl) ||
               wave_meet(S, ns, true, F[1].p, F[1].n, false, lane, tl);
    if (QT == Q3P) {
        // second backward step for 64 entities y of R_r2(c) at a time; every
        // pair (y, key) with key from the shorter of R_r1(y) and F0 is one
        // search in the longer, and all pairs of the 64 y's are spread over
        // the wavefront, four per lane, so they share one search chain
        for (int32_t k = 0; k < ns; k += 64) {
            if (lane == 0) tl.read(S + k, 4 * min(64, ns - k));
            int2 s2 = make_int2(0, 0);
            if (k + lane < ns) {
                // y without an in-edge under r1's signature class has none under r1
                const int32_t y = S[k + lane];
                tl.read(g.sig + y, 1);
                if (g.sig[y] & sig_bit(rel[1])) s2 = group_range(g.rev, y, rel[1], tl);
            }
            const int32_t len = s2.y - s2.x;
            const bool keys_in_list = len <= F[0].n;       // search R_r1(y) entries in F0
            const int32_t npair = len > 0 ? min(len, F[0].n) : 0;
            int32_t incl = npair;                           // inclusive prefix over the lanes
            for (int d = 1; d < 64; d <<= 1) {
                const int32_t v = __shfl_up(incl, d);
                if (lane >= d) incl += v;
            }
            const int32_t total = uni(__shfl(incl, 63));
            const int32_t excl = incl - npair;
            for (int32_t p0 = 0; p0 < total; p0 += 256) {
                const int32_t* Bk[4];
                int32_t nbk[4], x[4];
                bool cnt[4], found[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int32_t pi = p0 + 64 * u + lane;
                    const int32_t pq = pi < total ? pi : total - 1;
                    // owner lane of pair pq: the highest lane whose exclusive
                    // prefix is <= pq (binary lifting, every lane active)
                    int32_t lo = 0;
#pragma unroll
                    for (int step = 32; step >= 1; step >>= 1) {
                        const int32_t cand = lo + step;
                        const int32_t ev = __shfl(excl, cand > 63 ? 63 : cand);
                        if (cand <= 63 && ev <= pq) lo = cand;
                    }
                    const int32_t off = pq - __shfl(excl, lo);
                    const int32_t lx = __shfl(s2.x, lo);
                    const int32_t ln = __shfl(len, lo);
                    const int32_t kil = __shfl((int32_t)keys_in_list, lo);
                    Bk[u] = F[0].p;
                    nbk[u] = 0;
                    x[u] = -1;
                    cnt[u] = false;
                    if (pi < total) {
                        if (kil) {
                            x[u] = g.rev.nbr[lx + off];
                            tl.read(g.rev.nbr + lx + off, 4);
                            Bk[u] = F[0].p;
                            nbk[u] = F[0].n;
                        } else {
                            x[u] = F[0].p[off];
                            Bk[u] = g.rev.nbr + lx;
                            nbk[u] = ln;
                            cnt[u] = true;
                        }
                    }
                }
                search4v(Bk, nbk, x, cnt, found, tl);
                if (__ballot(found[0] || found[1] || found[2] || found[3])) return true;
            }
        }
        return false;
    }
    return false;
}

__device__ __forceinline__ bool query_ok(const GraphView& g, const smore_sample_out& out, int32_t b,
                                         int n_anc, int n_rel, int32_t R, int32_t* anc, int32_t* rel)
{
    bool ok = !out.positive || out.positive[b] >= 0;   // verification has no positives
    for (int k = 0; k < 3; ++k) {
        rel[k] = out.relations[3 * (int64_t)b + k];
        anc[k] = out.anchors[3 * (int64_t)b + k];
        if (k < n_rel && (rel[k] < 0 || rel[k] >= R)) ok = false;
        if (k < n_anc && (anc[k] < 0 || anc[k] >= g.V)) ok = false;
    }
    return ok;
}

// Per query: validity, forward-cached lists, staging plan, active list.
// Four neighbouring lanes per query: lane f looks up list f, so the
// dependent lookups of a query's lists run side by side; the staging plan
// is made from the sizes of all its lists, in list order.
template <int QT, class T>
__global__ __launch_bounds__(256) void k_prepare(GraphView g, SampleParams p, smore_sample_out out,
                                                 Ws ws, int64_t* stats, int32_t R)
{
    const int32_t gid = blockIdx.x * blockDim.x + threadIdx.x;
    const int32_t b = gid >> 2;
    const int f = gid & 3;
    if (b >= p.batch) return;   // whole groups: 4 divides the workgroup size
    if (gid == 0) {   // queue and list counters of the first round: every query is listed
        ws.ctrl[0] = 0;
        ws.ctrl[1] = 0;
        ws.ctrl[2] = p.batch;
        ws.ctrl[3] = 0;
        ws.ctrl[5] = 0;
    }
    int32_t anc[3], rel[3];
    int32_t* q = ws.qf + (int64_t)b * QF;
    if (f == 0) {
        ws.act[0][b] = b;
        if (stats)
            for (int k = 0; k < 4; ++k) stats[4 * (int64_t)b + k] = 0;
    }
    if (!query_ok(g, out, b, Shape<QT>::n_anc, Shape<QT>::n_rel, R, anc, rel)) {
        if (f == 0) {
            write_undrawn_row(p, out, b, false);
            q[6] = -1;   // skipped by the rounds
        }
        return;
    }
    T tl;
    int2 r = make_int2(0, 0);
    if (f < Shape<QT>::nf) {
        r = group_range(g.fwd, anc[Shape<QT>::fa[f]], rel[Shape<QT>::fr[f]], tl);
        q[2 * f] = r.x;
        q[2 * f + 1] = r.y;
    }
    const int base = (threadIdx.x & 63) & ~3;
    int32_t used = 0, staged = 0;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        const int32_t n = __shfl(r.y - r.x, base + k);
        if (k < Shape<QT>::nf && n <= STAGE - used) {
            staged |= 1 << k;
            used += n;
        }
    }
    if (f == 0) q[6] = staged;
    if constexpr (T::on) {
        // forward caching reads the list once; a staged anchor list too
        if (f < Shape<QT>::nf && (Shape<QT>::cached[f] || (staged >> f & 1)))
            tl.read(g.fwd.nbr + r.x, 4 * (r.y - r.x));
        uint64_t x = tl.b, y = tl.l;
        x += __shfl_xor(x, 1);
        y += __shfl_xor(y, 1);
        x += __shfl_xor(x, 2);
        y += __shfl_xor(y, 2);
        if (f == 0) {
            stats[4 * (int64_t)b] = (int64_t)x;
            stats[4 * (int64_t)b + 1] = (int64_t)y;
        }
    }
}

// Calls with n_neg = 0 draw nothing: one thread per query writes its
// n_valid (0, or -1 for a skipped query), and for per-query sampling its
// draw count.  No workspace is read or written.
template <int QT>
__global__ __launch_bounds__(256) void k_no_draws(GraphView g, SampleParams p, smore_sample_out out,
                                                  int64_t* stats, int32_t R)
{
    const int32_t b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= p.batch) return;
    int32_t anc[3], rel[3];
    const bool ok = query_ok(g, out, b, Shape<QT>::n_anc, Shape<QT>::n_rel, R, anc, rel);
    write_undrawn_row(p, out, b, ok);
    if (stats)
        for (int k = 0; k < 4; ++k) stats[4 * (int64_t)b + k] = 0;
}

// One wavefront per active query, in one-wave workgroups: a workgroup per
// query in the first round, persistent over the list in later rounds (no
// workgroup barrier).  The query's lists are
// staged once into the wave's LDS slice.  Draws are taken WIN at a time:
// every lane computes WIN / 64 draws and reads their in-edge bits (all
// loads in flight together); the draws with an in-edge are compacted into
// the wave's survivor list and then verified one per lane, so a window
// costs one dependent chain per 64 survivors instead of one per draw slot.
constexpr int WIN = 576;
constexpr int DPW = WIN / 64;
static_assert(SMORE_MAX_NEG_TRIES <= 4096 && LANE_SEG <= 8, "deep items pack j and length in 15 bits");

__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// SH: the candidates are the minibatch's shared set p.shared (j < its
// size) instead of the query's own draws.
template <int QT, class T, bool SH = false>
__global__ __launch_bounds__(CWG) void k_candidates(GraphView g, SampleParams p, smore_sample_out out,
                                                    Ws ws, int64_t* stats, int cur, int32_t j0,
                                                    int32_t j1)
{
    if constexpr (SH)
        if (p.n_shared) j1 = min(j1, uni(*p.n_shared));
    __shared__ int32_t stage_all[CWG / 64][STAGE];
    __shared__ int32_t sc_all[CWG / 64][WIN];
    __shared__ uint16_t sj_all[CWG / 64][WIN];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int32_t* stage = stage_all[w];
    int32_t* sc = sc_all[w];
    uint16_t* sj = sj_all[w];
    const uint64_t below = lanes_below(lane);
    const int32_t nact = uni(ws.ctrl[2 + cur]);
    const int32_t nwaves = gridDim.x * (CWG / 64);
    T tl;
    for (int32_t qi = uni(blockIdx.x * (CWG / 64) + w); qi < nact; qi += nwaves) {
        // the first round lists every query in order: the list is not read
        const int32_t b = j0 == 0 ? qi : uni(ws.act[cur][qi]);
        int32_t anc[3], rel[3];
        for (int k = 0; k < 3; ++k) {
            anc[k] = uni(out.anchors[3 * (int64_t)b + k]);
            rel[k] = uni(out.relations[3 * (int64_t)b + k]);
        }
        const int32_t* qb = ws.qf + (int64_t)b * QF;
        const int32_t staged = uni(qb[6]);
        if (staged < 0) continue;   // query without a valid positive
        // this round's draws: [j0, j1) in the first round, else the query's
        // own range, set by the previous round's selection
        int32_t qj0 = j0, qj1 = j1;
        if (j0 < 0) {
            const int32_t rg = uni(qb[7]);
            qj0 = range_lo(rg);
            qj1 = range_hi(rg);
        }
        FSet F[3];
        int32_t sbeg[3], used = 0;
#pragma unroll
        for (int f = 0; f < 3; ++f) {
            sbeg[f] = 0;
            if (f >= Shape<QT>::nf) { F[f] = FSet{nullptr, 0, true}; continue; }
            const int32_t beg = uni(qb[2 * f]), n = uni(qb[2 * f + 1]) - beg;
            if (staged >> f & 1) {
                sbeg[f] = beg;
                F[f] = FSet{stage + used, n, true};
                used += n;
            } else {
                F[f] = FSet{g.fwd.nbr + beg, n, false};
            }
        }
        // copy of the staged lists into the wave's LDS slice
        auto stage_lists = [&]() {
#pragma unroll
            for (int f = 0; f < 3; ++f) {
                if (f >= Shape<QT>::nf || !(staged >> f & 1)) continue;
                int32_t* dst = stage + (F[f].p - stage);
                for (int32_t k = lane; k < F[f].n; k += 64) dst[k] = g.fwd.nbr[sbeg[f] + k];
            }
            wave_sync();
        };
        uint8_t* sv = ws.status + (int64_t)b * p.neg_tries;
        // first test of every draw: the staged root-edge lists when the
        // shape has them (LDS only), else the in-edge mask; in the latter
        // case the lists are copied while the first window's mask words
        // are in flight
        constexpr int RM = RootLists<QT>::mask;
        const bool use_lists = RM != 0 && (RootLists<QT>::any ? (staged & RM) == RM : (staged & RM) != 0);
        // signature bits an answer must carry
        uint32_t need = 0;
#pragma unroll
        for (int k = 0; k < 3; ++k)
            if (RootRels<QT>::mask >> k & 1) need |= sig_bit(rel[k]);
        bool to_stage = used > 0;
        if (use_lists) {
            stage_lists();
            to_stage = false;
        }
        for (int32_t base = qj0; base < qj1; base += WIN) {
            // Every answer of every shape is reached by a projection, so a
            // draw without an in-edge is a non-answer: the in-edge mask (V
            // bits, resident in the last-level cache) decides most draws.
            // On a large graph the coarse mask (one bit per four entities,
            // small enough for the L2) is read first, and only draws whose
            // group of four has an in-edge read their in-relation
            // signature (a byte per entity), which must hold the bits of
            // the relations that end at the root: a draw with in-edges
            // only under other relation classes is a non-answer too.
            int32_t c[DPW];
            uint32_t word[DPW];
            const bool two_level = !use_lists && g.coarse;
#pragma unroll
            for (int k = 0; k < DPW; ++k) {
                const int32_t j = base + k * 64 + lane;
                c[k] = 0;
                word[k] = 0;
                if (j < qj1) {
                    c[k] = candidate(p, g.V, b, j);   // -1 (given candidates only): never a negative
                    if (!use_lists && c[k] >= 0)
                        word[k] = two_level ? g.has_in4[c[k] >> 7] : g.has_in[c[k] >> 5];
                }
            }
            if (to_stage) {
                stage_lists();
                to_stage = false;
            }
            if (two_level) {
#pragma unroll
                for (int k = 0; k < DPW; ++k) {
                    // accounted as one mask line per draw, as the one-level test
                    const bool live = base + k * 64 + lane < qj1 && c[k] >= 0;
                    const bool maybe = live && ((word[k] >> ((c[k] >> 2) & 31)) & 1u);
                    if (live) tl.read(g.has_in4 + (c[k] >> 7), 4);
                    const uint32_t sg = maybe ? (uint32_t)g.sig[c[k]] : 0u;
                    const bool pass = RootRels<QT>::any ? (sg & need) != 0 : (sg & need) == need;
                    word[k] = pass ? ~0u : 0u;
                }
            }
            if (use_lists) {
#pragma unroll
                for (int k = 0; k < DPW; ++k) {
                    if (c[k] < 0) continue;   // (candidates given by the caller only)
                    bool hit = !RootLists<QT>::any;
#pragma unroll
                    for (int f = 0; f < 3; ++f) {
                        if (!(RM >> f & 1) || !(staged >> f & 1)) continue;
                        const bool h = has(F[f], c[k], tl);
                        hit = RootLists<QT>::any ? (hit || h) : (hit && h);
                    }
                    word[k] = hit ? ~0u : 0u;
                }
            }
            int32_t nsurv = 0;
#pragma unroll
            for (int k = 0; k < DPW; ++k) {
                const int32_t j = base + k * 64 + lane;
                const bool live = j < qj1;
                const bool in = live && c[k] >= 0 && ((word[k] >> (c[k] & 31)) & 1u);
                if (live) {
                    if (!use_lists && !two_level && c[k] >= 0) tl.read(g.has_in + (c[k] >> 5), 4);
                    if (!in) sv[j] = c[k] >= 0 ? ST_NON : ST_DUP;   // ST_DUP: not an entity
                }
                const uint64_t m = __ballot(in);
                if (in) {
                    const int32_t at = nsurv + __popcll(m & below);
                    sc[at] = c[k];
                    sj[at] = (uint16_t)j;
                }
                nsurv += __popcll(m);
            }
            wave_sync();
            // shallow pass over the survivors, 64 at a time; candidates with
            // a short backward list are collected (in place, over entries
            // already consumed) for one deep pass, so the dependent steps of
            // the window's few deep candidates overlap
            int32_t ndeep = 0;
            for (int32_t s0 = 0; s0 < nsurv; s0 += 128) {
                bool act[2];
                int32_t cc[2], jj[2], st[2];
                int2 lst[2] = {make_int2(0, 0), make_int2(0, 0)};
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    const int32_t at = s0 + 64 * u + lane;
                    act[u] = at < nsurv;
                    cc[u] = act[u] ? sc[at] : 0;
                    jj[u] = act[u] ? sj[at] : 0;
                }
                wave_sync();
                shallow_test2<QT>(g, F, anc, rel, cc, act, st, lst, tl);
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    if (act[u] && st[u] != ST_DEEP) {
                        sv[jj[u]] = (uint8_t)st[u];
                        if (st[u] == ST_PEND) {
                            const int32_t slot = atomicAdd(&ws.ctrl[0], 1);   // capacity covers a round
                            ws.queue[slot] = make_int2(b, jj[u]);
                        }
                    }
                    const bool deep = act[u] && st[u] == ST_DEEP;
                    const uint64_t m = __ballot(deep);
                    if (deep) {
                        // j < 4096 and 1 <= length <= 8 pack into 15 bits
                        const int32_t at = ndeep + __popcll(m & below);
                        sc[at] = lst[u].x;
                        sj[at] = (uint16_t)((jj[u] << 3) | (lst[u].y - lst[u].x - 1));
                    }
                    ndeep += __popcll(m);
                }
            }
            wave_sync();
            for (int32_t d0 = 0; d0 < ndeep; d0 += 64) {
                if (d0 + lane < ndeep) {
                    const int32_t start = sc[d0 + lane], pk = sj[d0 + lane];
                    const int32_t j = pk >> 3;
                    const int32_t st = deep_test<QT>(g, F, rel, start, (pk & 7) + 1, tl);
                    sv[j] = (uint8_t)st;
                    if (st == ST_PEND) {
                        const int32_t slot = atomicAdd(&ws.ctrl[0], 1);
                        ws.queue[slot] = make_int2(b, j);
                    }
                }
            }
            wave_sync();   // the next window reuses the survivor list
        }
        flush_tally(tl, stats, b, lane);
        wave_sync();   // the next query restages the wave's slice
    }
}

// Persistent wavefronts draining the heavy queue.  Wavefront w takes items
// w, w + nwaves, ... (no shared counter to contend on).  It looks up its
// next 64 items at once, one per lane: the queue entry, the candidate, the
// query's relations and cached lists, and the candidate's backward list,
// so those dependent reads overlap instead of preceding each test in turn.
template <int QT, class T>
__global__ __launch_bounds__(HEAVY_WG) void k_heavy(GraphView g, SampleParams p, smore_sample_out out,
                                                    Ws ws, int64_t* stats, int nxt)
{
    constexpr int NF = Shape<QT>::nf;
    const int lane = threadIdx.x & 63;
    // the compaction that follows appends to the next round's list
    if (blockIdx.x == 0 && threadIdx.x == 0) ws.ctrl[2 + nxt] = 0;
    const int32_t total = uni(ws.ctrl[0]);
    const int32_t nwaves = gridDim.x * (HEAVY_WG / 64);
    const int32_t w0 = uni(blockIdx.x * (HEAVY_WG / 64) + (threadIdx.x >> 6));
    T tl;
    for (int64_t base = w0; base < total; base += 64 * (int64_t)nwaves) {
        const int64_t mine = base + (int64_t)lane * nwaves;
        int32_t mb = 0, mc = 0;
        int64_t mat = 0;
        int32_t mrel[3] = {0, 0, 0}, mf[2 * NF];
        int2 ms = make_int2(0, 0);
#pragma unroll
        for (int f = 0; f < 2 * NF; ++f) mf[f] = 0;
        if (mine < total) {
            const int2 it = ws.queue[mine];
            mb = it.x;
            mat = (int64_t)it.x * p.neg_tries + it.y;
            mc = candidate(p, g.V, it.x, it.y);
#pragma unroll
            for (int k = 0; k < 3; ++k) mrel[k] = out.relations[3 * (int64_t)mb + k];
            const int32_t* qb = ws.qf + (int64_t)mb * QF;
#pragma unroll
            for (int f = 0; f < 2 * NF; ++f) mf[f] = qb[f];
            ms = group_range(g.rev, mc, chain_r1<QT> ? mrel[1] : mrel[2]);
        }
        const int32_t n = uni((int32_t)min((int64_t)64, (total - base + nwaves - 1) / nwaves));
        for (int k = 0; k < n; ++k) {
            const int32_t b = readlane(mb, k);
            int32_t rel[3];
#pragma unroll
            for (int q = 0; q < 3; ++q) rel[q] = readlane(mrel[q], k);
            FSet F[3];
#pragma unroll
            for (int f = 0; f < 3; ++f) {
                if (f < NF) {
                    const int32_t beg = readlane(mf[2 * f], k), end = readlane(mf[2 * f + 1], k);
                    F[f] = FSet{g.fwd.nbr + beg, end - beg, false};
                } else {
                    F[f] = FSet{nullptr, 0, true};
                }
            }
            if constexpr (T::on) {
                // the candidate's lookup, charged once to its query
                T one;
                (void)group_range(g.rev, readlane(mc, k), chain_r1<QT> ? rel[1] : rel[2], one);
                if (lane == 0) tl = one;
            }
            const int2 s = make_int2(readlane(ms.x, k), readlane(ms.y, k));
            const bool ans = heavy_test<QT>(g, F, rel, s, lane, tl);
            if (lane == 0) ws.status[readlane64(mat, k)] = ans ? ST_ANS : ST_NON;
            flush_tally(tl, stats, b, lane, 2);
        }
    }
}

// Highest lane whose exclusive prefix excl is <= idx (binary lifting over
// the wavefront; every lane must be active).  excl is nondecreasing over
// the lanes and 0 in lane 0.
__device__ __forceinline__ int owner_lane(int32_t idx, int32_t excl)
{
    int lo = 0;
#pragma unroll
    for (int step = 32; step >= 1; step >>= 1) {
        const int cand = lo + step;
        const int32_t ev = __shfl(excl, cand > 63 ? 63 : cand);
        if (cand <= 63 && ev <= idx) lo = cand;
    }
    return lo;
}

__device__ __forceinline__ int32_t excl_prefix(int32_t v, int lane, int32_t* total)
{
    int32_t incl = v;
    for (int d = 1; d < 64; d <<= 1) {
        const int32_t t = __shfl_up(incl, d);
        if (lane >= d) incl += t;
    }
    *total = uni(__shfl(incl, 63));
    return incl - v;
}

// OR of a 64-bit value over the wavefront.
__device__ __forceinline__ uint64_t wave_or(uint64_t x)
{
    for (int s = 32; s > 0; s >>= 1)
        x |= (uint64_t)(uint32_t)__shfl_xor((int32_t)(uint32_t)x, s) |
             ((uint64_t)(uint32_t)__shfl_xor((int32_t)(x >> 32), s) << 32);
    return x;
}

// A slice of one queued 3p item, held by one lane: the item's draw (its
// query b and state index mat), relation r1, forward list F0 = A_r0(a0)
// (edges [f0b, f0b + f0n)), the candidate's list S = R_r2(c) (edges from
// sx), the range [y0, y1) of S's entities to expand and, for each of them,
// the range [k0, k1) of its (y, key) pairs to search (keys from the shorter
// of R_r1(y) and F0).
struct Slice3 {
    bool valid = false;
    int32_t b = -1;
    int64_t mat = 0;
    int32_t r1 = 0, f0b = 0, f0n = 0, sx = 0, y0 = 0, y1 = 0, k0 = 0, k1 = 0;
};

// Reserve n unit slots for a wavefront (all lanes call it with the same n):
// the first slot, or -1 when the queue is full, in which case the slots of
// the failed reservation that lie inside the queue are marked unused.
__device__ __forceinline__ int64_t reserve_units(Ws& ws, int32_t n, int lane)
{
    int32_t base = INT_MAX;
    // once the queue is full the counter is left alone (it cannot grow without bound)
    if (lane == 0 && ws.ctrl[5] < ws.ucap) base = atomicAdd(&ws.ctrl[5], n);
    base = uni(__shfl(base, 0));
    if ((int64_t)base + n <= ws.ucap) return base;
    for (int64_t k = (int64_t)base + lane; k < ws.ucap; k += 64) ws.units[k] = make_int4(-1, 0, 0, 2);
    return -1;
}

// Decide the slices of a wavefront, one per lane: the entities y of all of
// them expanded 64 at a time (signature class, then the group under r1),
// and the (y, key) pairs of all of them searched 256 at a time; a hit makes
// its slice's item an answer, whose remaining y's and pairs are dropped,
// the rest being laid out again after every step.  With PUSH (the
// long-list kernel), y's beyond the first UNIT_Y of a slice and pairs
// beyond the first UNIT_PAIRS of one y go to the unit queue (item index q)
// when it has room, else they are decided here.  Returns the answer bits.
template <bool PUSH, class T>
__device__ uint64_t decide_slices3(const GraphView& g, Ws& ws, Slice3 w, int64_t q, int lane, T& tl)
{
    if constexpr (PUSH) {
        const int32_t ny = w.valid ? w.y1 - w.y0 : 0;
        const int32_t nu = ny > UNIT_Y ? (ny - UNIT_Y + UNIT_Y - 1) / UNIT_Y : 0;
        int32_t tot;
        const int32_t ex = excl_prefix(nu, lane, &tot);
        if (tot > 0) {
            const int64_t at = reserve_units(ws, tot, lane);
            if (at >= 0) {
                for (int32_t k = 0; k < nu; ++k) {
                    const int32_t a = w.y0 + UNIT_Y * (k + 1);
                    ws.units[at + ex + k] = make_int4((int32_t)q, a, min(a + UNIT_Y, w.y1), 0);
                }
                if (nu > 0) w.y1 = w.y0 + UNIT_Y;
            }
        }
    }
    uint64_t ans = 0;     // bit i: the item of lane i is an answer
    int32_t ydone = 0;    // y's of this lane's slice expanded so far
    for (;;) {
        const int32_t yrem = (!w.valid || ((ans >> lane) & 1)) ? 0 : (w.y1 - w.y0) - ydone;
        int32_t ytotal;
        const int32_t yex = excl_prefix(yrem, lane, &ytotal);
        if (ytotal == 0) break;
        const int it = owner_lane(min(lane, ytotal - 1), yex);
        const int32_t ypos = __shfl(w.y0, it) + __shfl(ydone, it) + lane - __shfl(yex, it);
        const int32_t isx = __shfl(w.sx, it), ir1 = __shfl(w.r1, it);
        const int32_t if0b = __shfl(w.f0b, it), if0n = __shfl(w.f0n, it);
        int32_t k0 = __shfl(w.k0, it), k1 = __shfl(w.k1, it);
        int2 s2 = make_int2(0, 0);
        if (lane < ytotal) {
            // y without an in-edge under r1's signature class has none under r1
            const int32_t y = g.rev.nbr[isx + ypos];
            tl.read(g.rev.nbr + isx + ypos, 4);
            tl.read(g.sig + y, 1);
            if (g.sig[y] & sig_bit(ir1)) s2 = group_range(g.rev, y, ir1, tl);
        }
        const int32_t len = s2.y - s2.x;
        const bool kil = len <= if0n;            // search R_r1(y)'s entries in F0
        const int32_t nall = len > 0 ? min(len, if0n) : 0;
        if constexpr (PUSH) {
            // pairs beyond the first UNIT_PAIRS of a y: units of UNIT_PAIRS keys
            const int32_t nu = nall > UNIT_PAIRS ? (nall - 1) / UNIT_PAIRS : 0;
            if (__ballot(nu > 0)) {
                int32_t tot;
                const int32_t ex = excl_prefix(nu, lane, &tot);
                const int64_t at = reserve_units(ws, tot, lane);
                if (at >= 0) {
                    const int32_t iq = __shfl((int32_t)q, it);
                    for (int32_t k = 0; k < nu; ++k)
                        ws.units[at + ex + k] = make_int4(iq, ypos, UNIT_PAIRS * (k + 1), 1);
                    if (nu > 0) k1 = UNIT_PAIRS;
                }
            }
        }
        const int32_t kb = min(k0, nall), ke = min(k1, nall);   // this y's keys [kb, ke)
        int32_t pdone = 0;
        for (;;) {
            const int32_t rem = ((ans >> it) & 1) ? 0 : ke - kb - pdone;
            int32_t ptotal;
            const int32_t pex = excl_prefix(rem, lane, &ptotal);
            if (ptotal == 0) break;
            const int32_t* Bk[4];
            int32_t nbk[4], x[4], who[4];
            bool cnt[4], found[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int32_t pi = 64 * u + lane;
                const int32_t pq = pi < ptotal ? pi : ptotal - 1;
                const int yl = owner_lane(pq, pex);
                const int32_t off = __shfl(kb, yl) + __shfl(pdone, yl) + pq - __shfl(pex, yl);
                const int32_t lx = __shfl(s2.x, yl), ln = __shfl(len, yl);
                const int32_t k_in_l = __shfl((int32_t)kil, yl);
                const int32_t fb = __shfl(if0b, yl), fn = __shfl(if0n, yl);
                who[u] = __shfl(it, yl);
                Bk[u] = g.fwd.nbr + fb;
                nbk[u] = 0;
                x[u] = -1;
                cnt[u] = false;
                if (pi < ptotal) {
                    if (k_in_l) {
                        x[u] = g.rev.nbr[lx + off];
                        tl.read(g.rev.nbr + lx + off, 4);
                        nbk[u] = fn;
                    } else {
                        x[u] = g.fwd.nbr[fb + off];
                        Bk[u] = g.rev.nbr + lx;
                        nbk[u] = ln;
                        cnt[u] = true;
                    }
                }
            }
            search4q(Bk, nbk, x, cnt, found, tl);
            uint64_t m = 0;
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (found[u]) m |= 1ull << who[u];
            ans |= wave_or(m);
            pdone += min(rem, max(0, 256 - pex));   // this step took pairs pex .. 255
        }
        ydone += min(yrem, max(0, 64 - yex));       // this chunk took y's yex .. 63
    }
    return ans;
}

// The slice of queued item qi: the whole list S, all keys.
template <class T>
__device__ __forceinline__ Slice3 item_slice3(const GraphView& g, const SampleParams& p,
                                              const smore_sample_out& out, const Ws& ws, int64_t qi, T& tl)
{
    Slice3 w;
    const int2 it = ws.queue[qi];
    w.valid = true;
    w.b = it.x;
    w.mat = (int64_t)it.x * p.neg_tries + it.y;
    const int32_t c = candidate(p, g.V, it.x, it.y);
    w.r1 = out.relations[3 * (int64_t)w.b + 1];
    const int32_t r2 = out.relations[3 * (int64_t)w.b + 2];
    const int32_t* qb = ws.qf + (int64_t)w.b * QF;
    w.f0b = qb[0];
    w.f0n = qb[1] - w.f0b;
    const int2 S = group_range(g.rev, c, r2, tl);
    w.sx = S.x;
    w.y0 = 0;
    w.y1 = S.y - S.x;
    w.k0 = 0;
    w.k1 = INT_MAX;
    return w;
}

// The long-list kernel of 3p, batched: wavefront w takes items w,
// w + nwaves, ... like k_heavy, but decides up to 64 of them together, one
// per lane (decide_slices3), so their dependent chains overlap instead of
// running one item after the other; the parts of huge items go to the unit
// queue.  It writes every item's state.  With the read tally, a batch's
// reads are charged to the query of its first item (the sums over all
// queries are exact).
template <class T>
__global__ __launch_bounds__(HEAVY_WG) void k_heavy3(GraphView g, SampleParams p, smore_sample_out out,
                                                     Ws ws, int64_t* stats, int nxt)
{
    const int lane = threadIdx.x & 63;
    if (blockIdx.x == 0 && threadIdx.x == 0) ws.ctrl[2 + nxt] = 0;
    const int32_t total = uni(ws.ctrl[0]);
    const int32_t nwaves = gridDim.x * (HEAVY_WG / 64);
    const int32_t w0 = uni(blockIdx.x * (HEAVY_WG / 64) + (threadIdx.x >> 6));
    T tl;
    for (int64_t base = w0; base < total; base += 64 * (int64_t)nwaves) {
        const int64_t mine = base + (int64_t)lane * nwaves;
        Slice3 w;
        if (mine < total) w = item_slice3(g, p, out, ws, mine, tl);
        const uint64_t ans = decide_slices3<true>(g, ws, w, mine, lane, tl);
        if (mine < total) ws.status[w.mat] = ((ans >> lane) & 1) ? ST_ANS : ST_NON;
        flush_tally(tl, stats, uni(__shfl(w.b, 0)), lane, 2);
    }
}

// The units the long-list kernel left: wavefront w takes units w,
// w + nwaves, ..., up to 64 at a time, one per lane; a unit of an item
// already decided an answer is skipped, and a hit makes its item an answer
// (units never clear a state, so their order does not matter).
template <class T>
__global__ __launch_bounds__(HEAVY_WG) void k_units3(GraphView g, SampleParams p, smore_sample_out out,
                                                     Ws ws, int64_t* stats)
{
    const int lane = threadIdx.x & 63;
    const int32_t total = uni((int32_t)min((int64_t)ws.ctrl[5], ws.ucap));
    const int32_t nwaves = gridDim.x * (HEAVY_WG / 64);
    const int32_t w0 = uni(blockIdx.x * (HEAVY_WG / 64) + (threadIdx.x >> 6));
    T tl;
    for (int64_t base = w0; base < total; base += 64 * (int64_t)nwaves) {
        const int64_t mine = base + (int64_t)lane * nwaves;
        Slice3 w;
        if (mine < total) {
            const int4 u = ws.units[mine];
            if (u.w != 2) {
                w = item_slice3(g, p, out, ws, u.x, tl);
                if (ws.status[w.mat] == ST_ANS) {
                    w.valid = false;
                } else if (u.w == 0) {           // entities [a, b) of S, all keys
                    w.y0 = u.y;
                    w.y1 = u.z;
                } else {                         // entity a of S, keys [b, b + UNIT_PAIRS)
                    w.y0 = u.y;
                    w.y1 = u.y + 1;
                    w.k0 = u.z;
                    w.k1 = u.z + UNIT_PAIRS;
                }
            }
        }
        const uint64_t ans = decide_slices3<false>(g, ws, w, -1, lane, tl);
        if (w.valid && ((ans >> lane) & 1)) ws.status[w.mat] = ST_ANS;
        flush_tally(tl, stats, uni(__shfl(max(w.b, 0), 0)), lane, 2);
    }
}

__device__ __forceinline__ void ht_insert(int32_t* tv, int32_t* tj, uint32_t mask, int shift,
                                          int32_t c, int32_t j)
{
    uint32_t h = ((uint32_t)c * 0x9E3779B1u) >> shift;
    for (;;) {
        const int32_t old = atomicCAS(&tv[h], -1, c);
        if (old == -1 || old == c) {
            atomicMin(&tj[h], j);
            return;
        }
        h = (h + 1) & mask;
    }
}

__device__ __forceinline__ int32_t ht_first(const int32_t* tv, const int32_t* tj, uint32_t mask,
                                            int shift, int32_t c)
{
    uint32_t h = ((uint32_t)c * 0x9E3779B1u) >> shift;
    while (tv[h] != c) h = (h + 1) & mask;
    return tj[h];
}

// Per active query, one wavefront per query (one-wave workgroups; the LDS
// holds the round's first-occurrence table and the query's draws and
// states): keep draw j iff it is not an answer and no earlier draw has the
// same value; the first n_neg kept, in draw order, are the negatives.
// Queries neither complete nor out of budget go to the next round's list
// with their next draw range (next_round_end).
__global__ __launch_bounds__(64) void k_compact(SampleParams p, int32_t V, smore_sample_out out, Ws ws,
                                                int cur, int32_t j_end, int last, int next_last,
                                                int32_t tcap, int tshift, int ident)
{
    extern __shared__ int32_t lds[];
    int32_t* tv = lds;
    int32_t* tj = lds + tcap;
    int32_t* vals = lds + 2 * tcap;
    uint8_t* sts = (uint8_t*)(vals + j_end);
    const int lane = threadIdx.x;
    const uint64_t below = lanes_below(lane);
    const uint32_t tmask = (uint32_t)tcap - 1;
    const int32_t nact = uni(ws.ctrl[2 + cur]);
    // the heavy queue of this round is drained: ready it for the next round
    if (blockIdx.x == 0 && lane == 0) { ws.ctrl[0] = 0; ws.ctrl[1] = 0; ws.ctrl[5] = 0; }
    for (int32_t qi = blockIdx.x; qi < nact; qi += gridDim.x) {
        const int32_t b = uni(ws.act[cur][qi]);
        if (uni(ws.qf[(int64_t)b * QF + 6]) < 0) continue;   // query without a valid positive
        // the query's draws so far (at most j_end, which sizes the LDS)
        const int32_t jq = ident ? j_end : range_hi(uni(ws.qf[(int64_t)b * QF + 7]));
        const uint8_t* sv = ws.status + (int64_t)b * p.neg_tries;
        int32_t* row = out.negatives + (int64_t)b * p.n_neg;
        for (int32_t k = lane; k < tcap; k += 64) { tv[k] = -1; tj[k] = INT_MAX; }
        for (int32_t j = lane; j < jq; j += 64) {
            vals[j] = candidate(p, V, b, j);
            sts[j] = sv[j];
        }
        wave_sync();
        for (int32_t j = lane; j < jq; j += 64) ht_insert(tv, tj, tmask, tshift, vals[j], j);
        wave_sync();
        int32_t acc = 0;
        for (int32_t row0 = 0; row0 < jq && acc < p.n_neg; row0 += 64) {
            const int32_t j = row0 + lane;
            int32_t c = 0;
            bool keep = false;
            if (j < jq) {
                c = vals[j];
                keep = sts[j] == ST_NON && ht_first(tv, tj, tmask, tshift, c) == j;
            }
            const uint64_t m = __ballot(keep);
            const int32_t rank = acc + __popcll(m & below);
            if (keep && rank < p.n_neg) {
                row[rank] = c;
                if (rank == p.n_neg - 1) out.neg_draws[b] = j + 1;
            }
            acc = uni(min(p.n_neg, acc + __popcll(m)));
        }
        if (acc == p.n_neg || last || jq >= p.neg_tries) {
            for (int32_t k = acc + lane; k < p.n_neg; k += 64) row[k] = -1;
            if (lane == 0) {
                out.n_valid[b] = acc;
                if (acc < p.n_neg) out.neg_draws[b] = p.neg_tries;
            }
        } else if (lane == 0) {
            ws.qf[(int64_t)b * QF + 7] = pack_range(jq, next_round_end(p, jq, acc, next_last));
            ws.act[cur ^ 1][atomicAdd(&ws.ctrl[2 + (cur ^ 1)], 1)] = b;
        }
        wave_sync();
    }
}

// The same selection for rounds of at most 64 * CK draws, with every load
// in flight at once: each lane holds its CK draws (j = lane + 64 k) in
// registers, one wavefront per query, four per workgroup, and only the
// hash table lives in LDS.  Only non-answers enter the table: a value's
// state is the same at each of its occurrences, so the first non-answer
// occurrence of a value is its first occurrence.
constexpr int CK = 16;
constexpr int CWAVES = 4;

// One wavefront per listed query; its states are read in one round trip
// while its draws are recomputed (the first round lists every query in
// order, so the list itself is not read then, and the query's validity flag
// is loaded beside the states rather than before them).
template <int NK>
__global__ __launch_bounds__(64 * CWAVES) void k_compact_reg(SampleParams p, int32_t V,
                                                             smore_sample_out out, Ws ws, int cur,
                                                             int32_t j_end, int last, int next_last,
                                                             int32_t tcap, int tshift, int ident)
{
    extern __shared__ int32_t lds[];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int32_t* tv = lds + (size_t)w * tcap;
    const uint64_t below = lanes_below(lane);
    const uint32_t tmask = (uint32_t)tcap - 1;
    const int32_t nact = uni(ws.ctrl[2 + cur]);
    if (blockIdx.x == 0 && threadIdx.x == 0) { ws.ctrl[0] = 0; ws.ctrl[1] = 0; ws.ctrl[5] = 0; }
    for (int32_t qi = uni(blockIdx.x * CWAVES + w); qi < nact; qi += gridDim.x * CWAVES) {
        const int32_t b = ident ? qi : uni(ws.act[cur][qi]);
        const int32_t flag = ws.qf[(int64_t)b * QF + 6];   // < 0: query without a valid positive
        // the query's draws so far: all of the first round, or up to the end
        // of its own range in a later one
        const int32_t jq = ident ? j_end : range_hi(uni(ws.qf[(int64_t)b * QF + 7]));
        const int32_t nk = uni((jq + 63) >> 6);
        const uint8_t* sv = ws.status + (int64_t)b * p.neg_tries;
        int32_t* row = out.negatives + (int64_t)b * p.n_neg;
        int32_t c[NK];
        uint8_t st[NK];
#pragma unroll
        for (int k = 0; k < NK; ++k) {
            const int32_t j = 64 * k + lane;
            c[k] = -1;
            st[k] = ST_ANS;
            if (k < nk && j < jq) st[k] = sv[j];
        }
        // the draws themselves are recomputed while the states are in flight
#pragma unroll
        for (int k = 0; k < NK; ++k) {
            const int32_t j = 64 * k + lane;
            if (k < nk && j < jq) c[k] = candidate(p, V, b, j);
        }
        if (uni(flag) < 0) continue;
        bool non[NK];
#pragma unroll
        for (int k = 0; k < NK; ++k) non[k] = st[k] == ST_NON;
        int4* t4 = (int4*)tv;
        for (int32_t k = lane; k < tcap / 4; k += 64) t4[k] = make_int4(-1, -1, -1, -1);
        wave_sync();
        // insert every non-answer's value; first probes of every draw in
        // flight together, collisions probe on.  A draw that meets its own
        // value in the table has an equal draw (which of the two came first
        // is settled below); slots are never emptied, so two equal values
        // always end in the same slot and one of them meets the other.
        uint32_t h[NK];
        int32_t old[NK];
#pragma unroll
        for (int k = 0; k < NK; ++k) {
            h[k] = ((uint32_t)c[k] * 0x9E3779B1u) >> tshift;
            old[k] = non[k] ? atomicCAS(&tv[h[k]], -1, c[k]) : -1;
        }
        bool dup = false;
#pragma unroll
        for (int k = 0; k < NK; ++k) {
            if (!non[k]) continue;
            uint32_t at = h[k];
            int32_t o = old[k];
            while (o != -1 && o != c[k]) {
                at = (at + 1) & tmask;
                o = atomicCAS(&tv[at], -1, c[k]);
            }
            h[k] = at;
            dup = dup || o == c[k];
        }
        int32_t first[NK];
#pragma unroll
        for (int k = 0; k < NK; ++k) first[k] = non[k] ? 64 * k + lane : -1;
        if (__ballot(dup)) {
            // some value was drawn twice (rare): the first draw of each
            // value is the least draw index over its slot (one slot per
            // value, reused for the minimum)
#pragma unroll
            for (int k = 0; k < NK; ++k)
                if (non[k]) tv[h[k]] = INT_MAX;
            wave_sync();
#pragma unroll
            for (int k = 0; k < NK; ++k)
                if (non[k]) atomicMin(&tv[h[k]], 64 * k + lane);
            wave_sync();
#pragma unroll
            for (int k = 0; k < NK; ++k) first[k] = non[k] ? tv[h[k]] : -1;
        }
        int32_t acc = 0;
#pragma unroll
        for (int k = 0; k < NK; ++k) {
            if (k >= nk || acc >= p.n_neg) break;
            const int32_t j = 64 * k + lane;
            const bool keep = non[k] && first[k] == j;
            const uint64_t m = __ballot(keep);
            const int32_t rank = acc + __popcll(m & below);
            if (keep && rank < p.n_neg) {
                row[rank] = c[k];
                if (rank == p.n_neg - 1) out.neg_draws[b] = j + 1;
            }
            acc = uni(min(p.n_neg, acc + __popcll(m)));
        }
        if (acc == p.n_neg || last || jq >= p.neg_tries) {
            for (int32_t k = acc + lane; k < p.n_neg; k += 64) row[k] = -1;
            if (lane == 0) {
                out.n_valid[b] = acc;
                if (acc < p.n_neg) out.neg_draws[b] = p.neg_tries;
            }
        } else if (lane == 0) {
            ws.qf[(int64_t)b * QF + 7] = pack_range(jq, next_round_end(p, jq, acc, next_last));
            ws.act[cur ^ 1][atomicAdd(&ws.ctrl[2 + (cur ^ 1)], 1)] = b;
        }
        wave_sync();   // the next query clears the table
    }
}

// first-occurrence table of the compaction: load factor at most 0.6
inline int32_t compact_tcap(int32_t j_end)
{
    int32_t tcap = 64;
    while (tcap * 3 < 5 * j_end) tcap <<= 1;
    return tcap;
}

// table (value, first draw) + the query's draws and states
inline size_t compact_lds(int32_t j_end)
{
    return (size_t)2 * compact_tcap(j_end) * sizeof(int32_t) + (size_t)j_end * 5 + 16;
}

inline int check_launch(const char** err)
{
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) { *err = hipGetErrorString(e); return SMORE_E_HIP; }
    return SMORE_OK;
}

// One-shot event pairs of the next negatives call, one per kernel kind
// (0 candidate kernel, 1 long-list kernel, 2 selection), each independent.
struct ProfileArm {
    hipEvent_t start = nullptr, stop = nullptr;
};
thread_local ProfileArm g_prof[3];

// One-shot wait of the next negatives call: its stream waits on this event
// right before the first candidate kernel, after the preparation.
thread_local hipEvent_t g_wait = nullptr;

inline void prof_mark(int which, int round, bool after, hipStream_t st)
{
    ProfileArm& a = g_prof[which];
    if (round != 0 || !a.start || !a.stop) return;
    (void)hipEventRecord(after ? a.stop : a.start, st);
    if (after) a = ProfileArm{};
}

// parts: NEG_PREPARE the per-query preparation, NEG_CANDIDATES the first
// round's candidate kernel, NEG_REST the first round's long-list and
// selection kernels and every later round.
template <int QT, class T>
int run_negatives(const GraphView& gv, const SampleParams& p, const smore_sample_out& out, Ws ws,
                  int64_t* stats, int32_t R, int parts, hipStream_t st, const char** err)
{
    int rc;
    if (p.n_neg == 0) {   // nothing to draw: no preparation, no workspace
        if (!(parts & NEG_PREPARE)) return SMORE_OK;
        k_no_draws<QT><<<(p.batch + 255) / 256, 256, 0, st>>>(gv, p, out, stats, R);
        return check_launch(err);
    }
    if (parts & NEG_PREPARE) {
        k_prepare<QT, T><<<(p.batch + 63) / 64, 256, 0, st>>>(gv, p, out, ws, stats, R);
        if ((rc = check_launch(err))) return rc;
    }
    const int rounds = n_rounds(p);
    for (int r = 0; r < rounds; ++r) {
        const int cur = r & 1;
        // the first round's draws are the same for every query; a later
        // round's are each query's own (j0 = -1), ending at most at neg_tries
        const int32_t j0 = r == 0 ? 0 : -1;
        const int32_t j_end = r == 0 ? first_round(p) : p.neg_tries;
        // later rounds carry the few queries short of n_neg: a smaller grid
        // keeps their (often empty) launches cheap
        const int grid = r == 0 ? PERSIST_BLOCKS : PERSIST_BLOCKS / 4;
        const int cgrid = r == 0 ? max(p.batch, 1) : PERSIST_BLOCKS;   // one-wave workgroups
        if (parts & (r == 0 ? NEG_CANDIDATES : NEG_REST)) {
            if (r == 0 && g_wait) {
                const hipError_t e = hipStreamWaitEvent(st, g_wait, 0);
                g_wait = nullptr;
                if (e != hipSuccess) { *err = hipGetErrorString(e); return SMORE_E_HIP; }
            }
            prof_mark(0, r, false, st);
            k_candidates<QT, T><<<cgrid, CWG, 0, st>>>(gv, p, out, ws, stats, cur, j0, j_end);
            if ((rc = check_launch(err))) return rc;
            prof_mark(0, r, true, st);
        }
        if (!(parts & NEG_REST)) continue;
        prof_mark(1, r, false, st);
        if constexpr (QT == Q3P) {
            // a quarter grid in every round: these waves mostly wait on
            // dependent reads, and at four waves per SIMD a full grid would
            // hold the registers that the candidate kernels of shapes sampled
            // beside this one need
            k_heavy3<T><<<PERSIST_BLOCKS / 4, HEAVY_WG, 0, st>>>(gv, p, out, ws, stats, cur ^ 1);
            if ((rc = check_launch(err))) return rc;
            k_units3<T><<<PERSIST_BLOCKS / 4, HEAVY_WG, 0, st>>>(gv, p, out, ws, stats);
        } else {
            k_heavy<QT, T><<<grid, HEAVY_WG, 0, st>>>(gv, p, out, ws, stats, cur ^ 1);
        }
        if ((rc = check_launch(err))) return rc;
        prof_mark(1, r, true, st);
        if (j_end <= 64 * CK) {
            // value table only, at load factor at most 0.3 (short probe chains)
            const int32_t tcap = compact_tcap(2 * j_end);
            int tshift = 32;
            for (int32_t x = tcap; x > 1; x >>= 1) --tshift;
            prof_mark(2, r, false, st);
            const size_t tab = (size_t)CWAVES * tcap * sizeof(int32_t);
            if (j_end <= 64 * 9)
                k_compact_reg<9><<<grid, 64 * CWAVES, tab, st>>>(p, gv.V, out, ws, cur, j_end,
                                                                 r == rounds - 1, r + 1 == rounds - 1,
                                                                 tcap, tshift, r == 0);
            else
                k_compact_reg<CK><<<grid, 64 * CWAVES, tab, st>>>(p, gv.V, out, ws, cur, j_end,
                                                                  r == rounds - 1, r + 1 == rounds - 1,
                                                                  tcap, tshift, r == 0);
            if ((rc = check_launch(err))) return rc;
            prof_mark(2, r, true, st);
            continue;
        }
        const int32_t tcap = compact_tcap(j_end);
        int tshift = 32;
        for (int32_t x = tcap; x > 1; x >>= 1) --tshift;
        const size_t lds = compact_lds(j_end);
        static bool attr = false;
        if (lds > 65536 && !attr) {
            const hipError_t e = hipFuncSetAttribute((const void*)k_compact,
                                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                                     (int)compact_lds(SMORE_MAX_NEG_TRIES));
            if (e != hipSuccess) { *err = hipGetErrorString(e); return SMORE_E_HIP; }
            attr = true;
        }
        prof_mark(2, r, false, st);
        k_compact<<<grid * 4, 64, lds, st>>>(p, gv.V, out, ws, cur, j_end, r == rounds - 1,
                                             r + 1 == rounds - 1, tcap, tshift, r == 0);
        if ((rc = check_launch(err))) return rc;
        prof_mark(2, r, true, st);
    }
    return SMORE_OK;
}

template <class T>
int dispatch_negatives(QType qt, const GraphView& gv, const SampleParams& p, const smore_sample_out& out,
                       Ws ws, int64_t* stats, int32_t R, int parts, hipStream_t st, const char** err)
{
    switch (qt) {
        case Q1P: return run_negatives<Q1P, T>(gv, p, out, ws, stats, R, parts, st, err);
        case Q2P: return run_negatives<Q2P, T>(gv, p, out, ws, stats, R, parts, st, err);
        case Q3P: return run_negatives<Q3P, T>(gv, p, out, ws, stats, R, parts, st, err);
        case Q2I: return run_negatives<Q2I, T>(gv, p, out, ws, stats, R, parts, st, err);
        case Q3I: return run_negatives<Q3I, T>(gv, p, out, ws, stats, R, parts, st, err);
        case QIP: return run_negatives<QIP, T>(gv, p, out, ws, stats, R, parts, st, err);
        case QPI: return run_negatives<QPI, T>(gv, p, out, ws, stats, R, parts, st, err);
        case Q2U: return run_negatives<Q2U, T>(gv, p, out, ws, stats, R, parts, st, err);
        case QUP: return run_negatives<QUP, T>(gv, p, out, ws, stats, R, parts, st, err);
        case Q2IN: return run_negatives<Q2IN, T>(gv, p, out, ws, stats, R, parts, st, err);
        case Q3IN: return run_negatives<Q3IN, T>(gv, p, out, ws, stats, R, parts, st, err);
        case QINP: return run_negatives<QINP, T>(gv, p, out, ws, stats, R, parts, st, err);
        case QPIN: return run_negatives<QPIN, T>(gv, p, out, ws, stats, R, parts, st, err);
        case QPNI: return run_negatives<QPNI, T>(gv, p, out, ws, stats, R, parts, st, err);
        default: *err = "unknown shape"; return SMORE_E_UNSUPPORTED;
    }
}

// ------------------------------------------------- shared candidate sets
// The minibatch's candidate set: the first n_neg distinct values of the
// draws j < neg_tries of the shared stream, in draw order.  One workgroup
// takes the draws 256 at a time; an LDS table of (value, first draw)
// decides first occurrences (later blocks find the values of earlier ones).
constexpr int SSET_WG = 256;

__global__ __launch_bounds__(SSET_WG) void k_shared_set(SampleParams p, int32_t V, int32_t* shared,
                                                        int32_t* n_shared, int32_t tcap, int tshift)
{
    extern __shared__ int32_t lds[];   // tv[tcap], tj[tcap], wave_cnt[4]: all dynamic
    int32_t* tv = lds;
    int32_t* tj = lds + tcap;
    int32_t* wave_cnt = lds + 2 * tcap;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const uint32_t tmask = (uint32_t)tcap - 1;
    for (int32_t k = tid; k < tcap; k += SSET_WG) { tv[k] = -1; tj[k] = INT_MAX; }
    __syncthreads();
    int32_t acc = 0;   // the same in every thread: block-wide counts only
    for (int32_t base = 0; base < p.neg_tries && acc < p.n_neg; base += SSET_WG) {
        const int32_t j = base + tid;
        int32_t c = -1;
        if (j < p.neg_tries) {
            c = (int32_t)reduce_range(draw64(p.seed, TAG_SHARED, (uint32_t)p.query_offset, 0, (uint32_t)j),
                                      (uint32_t)V);
            ht_insert(tv, tj, tmask, tshift, c, j);
        }
        __syncthreads();
        const bool first = c >= 0 && ht_first(tv, tj, tmask, tshift, c) == j;
        const uint64_t m = __ballot(first);
        if (lane == 0) wave_cnt[w] = __popcll(m);
        __syncthreads();
        int32_t before = 0, total = 0;
        for (int k = 0; k < SSET_WG / 64; ++k) {
            before += k < w ? wave_cnt[k] : 0;
            total += wave_cnt[k];
        }
        const int32_t rank = acc + before + __popcll(m & lanes_below(lane));
        if (first && rank < p.n_neg) shared[rank] = c;
        acc = min(p.n_neg, acc + total);
        __syncthreads();   // wave_cnt is rewritten by the next block of draws
    }
    for (int32_t k = acc + tid; k < p.n_neg; k += SSET_WG) shared[k] = -1;
    if (tid == 0) *n_shared = acc;
}

// Mask rows from the pair states: bit k of row b set iff state (b, k) is a
// non-answer; n_valid = set bits.  One wavefront per query.
__global__ __launch_bounds__(256) void k_pack(SampleParams p, Ws ws, uint32_t* mask, int32_t* n_valid)
{
    const int lane = threadIdx.x & 63;
    const int32_t words = (p.n_neg + 31) >> 5;
    const int32_t ns = p.n_shared ? uni(*p.n_shared) : p.n_neg;
    const int32_t nwaves = gridDim.x * 4;
    for (int32_t b = uni(blockIdx.x * 4 + (threadIdx.x >> 6)); b < p.batch; b += nwaves) {
        uint32_t* row = mask + (int64_t)b * words;
        const bool valid = uni(ws.qf[(int64_t)b * QF + 6]) >= 0;
        const uint8_t* sv = ws.status + (int64_t)b * p.neg_tries;
        int32_t cnt = 0;
        for (int32_t wd = lane; wd < words; wd += 64) {
            uint32_t bits = 0;
            if (valid)
                for (int k = 0; k < 32; ++k) {
                    const int32_t j = wd * 32 + k;
                    if (j < ns && sv[j] == ST_NON) bits |= 1u << k;
                }
            row[wd] = bits;
            cnt += __popc(bits);
        }
        for (int s = 32; s > 0; s >>= 1) cnt += __shfl_xor(cnt, s);
        if (valid && lane == 0) n_valid[b] = cnt;
    }
}

// The minibatch's shared candidate set (one workgroup).
int draw_shared_set(const SampleParams& p, int32_t V, int32_t* shared, int32_t* n_shared,
                    hipStream_t st, const char** err)
{
    const int32_t tcap = compact_tcap(p.neg_tries > 0 ? p.neg_tries : 1);
    int tshift = 32;
    for (int32_t x = tcap; x > 1; x >>= 1) --tshift;
    // the table needs up to 64 KiB plus the counts: raise the kernel's LDS
    // limit to the largest request once (the default is 64 KiB in total)
    const size_t lds = ((size_t)2 * tcap + SSET_WG / 64) * sizeof(int32_t);
    static bool attr = false;
    if (!attr) {
        const size_t most = ((size_t)2 * compact_tcap(SMORE_MAX_NEG_TRIES) + SSET_WG / 64) * sizeof(int32_t);
        const hipError_t e = hipFuncSetAttribute((const void*)k_shared_set,
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)most);
        if (e != hipSuccess) { *err = hipGetErrorString(e); return SMORE_E_HIP; }
        attr = true;
    }
    k_shared_set<<<1, SSET_WG, lds, st>>>(p, V, shared, n_shared, tcap, tshift);
    return check_launch(err);
}

// Every (query, candidate) pair of p.shared (one set for all queries, or a
// list per query p.cand_stride apart): states, then mask rows and counts.
template <int QT>
int run_pairs(const GraphView& gv, const SampleParams& p, const smore_sample_out& q, Ws ws,
              uint32_t* mask, int32_t R, hipStream_t st, const char** err)
{
    int rc;
    if (p.n_neg == 0) {   // no candidates: n_valid only (0, or -1 for a skipped query)
        k_no_draws<QT><<<(p.batch + 255) / 256, 256, 0, st>>>(gv, p, q, nullptr, R);
        return check_launch(err);
    }
    k_prepare<QT, NoTally><<<(p.batch + 63) / 64, 256, 0, st>>>(gv, p, q, ws, nullptr, R);
    if ((rc = check_launch(err))) return rc;
    k_candidates<QT, NoTally, true><<<max(p.batch, 1), CWG, 0, st>>>(gv, p, q, ws, nullptr, 0, 0,
                                                                     p.n_neg);
    if ((rc = check_launch(err))) return rc;
    if constexpr (QT == Q3P) {
        k_heavy3<NoTally><<<PERSIST_BLOCKS, HEAVY_WG, 0, st>>>(gv, p, q, ws, nullptr, 1);
        if ((rc = check_launch(err))) return rc;
        k_units3<NoTally><<<PERSIST_BLOCKS, HEAVY_WG, 0, st>>>(gv, p, q, ws, nullptr);
    } else {
        k_heavy<QT, NoTally><<<PERSIST_BLOCKS, HEAVY_WG, 0, st>>>(gv, p, q, ws, nullptr, 1);
    }
    if ((rc = check_launch(err))) return rc;
    k_pack<<<(p.batch + 3) / 4 < PERSIST_BLOCKS ? (p.batch + 3) / 4 : PERSIST_BLOCKS, 256, 0, st>>>(
        p, ws, mask, q.n_valid);
    return check_launch(err);
}

int dispatch_pairs(QType qt, const GraphView& gv, const SampleParams& p, const smore_sample_out& q,
                   Ws ws, uint32_t* mask, int32_t R, hipStream_t st, const char** err)
{
    switch (qt) {
        case Q1P: return run_pairs<Q1P>(gv, p, q, ws, mask, R, st, err);
        case Q2P: return run_pairs<Q2P>(gv, p, q, ws, mask, R, st, err);
        case Q3P: return run_pairs<Q3P>(gv, p, q, ws, mask, R, st, err);
        case Q2I: return run_pairs<Q2I>(gv, p, q, ws, mask, R, st, err);
        case Q3I: return run_pairs<Q3I>(gv, p, q, ws, mask, R, st, err);
        case QIP: return run_pairs<QIP>(gv, p, q, ws, mask, R, st, err);
        case QPI: return run_pairs<QPI>(gv, p, q, ws, mask, R, st, err);
        case Q2U: return run_pairs<Q2U>(gv, p, q, ws, mask, R, st, err);
        case QUP: return run_pairs<QUP>(gv, p, q, ws, mask, R, st, err);
        case Q2IN: return run_pairs<Q2IN>(gv, p, q, ws, mask, R, st, err);
        case Q3IN: return run_pairs<Q3IN>(gv, p, q, ws, mask, R, st, err);
        case QINP: return run_pairs<QINP>(gv, p, q, ws, mask, R, st, err);
        case QPIN: return run_pairs<QPIN>(gv, p, q, ws, mask, R, st, err);
        case QPNI: return run_pairs<QPNI>(gv, p, q, ws, mask, R, st, err);
        default: *err = "unknown shape"; return SMORE_E_UNSUPPORTED;
    }
}

GraphView view_of(const smore_graph* g)
{
    GraphView gv;
    gv.fwd = DirView{g->f_node, g->f_grp, g->f_nbr};
    gv.rev = DirView{g->r_node, g->r_grp, g->r_nbr};
    gv.active_in = g->active_in;
    gv.has_in = g->has_in;
    gv.has_in4 = g->has_in4;
    gv.sig = g->sig;
    // above 2 MiB of fine mask (V > 2^24) the coarse mask (a quarter of
    // the size) answers most draws from the L2
    gv.coarse = g->V > (1 << 24);
    gv.V = g->V;
    gv.n_active = (int32_t)g->n_active;
    return gv;
}

}  // namespace

// Workspace of smore_sample_noalloc: a fixed array in device memory, one
// copy per GPU the library runs on, held until the process ends.  Host code
// never uses the array's name as an address: each device's address comes
// from hipGetSymbolAddress, taken once per device with that device current.
namespace {
static __device__ __align__(256) char scratch[SMORE_NOALLOC_SCRATCH_BYTES];
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES];
}  // namespace

int scratch_workspace(void** ptr, size_t* bytes, const char** err)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) {
        *err = "no usable current device for the fixed scratch";
        return SMORE_E_HIP;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            *err = e != hipSuccess ? hipGetErrorString(e) : "scratch has no device address";
            return SMORE_E_HIP;
        }
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    *bytes = SMORE_NOALLOC_SCRATCH_BYTES;
    return SMORE_OK;
}

void arm_wait(void* event) { g_wait = (hipEvent_t)event; }

void disarm()
{
    for (ProfileArm& a : g_prof) a = ProfileArm{};
    g_wait = nullptr;
}

void arm_profile(void* start_event, void* stop_event, int which)
{
    ProfileArm& a = g_prof[which];
    a.start = (start_event && stop_event) ? (hipEvent_t)start_event : nullptr;
    a.stop = (start_event && stop_event) ? (hipEvent_t)stop_event : nullptr;
}

size_t negatives_workspace_bytes(const SampleParams& p)
{
    return ws_layout(p, nullptr, nullptr);
}

int launch_positive(const smore_graph* g, const WalkProgram& wp, const SampleParams& p,
                    const smore_sample_out& out, hipStream_t st, const char** err)
{
    // attempt lanes per query (they divide 64): attempts past the first
    // successful one are wasted reads, so plans that usually succeed at once
    // run two.  Plans accept less often per attempt when sibling branches
    // hang off the root (two of them must not draw the same in-relation and
    // in-neighbour of the root, which seldom has many) or with a
    // complemented operand: four lanes, eight with three root siblings; and
    // a maximum expansion C rejects every attempt through a wider step:
    // eight lanes.
    const int pa = (wp.root_pairs >= 3 || p.max_fanout > 0) ? 8
                   : (wp.root_pairs > 0 || wp.neg_steps > 0) ? 4 : 2;
    const int64_t threads = (int64_t)p.batch * pa;
    const unsigned blocks = (unsigned)((threads + 255) / 256);
    if (pa == 8) k_positive<8><<<blocks, 256, 0, st>>>(view_of(g), wp, p, out);
    else if (pa == 4) k_positive<4><<<blocks, 256, 0, st>>>(view_of(g), wp, p, out);
    else k_positive<2><<<blocks, 256, 0, st>>>(view_of(g), wp, p, out);
    return check_launch(err);
}

int launch_negative(const smore_graph* g, QType qt, const SampleParams& p,
                    const smore_sample_out& out, int64_t* stats, void* workspace, size_t ws_bytes,
                    int parts, hipStream_t st, const char** err)
{
    Ws ws;
    const size_t need = ws_layout(p, &ws, (char*)workspace);
    if (p.n_neg > 0 && (!workspace || ws_bytes < need)) {
        *err = "workspace too small (see smore_sample_workspace_bytes)";
        return SMORE_E_INVALID_ARG;
    }
    const GraphView gv = view_of(g);
    return stats ? dispatch_negatives<Tally>(qt, gv, p, out, ws, stats, g->R, parts, st, err)
                 : dispatch_negatives<NoTally>(qt, gv, p, out, ws, nullptr, g->R, parts, st, err);
}

int launch_shared(const smore_graph* g, QType qt, const SampleParams& p0, const smore_sample_out& pos,
                  int32_t* shared, int32_t* n_shared, uint32_t* mask, void* workspace,
                  size_t ws_bytes, hipStream_t st, const char** err)
{
    SampleParams p = p0;
    p.shared_mode = 1;
    p.shared = shared;
    p.n_shared = n_shared;
    p.cand_stride = 0;
    Ws ws;
    const size_t need = ws_layout(p, &ws, (char*)workspace);
    if (p.n_neg > 0 && (!workspace || ws_bytes < need)) {
        *err = "workspace too small (see smore_sample_workspace_bytes)";
        return SMORE_E_INVALID_ARG;
    }
    const GraphView gv = view_of(g);
    const int rc = draw_shared_set(p, gv.V, shared, n_shared, st, err);
    // an empty set leaves nothing to verify: the positives' n_valid (0, or -1
    // without a positive) is the row count, and no mask word exists
    if (rc || p.n_neg == 0) return rc;
    return dispatch_pairs(qt, gv, p, pos, ws, mask, g->R, st, err);
}

int launch_verify(const smore_graph* g, QType qt, const SampleParams& p0, const int32_t* anchors,
                  const int32_t* relations, const int32_t* candidates, uint32_t* mask,
                  int32_t* n_valid, void* workspace, size_t ws_bytes, hipStream_t st,
                  const char** err)
{
    SampleParams p = p0;
    p.shared_mode = 2;
    p.shared = candidates;
    p.n_shared = nullptr;
    p.cand_stride = p.n_neg;
    Ws ws;
    const size_t need = ws_layout(p, &ws, (char*)workspace);
    if (p.n_neg > 0 && (!workspace || ws_bytes < need)) {
        *err = "workspace too small (see smore_sample_workspace_bytes)";
        return SMORE_E_INVALID_ARG;
    }
    smore_sample_out q;
    std::memset(&q, 0, sizeof(q));
    q.anchors = (int32_t*)anchors;
    q.relations = (int32_t*)relations;
    q.n_valid = n_valid;
    return dispatch_pairs(qt, view_of(g), p, q, ws, mask, g->R, st, err);
}

}  // namespace smore
