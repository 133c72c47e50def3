// sample.hip -- query sampling with verified negatives on gfx950.
//
// Two kernels per call, on the caller's stream:
//
//  k_positive: one thread per query.  Reverse directional sampling
//    (Sec. 3.1; appendix on reverse directional sampling): attempt t grounds
//    the root among entities with an in-edge, then runs the pre-order walk
//    program compiled from the plan, each projection picking an in-relation
//    of the current entity and an in-neighbour under it.  The first attempt
//    that reaches every anchor, keeps single-projection siblings apart and
//    respects max_fanout wins.
//
//  k_verify<shape>: one workgroup per query.  Bidirectional rejection
//    sampling (Sec. 3.2) at the node cut the planner picks for the shape:
//    forward caching turns the anchors into their neighbour lists A_r(a)
//    (sorted CSR groups, staged in LDS when small, used in place when not);
//    candidates are drawn in rounds, one per lane, deduplicated against all
//    earlier draws with an LDS hash table keyed by value holding the
//    smallest draw index, and verified backward from the candidate.  A lane
//    decides candidates whose backward lists are short; longer lists are
//    queued and intersected by a whole wavefront (coalesced reads, ballot).
//    Accepted candidates are compacted in draw order with wave ballots and
//    per-row prefix sums, so the output does not depend on scheduling.
#include <hip/hip_runtime.h>

#include <climits>

#include "philox.h"
#include "smore_internal.h"

namespace smore {
namespace {

constexpr int WG = 256;       // threads per verify workgroup
constexpr int NW = WG / 64;   // wavefronts per workgroup
constexpr int CHMAX = 512;    // candidates per round
constexpr int STAGE = 2048;   // LDS entries for staged forward lists
constexpr int LANE_SEG = 8;   // backward lists up to this length stay on one lane

enum : int32_t { ST_NON = 0, ST_ANS = 1, ST_DUP = 2, ST_PEND = 3 };

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

// Edges [x, y) of entity v under relation r in one direction ((0, 0) if
// none).  Reads the node-pointer pair, the relations probed by the binary
// search, and the group bounds.
template <class T>
__device__ __forceinline__ int2 group_range(const DirView& d, int32_t v, int32_t r, T& tl)
{
    int32_t lo = d.node[v];
    const int32_t end = d.node[v + 1];
    tl.read(d.node + v, 8);
    int32_t hi = end;
    while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        tl.read(&d.grp[mid].x, 4);
        if (d.grp[mid].x < r) lo = mid + 1; else hi = mid;
    }
    if (lo < end) {
        const int2 gr = d.grp[lo];
        if (gr.x == r) {
            tl.read(&d.grp[lo].y, 4);
            tl.read(&d.grp[lo + 1].y, 4);
            return make_int2(gr.y, d.grp[lo + 1].y);
        }
    }
    return make_int2(0, 0);
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

template <class T>
__device__ __forceinline__ bool has(const FSet& s, int32_t x, T& tl)
{
    return has(s.p, s.n, x, !s.lds, tl);
}

__device__ __forceinline__ uint64_t lanes_below(int lane)
{
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Do the sorted lists A and B share an element?  Whole wavefront; the
// shorter list is read 64 entries at a time and each entry is searched in
// the longer one.  a_glob / b_glob: whether the list is graph memory.
template <class T>
__device__ bool wave_meet(const int32_t* A, int32_t na, bool a_glob, const int32_t* B, int32_t nb,
                          bool b_glob, int lane, T& tl)
{
    if (na > nb) {
        const int32_t* t = A; A = B; B = t;
        const int32_t n = na; na = nb; nb = n;
        const bool g = a_glob; a_glob = b_glob; b_glob = g;
    }
    for (int32_t k = 0; k < na; k += 64) {
        if (a_glob && lane == 0) tl.read(A + k, 4 * min(64, na - k));
        const bool hit = k + lane < na && has(B, nb, A[k + lane], b_glob, tl);
        if (__ballot(hit)) return true;
    }
    return false;
}

// Does the sorted graph list S share one element with both A and B?
template <class T>
__device__ bool wave_meet3(const int32_t* S, int32_t ns, FSet A, FSet B, int lane, T& tl)
{
    // read the shortest of the three lists, search the other two
    if (A.n < ns && A.n <= B.n) {
        for (int32_t k = 0; k < A.n; k += 64) {
            if (!A.lds && lane == 0) tl.read(A.p + k, 4 * min(64, A.n - k));
            const bool hit = k + lane < A.n && has(B, A.p[k + lane], tl) &&
                             has(S, ns, A.p[k + lane], true, tl);
            if (__ballot(hit)) return true;
        }
        return false;
    }
    if (B.n < ns) {
        for (int32_t k = 0; k < B.n; k += 64) {
            if (!B.lds && lane == 0) tl.read(B.p + k, 4 * min(64, B.n - k));
            const bool hit = k + lane < B.n && has(A, B.p[k + lane], tl) &&
                             has(S, ns, B.p[k + lane], true, tl);
            if (__ballot(hit)) return true;
        }
        return false;
    }
    for (int32_t k = 0; k < ns; k += 64) {
        if (lane == 0) tl.read(S + k, 4 * min(64, ns - k));
        const bool hit = k + lane < ns && has(A, S[k + lane], tl) && has(B, S[k + lane], tl);
        if (__ballot(hit)) return true;
    }
    return false;
}

// ------------------------------------------------------------- positive
__device__ __forceinline__ int32_t sel4(int i, int32_t a, int32_t b, int32_t c, int32_t d)
{
    return i == 0 ? a : i == 1 ? b : i == 2 ? c : d;
}

__global__ __launch_bounds__(256) void k_positive(GraphView g, WalkProgram wp, SampleParams p,
                                                  smore_sample_out out)
{
    const int32_t b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= p.batch) return;
    const uint32_t q = (uint32_t)(p.query_offset + (uint64_t)b);
    int32_t e0 = -1, e1 = -1, e2 = -1, e3 = -1;   // registers: root, then one per step
    int32_t q0 = -1, q1 = -1, q2 = -1;            // relation grounded by step k
    int t = 0;
    bool found = false;
    for (; t < p.pos_tries && !found; ++t) {
        if (g.n_active == 0) continue;
        e0 = g.active_in[reduce_range(draw64(p.seed, TAG_POS, q, t, 0), (uint32_t)g.n_active)];
        bool ok = true;
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            if (!ok || k >= wp.n_steps) break;
            const int32_t e = sel4(wp.src[k], e0, e1, e2, e3);
            const uint64_t u0 = draw64(p.seed, TAG_POS, q, t, 1 + 2 * k);
            const uint64_t u1 = draw64(p.seed, TAG_POS, q, t, 2 + 2 * k);
            const int32_t s0 = g.rev.node[e], s1 = g.rev.node[e + 1];
            if (s0 == s1) { ok = false; break; }          // no in-edge: dead end
            const int32_t s = s0 + (int32_t)reduce_range(u0, (uint32_t)(s1 - s0));
            const int2 gr = g.rev.grp[s];
            const int32_t len = g.rev.grp[s + 1].y - gr.y;
            const int32_t x = g.rev.nbr[gr.y + (int32_t)reduce_range(u1, (uint32_t)len)];
            if (p.max_fanout > 0) {
                const int2 fr = group_range(g.fwd, x, gr.x);
                if (fr.y - fr.x > p.max_fanout) { ok = false; break; }
            }
            if (k == 0) { e1 = x; q0 = gr.x; }
            if (k == 1) { e2 = x; q1 = gr.x; }
            if (k == 2) { e3 = x; q2 = gr.x; }
        }
        if (ok) {
            for (int pr = 0; pr < wp.n_pairs; ++pr) {
                const int32_t xa = sel4(wp.anchor_reg[wp.pair_anchor[pr][0]], e0, e1, e2, e3);
                const int32_t xb = sel4(wp.anchor_reg[wp.pair_anchor[pr][1]], e0, e1, e2, e3);
                int32_t ra = -1, rb = -1;
                for (int k = 0; k < wp.n_steps; ++k) {
                    const int32_t rk = sel4(k, q0, q1, q2, -1);
                    if (wp.rel_slot[k] == wp.pair_rel[pr][0]) ra = rk;
                    if (wp.rel_slot[k] == wp.pair_rel[pr][1]) rb = rk;
                }
                if (xa == xb && ra == rb) ok = false;      // degenerate sibling branches
            }
        }
        found = ok;
    }
    int32_t* A = out.anchors + 3 * (int64_t)b;
    int32_t* R = out.relations + 3 * (int64_t)b;
    if (!found) {
        for (int k = 0; k < 3; ++k) { A[k] = -1; R[k] = -1; }
        out.positive[b] = -1;
        out.n_valid[b] = -1;
        out.pos_attempts[b] = p.pos_tries;
        return;
    }
    for (int a = 0; a < 3; ++a) A[a] = a < wp.n_anchor ? sel4(wp.anchor_reg[a], e0, e1, e2, e3) : -1;
    for (int s = 0; s < 3; ++s) {
        int32_t v = -1;
        for (int k = 0; k < wp.n_steps; ++k)
            if (wp.rel_slot[k] == s) v = sel4(k, q0, q1, q2, -1);
        R[s] = v;
    }
    out.positive[b] = e0;
    out.n_valid[b] = 0;
    out.pos_attempts[b] = t;      // t was advanced past the accepted attempt
}

// --------------------------------------------------------------- verify
// Forward-cached lists per shape (anchor slot, relation slot) at the cut the
// planner picks:  1p {a0}, 2p/3p {V1}, 2i/3i/2u {anchors}, ip/up {Y0, Y1},
// pi {V1, a1}.  A cut at an anchor is tested from the anchor side (c in
// A_r(a)), which decides the same edge.  n_anc / n_rel: slots the shape uses.
template <int QT> struct Shape;
template <> struct Shape<Q1P> { static constexpr int nf = 1, n_anc = 1, n_rel = 1; static constexpr int fa[3] = {0, 0, 0}, fr[3] = {0, 0, 0}; };
template <> struct Shape<Q2P> { static constexpr int nf = 1, n_anc = 1, n_rel = 2; static constexpr int fa[3] = {0, 0, 0}, fr[3] = {0, 0, 0}; };
template <> struct Shape<Q3P> { static constexpr int nf = 1, n_anc = 1, n_rel = 3; static constexpr int fa[3] = {0, 0, 0}, fr[3] = {0, 0, 0}; };
template <> struct Shape<Q2I> { static constexpr int nf = 2, n_anc = 2, n_rel = 2; static constexpr int fa[3] = {0, 1, 0}, fr[3] = {0, 1, 0}; };
template <> struct Shape<Q3I> { static constexpr int nf = 3, n_anc = 3, n_rel = 3; static constexpr int fa[3] = {0, 1, 2}, fr[3] = {0, 1, 2}; };
template <> struct Shape<QIP> { static constexpr int nf = 2, n_anc = 2, n_rel = 3; static constexpr int fa[3] = {0, 1, 0}, fr[3] = {0, 1, 0}; };
template <> struct Shape<QPI> { static constexpr int nf = 2, n_anc = 2, n_rel = 3; static constexpr int fa[3] = {0, 1, 0}, fr[3] = {0, 2, 0}; };
template <> struct Shape<Q2U> { static constexpr int nf = 2, n_anc = 2, n_rel = 2; static constexpr int fa[3] = {0, 1, 0}, fr[3] = {0, 1, 0}; };
template <> struct Shape<QUP> { static constexpr int nf = 2, n_anc = 2, n_rel = 3; static constexpr int fa[3] = {0, 1, 0}, fr[3] = {0, 1, 0}; };

// Lane-level test of candidate c.  Returns ST_NON / ST_ANS, or ST_PEND with
// *seg = the backward list a wavefront must intersect.
template <int QT, class T>
__device__ __forceinline__ int32_t lane_test(const GraphView& g, const FSet* F, const int32_t* rel,
                                             int32_t c, int2* seg, T& tl)
{
    if (QT == Q1P) return has(F[0], c, tl) ? ST_ANS : ST_NON;
    if (QT == Q2I) return (has(F[0], c, tl) && has(F[1], c, tl)) ? ST_ANS : ST_NON;
    if (QT == Q3I) return (has(F[0], c, tl) && has(F[1], c, tl) && has(F[2], c, tl)) ? ST_ANS : ST_NON;
    if (QT == Q2U) return (has(F[0], c, tl) || has(F[1], c, tl)) ? ST_ANS : ST_NON;
    if (QT == QPI && !has(F[1], c, tl)) return ST_NON;   // the one-hop branch fails
    // backward step from c under the relation entering the root
    const int32_t rb = (QT == Q2P || QT == QPI) ? rel[1] : rel[2];
    const int2 s = group_range(g.rev, c, rb, tl);
    if (s.y == s.x) return ST_NON;
    if (s.y - s.x > LANE_SEG) { *seg = s; return ST_PEND; }
    tl.read(g.rev.nbr + s.x, 4 * (s.y - s.x));
    for (int32_t k = s.x; k < s.y; ++k) {
        const int32_t y = g.rev.nbr[k];
        if (QT == Q2P || QT == QPI) { if (has(F[0], y, tl)) return ST_ANS; }
        else if (QT == QIP) { if (has(F[0], y, tl) && has(F[1], y, tl)) return ST_ANS; }
        else if (QT == QUP) { if (has(F[0], y, tl) || has(F[1], y, tl)) return ST_ANS; }
        else {  // 3p: second backward step from y under r1
            const int2 s2 = group_range(g.rev, y, rel[1], tl);
            if (s2.y - s2.x > LANE_SEG) { *seg = s; return ST_PEND; }
            tl.read(g.rev.nbr + s2.x, 4 * (s2.y - s2.x));
            for (int32_t m = s2.x; m < s2.y; ++m)
                if (has(F[0], g.rev.nbr[m], tl)) return ST_ANS;
        }
    }
    return ST_NON;
}

// Wavefront-level test of a queued candidate whose backward list is s.
template <int QT, class T>
__device__ bool wave_test(const GraphView& g, const FSet* F, const int32_t* rel, int2 s, int lane,
                          T& tl)
{
    const int32_t* S = g.rev.nbr + s.x;
    const int32_t ns = s.y - s.x;
    if (QT == Q2P || QT == QPI) return wave_meet(S, ns, true, F[0].p, F[0].n, !F[0].lds, lane, tl);
    if (QT == QIP) return wave_meet3(S, ns, F[0], F[1], lane, tl);
    if (QT == QUP)
        return wave_meet(S, ns, true, F[0].p, F[0].n, !F[0].lds, lane, tl) ||
               wave_meet(S, ns, true, F[1].p, F[1].n, !F[1].lds, lane, tl);
    if (QT == Q3P) {
        for (int32_t k = 0; k < ns; k += 64) {
            if (lane == 0) tl.read(S + k, 4 * min(64, ns - k));
            int2 s2 = make_int2(0, 0);
            if (k + lane < ns) s2 = group_range(g.rev, S[k + lane], rel[1], tl);
            uint64_t todo = __ballot(s2.y > s2.x);
            while (todo) {
                const int src = __ffsll((unsigned long long)todo) - 1;
                todo &= todo - 1;
                const int32_t x = __shfl(s2.x, src), y = __shfl(s2.y, src);
                if (wave_meet(g.rev.nbr + x, y - x, true, F[0].p, F[0].n, !F[0].lds, lane, tl))
                    return true;
            }
        }
        return false;
    }
    return false;
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

template <int QT, class T>
__global__ __launch_bounds__(WG) void k_verify(GraphView g, SampleParams p, smore_sample_out out,
                                               int64_t* stats, int32_t tcap, int tshift,
                                               int32_t R)
{
    extern __shared__ int32_t lds[];
    int32_t* tv = lds;                  // hash table: candidate value
    int32_t* tj = tv + tcap;            // hash table: smallest draw index of that value
    int32_t* stage = tj + tcap;         // staged forward lists
    int32_t* cval = stage + STAGE;      // candidates of the round
    int32_t* cst = cval + CHMAX;        // their status
    int32_t* qi = cst + CHMAX;          // queue: candidate index
    int2* qs = (int2*)(qi + CHMAX);     // queue: backward list
    __shared__ int32_t s_f[3][2];
    __shared__ int32_t s_qlen;
    __shared__ int32_t s_cnt[NW];
    __shared__ unsigned long long s_tally[2];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int32_t b = blockIdx.x;
    const uint32_t q = (uint32_t)(p.query_offset + (uint64_t)b);
    int32_t* negrow = out.negatives + (int64_t)b * p.n_neg;
    int32_t rel[3], anc[3];
    bool valid = out.positive[b] >= 0;
    for (int k = 0; k < 3; ++k) {
        rel[k] = out.relations[3 * (int64_t)b + k];
        anc[k] = out.anchors[3 * (int64_t)b + k];
        // ids the shape uses must index the graph (rows built by a caller)
        if (k < Shape<QT>::n_rel && (rel[k] < 0 || rel[k] >= R)) valid = false;
        if (k < Shape<QT>::n_anc && (anc[k] < 0 || anc[k] >= g.V)) valid = false;
    }
    if (!valid) {                                      // no query to verify
        for (int32_t k = tid; k < p.n_neg; k += WG) negrow[k] = -1;
        if (tid == 0) {
            out.n_valid[b] = -1;
            out.neg_draws[b] = -1;
            if (stats) { stats[2 * (int64_t)b] = 0; stats[2 * (int64_t)b + 1] = 0; }
        }
        return;
    }
    if (p.n_neg == 0) {
        if (tid == 0) {
            out.n_valid[b] = 0;
            out.neg_draws[b] = 0;
            if (stats) { stats[2 * (int64_t)b] = 0; stats[2 * (int64_t)b + 1] = 0; }
        }
        return;
    }
    T tl;
    // forward caching: the anchors' neighbour lists at the cut
    constexpr int NF = Shape<QT>::nf;
    if (tid < NF) {
        const int2 r = group_range(g.fwd, anc[Shape<QT>::fa[tid]], rel[Shape<QT>::fr[tid]], tl);
        s_f[tid][0] = r.x;
        s_f[tid][1] = r.y;
    }
    if (tid < 2) s_tally[tid] = 0;
    for (int32_t k = tid; k < tcap; k += WG) { tv[k] = -1; tj[k] = INT_MAX; }
    __syncthreads();
    FSet F[3];
    int32_t used = 0;
#pragma unroll
    for (int f = 0; f < 3; ++f) {
        if (f >= NF) { F[f] = FSet{nullptr, 0, true}; continue; }
        const int32_t beg = s_f[f][0], n = s_f[f][1] - s_f[f][0];
        if (n <= STAGE - used) {
            for (int32_t k = tid; k < n; k += WG) stage[used + k] = g.fwd.nbr[beg + k];
            if (tid == 0) tl.read(g.fwd.nbr + beg, 4 * n);
            F[f] = FSet{stage + used, n, true};
            used += n;
        } else {
            F[f] = FSet{g.fwd.nbr + beg, n, false};
        }
    }
    __syncthreads();

    const uint32_t tmask = (uint32_t)tcap - 1;
    int32_t acc = 0;
    for (int32_t j0 = 0; acc < p.n_neg && j0 < p.neg_tries;) {
        const int32_t need = p.n_neg - acc;
        int32_t ch = ((need + need / 8 + 16 + 63) / 64) * 64;
        ch = min(ch, CHMAX);
        ch = min(ch, p.neg_tries - j0);
        // draw and register in the first-occurrence table
        for (int32_t i = tid; i < ch; i += WG) {
            const int32_t c = (int32_t)reduce_range(draw64(p.seed, TAG_NEG, q, 0, (uint32_t)(j0 + i)),
                                                    (uint32_t)g.V);
            cval[i] = c;
            ht_insert(tv, tj, tmask, tshift, c, j0 + i);
        }
        if (tid == 0) s_qlen = 0;
        __syncthreads();
        // lane-level verification of first occurrences
        for (int32_t i = tid; i < ch; i += WG) {
            const int32_t c = cval[i];
            int32_t st;
            if (ht_first(tv, tj, tmask, tshift, c) != j0 + i) {
                st = ST_DUP;
            } else {
                int2 s;
                st = lane_test<QT>(g, F, rel, c, &s, tl);
                if (st == ST_PEND) {
                    const int32_t slot = atomicAdd(&s_qlen, 1);
                    qi[slot] = i;
                    qs[slot] = s;
                }
            }
            cst[i] = st;
        }
        __syncthreads();
        // wavefront-level verification of long backward lists
        const int32_t nq = s_qlen;
        for (int32_t it = w; it < nq; it += NW) {
            const bool ans = wave_test<QT>(g, F, rel, qs[it], lane, tl);
            if (lane == 0) cst[qi[it]] = ans ? ST_ANS : ST_NON;
        }
        __syncthreads();
        // keep non-answers in draw order
        for (int32_t row = 0; row < ch; row += WG) {
            const int32_t i = row + tid;
            const bool keep = i < ch && cst[i] == ST_NON;
            const uint64_t m = __ballot(keep);
            if (lane == 0) s_cnt[w] = __popcll(m);
            __syncthreads();
            int32_t before = acc, total = 0;
            for (int ww = 0; ww < NW; ++ww) {
                if (ww < w) before += s_cnt[ww];
                total += s_cnt[ww];
            }
            const int32_t rank = before + __popcll(m & lanes_below(lane));
            if (keep && rank < p.n_neg) {
                negrow[rank] = cval[i];
                if (rank == p.n_neg - 1) out.neg_draws[b] = j0 + i + 1;
            }
            acc = min(p.n_neg, acc + total);
            __syncthreads();
        }
        j0 += ch;
    }
    for (int32_t k = acc + tid; k < p.n_neg; k += WG) negrow[k] = -1;
    if (tid == 0) {
        out.n_valid[b] = acc;
        if (acc < p.n_neg) out.neg_draws[b] = p.neg_tries;
    }
    if constexpr (T::on) {
        atomicAdd(&s_tally[0], (unsigned long long)tl.b);
        atomicAdd(&s_tally[1], (unsigned long long)tl.l);
        __syncthreads();
        if (tid == 0) {
            stats[2 * (int64_t)b] = (int64_t)s_tally[0];
            stats[2 * (int64_t)b + 1] = (int64_t)s_tally[1];
        }
    }
}

size_t verify_lds_bytes(int32_t tcap)
{
    return ((size_t)2 * tcap + STAGE + 5 * CHMAX) * sizeof(int32_t);
}

template <int QT, class T>
int launch_verify(const GraphView& gv, const SampleParams& p, const smore_sample_out& out,
                  int64_t* stats, int32_t R, hipStream_t st, const char** err)
{
    int32_t tcap = 64;
    while (tcap < 2 * p.neg_tries) tcap <<= 1;
    int tshift = 32;
    for (int32_t x = tcap; x > 1; x >>= 1) --tshift;
    // more than 64 KiB of LDS per workgroup must be requested explicitly
    static bool attr_set = false;
    if (verify_lds_bytes(tcap) > 65536 && !attr_set) {
        hipError_t e = hipFuncSetAttribute((const void*)k_verify<QT, T>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)verify_lds_bytes(2 * SMORE_MAX_NEG_TRIES));
        if (e != hipSuccess) { *err = hipGetErrorString(e); return SMORE_E_HIP; }
        attr_set = true;
    }
    k_verify<QT, T><<<p.batch, WG, verify_lds_bytes(tcap), st>>>(gv, p, out, stats, tcap, tshift, R);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) { *err = hipGetErrorString(e); return SMORE_E_HIP; }
    return SMORE_OK;
}

template <class T>
int dispatch_verify(QType qt, const GraphView& gv, const SampleParams& p, const smore_sample_out& out,
                    int64_t* stats, int32_t R, hipStream_t st, const char** err)
{
    switch (qt) {
        case Q1P: return launch_verify<Q1P, T>(gv, p, out, stats, R, st, err);
        case Q2P: return launch_verify<Q2P, T>(gv, p, out, stats, R, st, err);
        case Q3P: return launch_verify<Q3P, T>(gv, p, out, stats, R, st, err);
        case Q2I: return launch_verify<Q2I, T>(gv, p, out, stats, R, st, err);
        case Q3I: return launch_verify<Q3I, T>(gv, p, out, stats, R, st, err);
        case QIP: return launch_verify<QIP, T>(gv, p, out, stats, R, st, err);
        case QPI: return launch_verify<QPI, T>(gv, p, out, stats, R, st, err);
        case Q2U: return launch_verify<Q2U, T>(gv, p, out, stats, R, st, err);
        case QUP: return launch_verify<QUP, T>(gv, p, out, stats, R, st, err);
        default: *err = "unknown shape"; return SMORE_E_UNSUPPORTED;
    }
}

GraphView view_of(const smore_graph* g)
{
    GraphView gv;
    gv.fwd = DirView{g->f_node, g->f_grp, g->f_nbr};
    gv.rev = DirView{g->r_node, g->r_grp, g->r_nbr};
    gv.active_in = g->active_in;
    gv.V = g->V;
    gv.n_active = (int32_t)g->n_active;
    return gv;
}

}  // namespace

int launch_positive(const smore_graph* g, const WalkProgram& wp, const SampleParams& p,
                    const smore_sample_out& out, hipStream_t st, const char** err)
{
    k_positive<<<(p.batch + 255) / 256, 256, 0, st>>>(view_of(g), wp, p, out);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) { *err = hipGetErrorString(e); return SMORE_E_HIP; }
    return SMORE_OK;
}

int launch_negative(const smore_graph* g, QType qt, const SampleParams& p,
                    const smore_sample_out& out, int64_t* stats, hipStream_t st, const char** err)
{
    const GraphView gv = view_of(g);
    if (stats) return dispatch_verify<Tally>(qt, gv, p, out, stats, g->R, st, err);
    return dispatch_verify<NoTally>(qt, gv, p, out, nullptr, g->R, st, err);
}

}  // namespace smore
