// graph_build.hip -- builds the device adjacency of a knowledge graph on gfx950.
//
// The KG is a set of triples (Sec. 2) and the sampler needs, per entity and
// relation, the sorted neighbour list A_r(v) (appendix on the computation
// plan) in both directions.  Steps, all on the GPU:
//   1. upload and validate the triples, optionally adding (t, r + R, h);
//   2. stable LSD radix sort (8-bit digits) of the (h, r, t) records by t,
//      then r, then h; drop adjacent duplicates;
//   3. forward groups = runs of equal (h, r); node pointers by binary search
//      of each entity among the group heads;
//   4. a stable sort of the deduplicated records by r, then t, gives
//      (t, r, h) order (the input is already ordered by h within (t, r));
//      reverse groups and node pointers as in 3;
//   5. active_in = entities whose reverse node range is non-empty, the
//      in-edge mask (one bit per entity) and the coarse mask (one bit per
//      four entities) built from it.
// One-time and synchronous; the sampler never calls it.
#include <hip/hip_runtime.h>

#include <climits>
#include <vector>

#include "smore_internal.h"

namespace smore {
namespace {

constexpr int BT = 256;                  // threads per block
constexpr int RITEMS = 16;               // radix rows per tile
constexpr int RTILE = BT * RITEMS;       // radix tile
constexpr int SITEMS = 8;                // scan items per thread
constexpr int STILE = BT * SITEMS;       // scan tile

__global__ void k_load(const int32_t* __restrict__ tr, int64_t n, int32_t V, int32_t R, int inv,
                       int32_t* __restrict__ H, int32_t* __restrict__ Rl, int32_t* __restrict__ T,
                       int* __restrict__ bad)
{
    const int64_t i = (int64_t)blockIdx.x * BT + threadIdx.x;
    if (i >= n) return;
    const int32_t h = tr[3 * i], r = tr[3 * i + 1], t = tr[3 * i + 2];
    if (h < 0 || h >= V || t < 0 || t >= V || r < 0 || r >= R) atomicOr(bad, 1);
    H[i] = h;
    Rl[i] = r;
    T[i] = t;
    if (inv) {
        H[n + i] = t;
        Rl[n + i] = r + R;
        T[n + i] = h;
    }
}

// per-tile digit histogram, digit-major: hist[d * nblk + blk]
__global__ void k_radix_hist(const int32_t* __restrict__ key, int32_t n, int shift,
                             int32_t* __restrict__ hist, int32_t nblk)
{
    __shared__ int32_t h[256];
    h[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * RTILE;
    for (int row = 0; row < RITEMS; ++row) {
        const int64_t i = base + row * BT + threadIdx.x;
        if (i < n) atomicAdd(&h[((uint32_t)key[i] >> shift) & 255u], 1);
    }
    __syncthreads();
    hist[(int64_t)threadIdx.x * nblk + blockIdx.x] = h[threadIdx.x];
}

// Stable scatter of one radix pass.  Rows of 256 consecutive records are
// ranked in order: within a wave by ballot-matching lanes of equal digit,
// across waves and rows by running per-digit counts in LDS.
__global__ __launch_bounds__(BT) void k_radix_scatter(
    const int32_t* __restrict__ a, const int32_t* __restrict__ b, const int32_t* __restrict__ c,
    int32_t* __restrict__ a2, int32_t* __restrict__ b2, int32_t* __restrict__ c2, int32_t n,
    int field, int shift, const int32_t* __restrict__ off, int32_t nblk)
{
    __shared__ int32_t run[256];
    __shared__ int32_t wcnt[BT / 64][256];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    run[tid] = 0;
    int32_t va[RITEMS], vb[RITEMS], vc[RITEMS], pos[RITEMS];
    const int64_t base = (int64_t)blockIdx.x * RTILE;
    for (int row = 0; row < RITEMS; ++row) {
        const int64_t i = base + row * BT + tid;
        const bool valid = i < n;
        int d = 256;
        if (valid) {
            va[row] = a[i];
            vb[row] = b[i];
            vc[row] = c[i];
            const int32_t k = field == 0 ? va[row] : field == 1 ? vb[row] : vc[row];
            d = ((uint32_t)k >> shift) & 255u;
        }
#pragma unroll
        for (int ww = 0; ww < BT / 64; ++ww) wcnt[ww][tid] = 0;
        __syncthreads();
        uint64_t peers = ~0ull;
#pragma unroll
        for (int bit = 0; bit < 9; ++bit) {
            const int on = (d >> bit) & 1;
            const uint64_t m = __ballot(on);
            peers &= on ? m : ~m;
        }
        const int rank = __popcll(peers & lt);
        if (valid && rank == 0) wcnt[w][d] = __popcll(peers);
        __syncthreads();
        if (valid) {
            int32_t p = run[d];
            for (int ww = 0; ww < w; ++ww) p += wcnt[ww][d];
            pos[row] = p + rank;
        }
        __syncthreads();
        int32_t add = 0;
#pragma unroll
        for (int ww = 0; ww < BT / 64; ++ww) add += wcnt[ww][tid];
        run[tid] += add;
        __syncthreads();
    }
    for (int row = 0; row < RITEMS; ++row) {
        const int64_t i = base + row * BT + tid;
        if (i >= n) break;
        const int32_t k = field == 0 ? va[row] : field == 1 ? vb[row] : vc[row];
        const int d = ((uint32_t)k >> shift) & 255u;
        const int64_t g = (int64_t)off[(int64_t)d * nblk + blockIdx.x] + pos[row];
        a2[g] = va[row];
        b2[g] = vb[row];
        c2[g] = vc[row];
    }
}

// exclusive scan of one tile in place; sums[blk] = tile total
__global__ __launch_bounds__(BT) void k_scan_tile(int32_t* __restrict__ d, int64_t n,
                                                  int32_t* __restrict__ sums)
{
    __shared__ int32_t wsum[BT / 64];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t base = (int64_t)blockIdx.x * STILE + (int64_t)tid * SITEMS;
    int32_t v[SITEMS];
    int32_t t = 0;
#pragma unroll
    for (int k = 0; k < SITEMS; ++k) {
        const int32_t x = base + k < n ? d[base + k] : 0;
        v[k] = t;
        t += x;
    }
    int32_t incl = t;
#pragma unroll
    for (int s = 1; s < 64; s <<= 1) {
        const int32_t y = __shfl_up(incl, s);
        if (lane >= s) incl += y;
    }
    if (lane == 63) wsum[w] = incl;
    __syncthreads();
    int32_t woff = 0;
    for (int ww = 0; ww < w; ++ww) woff += wsum[ww];
    const int32_t excl = woff + incl - t;
#pragma unroll
    for (int k = 0; k < SITEMS; ++k)
        if (base + k < n) d[base + k] = v[k] + excl;
    if (tid == BT - 1) sums[blockIdx.x] = woff + incl;
}

__global__ void k_add_offsets(int32_t* __restrict__ d, int64_t n, const int32_t* __restrict__ sums)
{
    const int64_t base = (int64_t)blockIdx.x * STILE;
    const int32_t o = sums[blockIdx.x];
    for (int k = threadIdx.x; k < STILE; k += BT)
        if (base + k < n) d[base + k] += o;
}

__device__ __forceinline__ bool same3(const int32_t* H, const int32_t* R, const int32_t* T, int64_t i)
{
    return H[i] == H[i - 1] && R[i] == R[i - 1] && T[i] == T[i - 1];
}

__global__ void k_flag_unique(const int32_t* __restrict__ H, const int32_t* __restrict__ R,
                              const int32_t* __restrict__ T, int64_t n, int32_t* __restrict__ f)
{
    const int64_t i = (int64_t)blockIdx.x * BT + threadIdx.x;
    if (i < n) f[i] = (i == 0 || !same3(H, R, T, i)) ? 1 : 0;
}

__global__ void k_compact3(const int32_t* __restrict__ H, const int32_t* __restrict__ R,
                           const int32_t* __restrict__ T, int64_t n, const int32_t* __restrict__ pos,
                           int32_t* __restrict__ H2, int32_t* __restrict__ R2,
                           int32_t* __restrict__ T2)
{
    const int64_t i = (int64_t)blockIdx.x * BT + threadIdx.x;
    if (i >= n || (i > 0 && same3(H, R, T, i))) return;
    const int32_t p = pos[i];
    H2[p] = H[i];
    R2[p] = R[i];
    T2[p] = T[i];
}

__global__ void k_flag_groups(const int32_t* __restrict__ P, const int32_t* __restrict__ R, int64_t n,
                              int32_t* __restrict__ f)
{
    const int64_t i = (int64_t)blockIdx.x * BT + threadIdx.x;
    if (i < n) f[i] = (i == 0 || P[i] != P[i - 1] || R[i] != R[i - 1]) ? 1 : 0;
}

__global__ void k_write_groups(const int32_t* __restrict__ P, const int32_t* __restrict__ R, int64_t n,
                               const int32_t* __restrict__ pos, int2* __restrict__ grp,
                               int32_t* __restrict__ head)
{
    const int64_t i = (int64_t)blockIdx.x * BT + threadIdx.x;
    if (i >= n) return;
    if (i > 0 && P[i] == P[i - 1] && R[i] == R[i - 1]) return;
    const int32_t g = pos[i];
    grp[g] = make_int2(R[i], (int32_t)i);
    head[g] = P[i];
}

// node[v] = number of groups whose entity is < v, for v in [0, V]
__global__ void k_node_ptr(const int32_t* __restrict__ head, int64_t S, int32_t V,
                           int32_t* __restrict__ node)
{
    const int64_t v = (int64_t)blockIdx.x * BT + threadIdx.x;
    if (v > V) return;
    int64_t lo = 0, hi = S;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (head[mid] < v) lo = mid + 1; else hi = mid;
    }
    node[v] = (int32_t)lo;
}

__global__ void k_flag_active(const int32_t* __restrict__ node, int32_t V, int32_t* __restrict__ f)
{
    const int64_t v = (int64_t)blockIdx.x * BT + threadIdx.x;
    if (v < V) f[v] = node[v + 1] > node[v] ? 1 : 0;
}

__global__ void k_compact_active(const int32_t* __restrict__ node, int32_t V,
                                 const int32_t* __restrict__ pos, int32_t* __restrict__ out)
{
    const int64_t v = (int64_t)blockIdx.x * BT + threadIdx.x;
    if (v < V && node[v + 1] > node[v]) out[pos[v]] = (int32_t)v;
}

// bit v of the mask: entity v has at least one in-edge
__global__ void k_has_in(const int32_t* __restrict__ node, int32_t V, uint32_t* __restrict__ bits)
{
    const int64_t w = (int64_t)blockIdx.x * BT + threadIdx.x;
    if (w * 32 >= V) return;
    uint32_t word = 0;
    for (int b = 0; b < 32; ++b) {
        const int64_t v = w * 32 + b;
        if (v < V && node[v + 1] > node[v]) word |= 1u << b;
    }
    bits[w] = word;
}

// bit i of the coarse mask: one of entities 4i .. 4i + 3 has an in-edge
// (word w covers fine words 4w .. 4w + 3, eight bits from each)
__global__ void k_has_in4(const uint32_t* __restrict__ bits, int64_t words, uint32_t* __restrict__ coarse)
{
    const int64_t w = (int64_t)blockIdx.x * BT + threadIdx.x;
    if (w * 4 >= words) return;
    uint32_t out = 0;
    for (int f = 0; f < 4; ++f) {
        const uint32_t x = w * 4 + f < words ? bits[w * 4 + f] : 0u;
        for (int n = 0; n < 8; ++n)
            if ((x >> (4 * n)) & 0xFu) out |= 1u << (8 * f + n);
    }
    coarse[w] = out;
}

// in-relation signatures of entities 4w .. 4w + 3, one byte each: the OR
// of sig_bit(r) over the relations r of the entity's reverse groups
__global__ void k_sig(const int32_t* __restrict__ node, const int2* __restrict__ grp, int32_t V,
                      uint32_t* __restrict__ out)
{
    const int64_t w = (int64_t)blockIdx.x * BT + threadIdx.x;
    if (w * 4 >= V) return;
    uint32_t word = 0;
    for (int b = 0; b < 4; ++b) {
        const int64_t v = w * 4 + b;
        if (v >= V) break;
        uint32_t sg = 0;
        for (int32_t k = node[v]; k < node[v + 1]; ++k) sg |= sig_bit(grp[k].x);
        word |= sg << (8 * b);
    }
    out[w] = word;
}

inline unsigned grid_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

// Owns temporary device buffers for the duration of a build.
struct Scratch {
    std::vector<void*> bufs;
    ~Scratch()
    {
        for (void* p : bufs) (void)hipFree(p);
    }
    template <class T>
    T* get(int64_t count, hipError_t* e)
    {
        void* p = nullptr;
        *e = hipMalloc(&p, (size_t)(count > 0 ? count : 1) * sizeof(T));
        if (*e != hipSuccess) return nullptr;
        bufs.push_back(p);
        return (T*)p;
    }
    void release(void* p)
    {
        for (auto& b : bufs)
            if (b == p) {
                (void)hipFree(b);
                b = nullptr;
            }
    }
};

#define TRY(x)                                   \
    do {                                         \
        hipError_t e_ = (x);                     \
        if (e_ != hipSuccess) {                  \
            *err = hipGetErrorString(e_);        \
            return e_ == hipErrorOutOfMemory ? SMORE_E_NOMEM : SMORE_E_HIP; \
        }                                        \
    } while (0)

#define TRYALLOC(ptr, T, count)                  \
    do {                                         \
        hipError_t e_;                           \
        ptr = S.get<T>(count, &e_);              \
        if (!ptr) {                              \
            *err = hipGetErrorString(e_);        \
            return SMORE_E_NOMEM;                \
        }                                        \
    } while (0)

// Exclusive scan of d[0..n) in place (recursive over tile sums).
int scan_exclusive(int32_t* d, int64_t n, Scratch& S, const char** err)
{
    const int64_t nb = (n + STILE - 1) / STILE;
    if (nb == 0) return SMORE_OK;
    int32_t* sums;
    TRYALLOC(sums, int32_t, nb);
    k_scan_tile<<<(unsigned)nb, BT>>>(d, n, sums);
    TRY(hipGetLastError());
    if (nb > 1) {
        int rc = scan_exclusive(sums, nb, S, err);
        if (rc) return rc;
        k_add_offsets<<<(unsigned)nb, BT>>>(d, n, sums);
        TRY(hipGetLastError());
    }
    return SMORE_OK;
}

int bits_for(int64_t max_value)
{
    int b = 0;
    while (b < 31 && (int64_t(1) << b) <= max_value) ++b;
    return b;
}

// Stable sort of records (x[0], x[1], x[2]) by the listed keys, least
// significant first; each key is (field, bit width).  The sorted records
// end up in x[] (buffers are swapped with y[] as passes run).
int radix_sort3(int32_t* x[3], int32_t* y[3], int64_t n, const int (*keys)[2], int nkeys,
                Scratch& S, const char** err)
{
    if (n <= 1) return SMORE_OK;
    const int64_t nblk = (n + RTILE - 1) / RTILE;
    int32_t* hist;
    TRYALLOC(hist, int32_t, 256 * nblk);
    for (int k = 0; k < nkeys; ++k) {
        const int field = keys[k][0];
        for (int shift = 0; shift < keys[k][1]; shift += 8) {
            k_radix_hist<<<(unsigned)nblk, BT>>>(x[field], (int32_t)n, shift, hist, (int32_t)nblk);
            TRY(hipGetLastError());
            int rc = scan_exclusive(hist, 256 * nblk, S, err);
            if (rc) return rc;
            k_radix_scatter<<<(unsigned)nblk, BT>>>(x[0], x[1], x[2], y[0], y[1], y[2], (int32_t)n,
                                                    field, shift, hist, (int32_t)nblk);
            TRY(hipGetLastError());
            for (int f = 0; f < 3; ++f) {
                int32_t* t = x[f];
                x[f] = y[f];
                y[f] = t;
            }
        }
    }
    return SMORE_OK;
}

int32_t read_i32(const int32_t* dev, const char** err, int* rc)
{
    int32_t v = 0;
    hipError_t e = hipMemcpy(&v, dev, 4, hipMemcpyDeviceToHost);
    if (e != hipSuccess) {
        *err = hipGetErrorString(e);
        *rc = SMORE_E_HIP;
    }
    return v;
}

// Groups (runs of equal (P, R)) and node pointers over sorted records.
int build_dir(const int32_t* P, const int32_t* R, int64_t n, int32_t V, Scratch& S, int32_t** node_out,
              int2** grp_out, int64_t* S_out, const char** err)
{
    int32_t* f;
    TRYALLOC(f, int32_t, n + 1);
    TRY(hipMemset(f + n, 0, 4));
    if (n > 0) {
        k_flag_groups<<<grid_for(n, BT), BT>>>(P, R, n, f);
        TRY(hipGetLastError());
    }
    int rc = scan_exclusive(f, n + 1, S, err);
    if (rc) return rc;
    const int32_t ngrp = read_i32(f + n, err, &rc);
    if (rc) return rc;
    int2* grp = nullptr;
    int32_t* node = nullptr;
    TRY(hipMalloc(&grp, (size_t)(ngrp + 1) * sizeof(int2)));
    *grp_out = grp;
    TRY(hipMalloc(&node, (size_t)(V + 1) * sizeof(int32_t)));
    *node_out = node;
    int32_t* head;
    TRYALLOC(head, int32_t, ngrp);
    if (n > 0) {
        k_write_groups<<<grid_for(n, BT), BT>>>(P, R, n, f, grp, head);
        TRY(hipGetLastError());
    }
    const int2 sentinel = make_int2(INT32_MAX, (int32_t)n);
    TRY(hipMemcpy(grp + ngrp, &sentinel, sizeof(int2), hipMemcpyHostToDevice));
    k_node_ptr<<<grid_for((int64_t)V + 1, BT), BT>>>(head, ngrp, V, node);
    TRY(hipGetLastError());
    S.release(head);
    S.release(f);
    *S_out = ngrp;
    return SMORE_OK;
}

}  // namespace

int build_graph_device(const int32_t* triples_host, int64_t n, int32_t V, int32_t R, bool inv,
                       smore_graph* g, const char** err)
{
    TRY(hipGetDevice(&g->device));
    g->V = V;
    g->R = inv ? 2 * R : R;
    Scratch S;
    const int64_t m = inv ? 2 * n : n;
    int32_t *x[3], *y[3];
    for (int k = 0; k < 3; ++k) {
        TRYALLOC(x[k], int32_t, m);
        TRYALLOC(y[k], int32_t, m);
    }
    int* bad;
    TRYALLOC(bad, int, 1);
    TRY(hipMemset(bad, 0, sizeof(int)));
    if (n > 0) {
        int32_t* tr;
        TRYALLOC(tr, int32_t, 3 * n);
        TRY(hipMemcpy(tr, triples_host, (size_t)n * 12, hipMemcpyHostToDevice));
        k_load<<<grid_for(n, BT), BT>>>(tr, n, V, R, inv ? 1 : 0, x[0], x[1], x[2], bad);
        TRY(hipGetLastError());
        int hbad = 0;
        TRY(hipMemcpy(&hbad, bad, sizeof(int), hipMemcpyDeviceToHost));
        S.release(tr);
        if (hbad) {
            *err = "a triple has an entity or relation id out of range";
            return SMORE_E_RANGE;
        }
    }
    const int vb = bits_for(V - 1), rb = bits_for(g->R - 1);
    // forward order (h, r, t): sort by t, then r, then h
    const int fkeys[3][2] = {{2, vb}, {1, rb}, {0, vb}};
    int rc = radix_sort3(x, y, m, fkeys, 3, S, err);
    if (rc) return rc;
    // drop duplicates
    int32_t* f;
    TRYALLOC(f, int32_t, m + 1);
    TRY(hipMemset(f + m, 0, 4));
    if (m > 0) {
        k_flag_unique<<<grid_for(m, BT), BT>>>(x[0], x[1], x[2], m, f);
        TRY(hipGetLastError());
    }
    rc = scan_exclusive(f, m + 1, S, err);
    if (rc) return rc;
    const int32_t E = read_i32(f + m, err, &rc);
    if (rc) return rc;
    if (m > 0) {
        k_compact3<<<grid_for(m, BT), BT>>>(x[0], x[1], x[2], m, f, y[0], y[1], y[2]);
        TRY(hipGetLastError());
    }
    S.release(f);
    for (int k = 0; k < 3; ++k) {
        int32_t* t = x[k];
        x[k] = y[k];
        y[k] = t;
    }
    g->E = E;
    // forward adjacency: groups over (h, r), neighbours = tails
    rc = build_dir(x[0], x[1], E, V, S, &g->f_node, &g->f_grp, &g->S_fwd, err);
    if (rc) return rc;
    TRY(hipMalloc(&g->f_nbr, (size_t)(E > 0 ? E : 1) * 4));
    if (E > 0) TRY(hipMemcpy(g->f_nbr, x[2], (size_t)E * 4, hipMemcpyDeviceToDevice));
    // reverse order (t, r, h): stable sort of the (h, r, t)-ordered records by r, then t
    const int rkeys[2][2] = {{1, rb}, {2, vb}};
    rc = radix_sort3(x, y, E, rkeys, 2, S, err);
    if (rc) return rc;
    rc = build_dir(x[2], x[1], E, V, S, &g->r_node, &g->r_grp, &g->S_rev, err);
    if (rc) return rc;
    TRY(hipMalloc(&g->r_nbr, (size_t)(E > 0 ? E : 1) * 4));
    if (E > 0) TRY(hipMemcpy(g->r_nbr, x[0], (size_t)E * 4, hipMemcpyDeviceToDevice));
    for (int k = 0; k < 3; ++k) {
        S.release(x[k]);
        S.release(y[k]);
    }
    // entities with at least one in-edge
    TRYALLOC(f, int32_t, (int64_t)V + 1);
    TRY(hipMemset(f + V, 0, 4));
    k_flag_active<<<grid_for(V, BT), BT>>>(g->r_node, V, f);
    TRY(hipGetLastError());
    rc = scan_exclusive(f, (int64_t)V + 1, S, err);
    if (rc) return rc;
    const int32_t na = read_i32(f + V, err, &rc);
    if (rc) return rc;
    TRY(hipMalloc(&g->active_in, (size_t)(na > 0 ? na : 1) * 4));
    k_compact_active<<<grid_for(V, BT), BT>>>(g->r_node, V, f, g->active_in);
    TRY(hipGetLastError());
    const int64_t words = ((int64_t)V + 31) / 32;
    TRY(hipMalloc(&g->has_in, (size_t)words * 4));
    k_has_in<<<grid_for(words, BT), BT>>>(g->r_node, V, g->has_in);
    TRY(hipGetLastError());
    const int64_t cwords = ((int64_t)V + 127) / 128;
    TRY(hipMalloc(&g->has_in4, (size_t)cwords * 4));
    k_has_in4<<<grid_for(cwords, BT), BT>>>(g->has_in, words, g->has_in4);
    TRY(hipGetLastError());
    const int64_t swords = ((int64_t)V + 3) / 4;
    TRY(hipMalloc(&g->sig, (size_t)(swords > 0 ? swords : 1) * 4));
    k_sig<<<grid_for(swords, BT), BT>>>(g->r_node, g->r_grp, V, (uint32_t*)g->sig);
    TRY(hipGetLastError());
    TRY(hipDeviceSynchronize());
    g->n_active = na;
    g->bytes = (size_t)(2 * ((int64_t)V + 1) + 2 * E + na + words + cwords + swords) * 4 +
               (size_t)(g->S_fwd + g->S_rev + 2) * sizeof(int2);
    return SMORE_OK;
}

}  // namespace smore
