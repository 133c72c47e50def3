/*
 * oracle_asan_main.c -- drives every entry point of the CPU oracle in a build
 * with the address and undefined-behaviour sanitizers (test infrastructure).
 *
 * Input on stdin: "V R add_inverse n" then n triples "h r t".  For every
 * query shape it runs sampling (with and without negatives, a draw budget
 * equal to n_neg, max_fanout), shared-candidate minibatches (empty and
 * non-empty sets), verification of given candidates (none, and candidates
 * out of range), the exhaustive answer set, the bidirectional check and the
 * count of the lines it reads on every node cut, and the line count of a
 * query whose cached set is just under and just over the staging budget.
 * Every output array is printed as one line "<case> <values...>" so that
 * the test can compare it with the ordinary build of the oracle called
 * through its Python wrapper.
 */
#include <stdio.h>
#include <stdlib.h>

#include "oracle.h"

static const char *TYPES[14] = {"1p", "2p", "3p", "2i", "3i", "ip", "pi",
                                "2u", "up", "2in", "3in", "inp", "pin", "pni"};

static void put(const char *tag, const char *ty, int k, const int32_t *v, int64_t n)
{
    printf("%s %s %d", tag, ty, k);
    for (int64_t i = 0; i < n; i++) printf(" %d", v[i]);
    printf("\n");
}

int main(void)
{
    int32_t V, R, inv;
    int64_t n;
    if (scanf("%d %d %d %ld", &V, &R, &inv, &n) != 4) return 2;
    int32_t *tr = malloc((size_t)(n > 0 ? n : 1) * 12);
    for (int64_t i = 0; i < 3 * n; i++)
        if (scanf("%d", &tr[i]) != 1) return 2;
    okg *g = oracle_graph_build(tr, n, V, R, inv, 2);
    free(tr);
    if (!g) return 3;
    const int B = 24;
    for (int ty = 0; ty < 14; ty++) {
        const char *name = TYPES[ty];
        /* sampling: (n_neg, neg_tries, max_fanout) */
        const int32_t cases[4][3] = {{0, 0, 0}, {5, 20, 0}, {5, 5, 0}, {3, 12, 2}};
        int32_t *anc = malloc(B * 12), *rel = malloc(B * 12);
        for (int k = 0; k < 4; k++) {
            oracle_args a = {B, cases[k][0], 8, cases[k][1], cases[k][2], 11, 7};
            int32_t *neg = malloc((size_t)(B * a.n_neg > 0 ? B * a.n_neg : 1) * 4);
            int32_t pos[24], nv[24], pa[24], nd[24];
            if (oracle_sample(g, ty, &a, anc, rel, pos, neg, nv, pa, nd, 2)) return 4;
            put("anchors", name, k, anc, 3 * B);
            put("relations", name, k, rel, 3 * B);
            put("positive", name, k, pos, B);
            put("negatives", name, k, neg, (int64_t)B * a.n_neg);
            put("n_valid", name, k, nv, B);
            put("pos_attempts", name, k, pa, B);
            put("neg_draws", name, k, nd, B);
            free(neg);
        }
        /* shared-candidate minibatches: set sizes 0 and 7 */
        for (int k = 0; k < 2; k++) {
            const int32_t ns = k ? 7 : 0;
            oracle_args a = {B, ns, 8, 4 * ns, 0, 5, 3};
            int32_t sh[8], nsh = -1, pos[24], pa[24], nv[24];
            uint32_t mask[24];
            if (oracle_sample_shared(g, ty, &a, anc, rel, pos, pa, ns ? sh : NULL, &nsh,
                                     ns ? mask : NULL, nv, 2))
                return 5;
            put("shared", name, k, sh, ns);
            put("n_shared", name, k, &nsh, 1);
            put("mask", name, k, (const int32_t *)mask, ns ? B : 0);
            put("shared_n_valid", name, k, nv, B);
        }
        /* verification of given candidates (0 and 9 per query, some out of
           range), on the queries of the last shared call */
        for (int k = 0; k < 2; k++) {
            const int32_t m = k ? 9 : 0;
            int32_t cand[24 * 9], nv[24];
            uint32_t mask[24];
            for (int i = 0; i < B * m; i++) cand[i] = (int32_t)((i * 7919) % (V + 6)) - 3;
            if (oracle_verify(g, ty, B, m, anc, rel, m ? cand : NULL, m ? mask : NULL, nv, 2))
                return 6;
            put("verify_mask", name, k, (const int32_t *)mask, m ? B : 0);
            put("verify_n_valid", name, k, nv, B);
        }
        /* answer set and bidirectional check of the first query with a
           positive, on every node cut, for every entity */
        for (int b = 0; b < B; b++) {
            if (anc[3 * b] < 0) continue;
            int32_t *ans = malloc((size_t)V * 4);
            const int64_t na = oracle_answer_set(g, ty, anc + 3 * b, rel + 3 * b, ans, V);
            put("answers", name, 0, ans, na);
            free(ans);
            int32_t *in = malloc((size_t)V * 4);
            for (uint32_t cut = 1; cut < 256; cut++) {
                int is_cut = 1;
                for (int32_t c = 0; c < V; c++) {
                    const int r = oracle_bidir_check(g, ty, anc + 3 * b, rel + 3 * b, cut, c, NULL);
                    if (r < 0) { is_cut = 0; break; }
                    in[c] = r;
                }
                if (is_cut) {
                    put("bidir", name, (int)cut, in, V);
                    /* lines read by the check of 40 draws of this query */
                    int64_t l64[3];
                    if (oracle_verify_lines(g, ty, anc + 3 * b, rel + 3 * b, cut, 5, (uint32_t)b, 40, l64))
                        return 7;
                    const int32_t l32[4] = {b, (int32_t)l64[0], (int32_t)l64[1], (int32_t)l64[2]};
                    put("lines", name, (int)cut, l32, 4);
                }
            }
            free(in);
            break;
        }
        free(anc);
        free(rel);
    }
    oracle_graph_free(g);
    /* line counts with a cached set over the per-query staging budget: a
       2p query whose first hop has nf entries (1,024 staged, 1,025 not) */
    for (int nf = 1024; nf <= 1025; nf++) {
        const int64_t nh = nf + 3;
        int32_t *ht = malloc((size_t)nh * 12);
        for (int i = 0; i < nf; i++) { ht[3 * i] = 0; ht[3 * i + 1] = 0; ht[3 * i + 2] = 1 + i; }
        const int32_t extra[3][3] = {{3, 1, 1150}, {1105, 1, 1151}, {1110, 1, 1151}};
        for (int i = 0; i < 3; i++)
            for (int k = 0; k < 3; k++) ht[3 * (nf + i) + k] = extra[i][k];
        okg *h = oracle_graph_build(ht, nh, 1200, 2, 0, 2);
        free(ht);
        if (!h) return 8;
        const int t2p = oracle_type_id("2p");
        const int32_t ha[3] = {0, -1, -1}, hr[3] = {0, 1, -1};
        for (uint32_t cut = 1; cut < 8; cut++) {
            int64_t l64[3];
            if (oracle_verify_lines(h, t2p, ha, hr, cut, 3, 0, 4000, l64)) continue;
            const int32_t l32[3] = {(int32_t)l64[0], (int32_t)l64[1], (int32_t)l64[2]};
            put("hublines", "2p", nf * 16 + (int)cut, l32, 3);
        }
        oracle_graph_free(h);
    }
    return 0;
}
