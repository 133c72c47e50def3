// capi_asan_main.cpp -- host-side checks of the sampling library in a build
// whose host code carries the address sanitizer (test infrastructure; no GPU
// is needed: every call here returns before any device work).
//
//  1. The rows a query that draws no candidates writes (write_undrawn_row):
//     per-query sampling writes its negatives row and draw count, while a
//     shared-candidate minibatch and verification of given candidates must
//     never touch those arrays, whose pointers are NULL there (an empty
//     shared set, n_neg = 0, is passed exactly like that).
//  2. The C ABI's host paths: presets, the node-cut planner under both
//     tie-breaks, workspace sizing, and argument validation of every
//     sampling entry point, each error path with its code and message.
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "rows.h"
#include "smore.h"

static int n_fail = 0;

#define CHECK(c)                                                          \
    do {                                                                  \
        if (!(c)) {                                                       \
            std::fprintf(stderr, "check failed line %d: %s\n", __LINE__, #c); \
            ++n_fail;                                                     \
        }                                                                 \
    } while (0)

static void undrawn_rows()
{
    for (int mode = 0; mode < 3; ++mode)
        for (int n_neg : {0, 3})
            for (int ok = 0; ok < 2; ++ok) {
                smore::SampleParams p;
                p.batch = 4;
                p.n_neg = n_neg;
                p.shared_mode = mode;
                smore_sample_out out;
                std::memset(&out, 0, sizeof(out));
                int32_t n_valid[4] = {7, 7, 7, 7};
                out.n_valid = n_valid;
                // per-query arrays exist only in per-query mode; elsewhere
                // they stay NULL and any access is a sanitizer error
                int32_t* negs = nullptr;
                int32_t* draws = nullptr;
                if (mode == 0) {
                    negs = (int32_t*)std::malloc(sizeof(int32_t) * (4 * n_neg + 1));
                    draws = (int32_t*)std::malloc(sizeof(int32_t) * 4);
                    for (int k = 0; k < 4 * n_neg; ++k) negs[k] = 9;
                    for (int k = 0; k < 4; ++k) draws[k] = 9;
                    out.negatives = n_neg ? negs : nullptr;
                    out.neg_draws = draws;
                }
                smore::write_undrawn_row(p, out, 2, ok != 0);
                CHECK(n_valid[2] == (ok ? 0 : -1));
                CHECK(n_valid[1] == 7 && n_valid[3] == 7);
                if (mode == 0) {
                    CHECK(draws[2] == (ok ? 0 : -1));
                    CHECK(draws[1] == 9 && draws[3] == 9);
                    for (int k = 0; k < n_neg; ++k) {
                        CHECK(negs[2 * n_neg + k] == -1);
                        CHECK(negs[n_neg + k] == 9 && negs[3 * n_neg + k] == 9);
                    }
                }
                std::free(negs);
                std::free(draws);
            }
}

static const char* kNames[14] = {"1p", "2p", "3p", "2i", "3i", "ip", "pi",
                                 "2u", "up", "2in", "3in", "inp", "pin", "pni"};

static void presets_and_planner()
{
    for (const char* nm : kNames) {
        smore_query_dag d;
        CHECK(smore_query_preset(nm, &d) == SMORE_OK);
        int32_t cut[16], n = -1;
        for (int tie = 0; tie < 2; ++tie) {
            CHECK(smore_plan(&d, tie, cut, &n) == SMORE_OK);
            CHECK(n >= 1 && n <= 3);
        }
        CHECK(smore_plan(&d, 2, cut, &n) == SMORE_E_INVALID_ARG);
        CHECK(smore_plan(&d, 0, nullptr, &n) == SMORE_E_INVALID_ARG);
    }
    smore_query_dag d;
    CHECK(smore_query_preset("4p", &d) == SMORE_E_UNSUPPORTED);
    CHECK(std::strlen(smore_last_error()) > 0);
    CHECK(smore_query_preset(nullptr, &d) == SMORE_E_INVALID_ARG);
    // a plan that is not a tree
    std::memset(&d, 0, sizeof(d));
    d.n_nodes = 2;
    d.root = 1;
    d.node[0] = {SMORE_OP_ANCHOR, 0, {-1, -1, -1}, 0};
    d.node[1] = {SMORE_OP_PROJ, 1, {1, -1, -1}, 0};
    int32_t cut[16], n = 0;
    CHECK(smore_plan(&d, 0, cut, &n) == SMORE_E_INVALID_ARG);
}

static void validation()
{
    smore_query_dag d;
    smore_query_preset("3p", &d);
    smore_sample_args a;
    std::memset(&a, 0, sizeof(a));
    a.batch = 8;
    a.n_neg = 4;
    a.pos_tries = 4;
    a.neg_tries = 16;
    size_t bytes = 0;
    CHECK(smore_sample_workspace_bytes(nullptr, &d, &a, &bytes) == SMORE_OK && bytes > 0);
    a.n_neg = 0;
    a.neg_tries = 0;
    CHECK(smore_sample_workspace_bytes(nullptr, &d, &a, &bytes) == SMORE_OK);
    a.neg_tries = SMORE_MAX_NEG_TRIES + 1;
    CHECK(smore_sample_workspace_bytes(nullptr, &d, &a, &bytes) == SMORE_E_INVALID_ARG);
    a.n_neg = 4;
    a.neg_tries = 16;
    int32_t dummy[64];
    smore_sample_out o = {dummy, dummy, dummy, dummy, dummy, dummy, dummy};
    // arms of the instrumentation hooks are taken and dropped by failing calls
    CHECK(smore_profile_kernel(dummy, dummy, 0) == SMORE_OK);
    CHECK(smore_wait_before_kernel(dummy, 0) == SMORE_OK);
    CHECK(smore_profile_kernel(dummy, dummy, 3) == SMORE_E_INVALID_ARG);
    CHECK(smore_wait_before_kernel(dummy, 1) == SMORE_E_INVALID_ARG);
    // no graph: refused after the host checks
    CHECK(smore_sample(nullptr, &d, &a, &o, dummy, sizeof(dummy), nullptr) == SMORE_E_INVALID_ARG);
    CHECK(std::strstr(smore_last_error(), "graph") != nullptr);
    CHECK(smore_sample_negatives(nullptr, &d, &a, &o, nullptr, dummy, 8, nullptr) == SMORE_E_INVALID_ARG);
    CHECK(smore_sample_negatives_part(nullptr, &d, &a, &o, nullptr, 3, dummy, 8, nullptr) ==
          SMORE_E_INVALID_ARG);
    CHECK(smore_sample_positives(nullptr, &d, &a, &o, nullptr) == SMORE_E_INVALID_ARG);
    // argument errors
    smore_sample_args b = a;
    b.batch = 0;
    CHECK(smore_sample(nullptr, &d, &b, &o, dummy, 8, nullptr) == SMORE_E_INVALID_ARG);
    b = a;
    b.neg_tries = 2;
    CHECK(smore_sample(nullptr, &d, &b, &o, dummy, 8, nullptr) == SMORE_E_INVALID_ARG);
    b = a;
    b.neg_tries = SMORE_MAX_NEG_TRIES + 1;
    CHECK(smore_sample(nullptr, &d, &b, &o, dummy, 8, nullptr) == SMORE_E_UNSUPPORTED);
    b = a;
    b.query_offset = (1ull << 32) - 4;
    CHECK(smore_sample(nullptr, &d, &b, &o, dummy, 8, nullptr) == SMORE_E_OVERFLOW);
    b = a;
    b.flags = 1u << 30;
    CHECK(smore_sample(nullptr, &d, &b, &o, dummy, 8, nullptr) == SMORE_E_INVALID_ARG);
    b = a;
    b.max_fanout = -1;
    CHECK(smore_sample(nullptr, &d, &b, &o, dummy, 8, nullptr) == SMORE_E_INVALID_ARG);
    smore_sample_out o2 = o;
    o2.neg_draws = nullptr;
    CHECK(smore_sample(nullptr, &d, &a, &o2, dummy, 8, nullptr) == SMORE_E_INVALID_ARG);
    CHECK(smore_sample(nullptr, &d, nullptr, &o, dummy, 8, nullptr) == SMORE_E_INVALID_ARG);
    CHECK(smore_sample(nullptr, nullptr, &a, &o, dummy, 8, nullptr) == SMORE_E_INVALID_ARG);
    // shared minibatches and verification: an empty set needs no mask,
    // no set and no workspace, and is refused only for the missing graph
    smore_shared_out so = {dummy, dummy, dummy, dummy, nullptr, dummy, nullptr, dummy};
    b = a;
    b.n_neg = 0;
    b.neg_tries = 0;
    CHECK(smore_sample_shared(nullptr, &d, &b, &so, nullptr, 0, nullptr) == SMORE_E_INVALID_ARG);
    CHECK(std::strstr(smore_last_error(), "graph") != nullptr);
    CHECK(smore_sample_shared(nullptr, &d, &a, &so, dummy, 8, nullptr) == SMORE_E_INVALID_ARG);
    CHECK(std::strstr(smore_last_error(), "output pointer") != nullptr);
    CHECK(smore_verify(nullptr, &d, &b, dummy, dummy, nullptr, nullptr, dummy, nullptr, 0, nullptr) ==
          SMORE_E_INVALID_ARG);
    CHECK(std::strstr(smore_last_error(), "graph") != nullptr);
    CHECK(smore_verify(nullptr, &d, &a, dummy, dummy, nullptr, nullptr, dummy, dummy, 8, nullptr) ==
          SMORE_E_INVALID_ARG);
    CHECK(std::strstr(smore_last_error(), "pointer") != nullptr);
    // the entry point without a workspace refuses arguments that need more
    // than its fixed scratch before it looks at the graph
    b = a;
    b.batch = 16384;
    b.n_neg = 512;
    b.neg_tries = 2048;
    CHECK(smore_sample_noalloc(nullptr, &d, &b, &o, nullptr) == SMORE_E_UNSUPPORTED);
    CHECK(std::strstr(smore_last_error(), "scratch") != nullptr);
    CHECK(smore_sample_noalloc(nullptr, &d, &a, &o, nullptr) == SMORE_E_INVALID_ARG);
    CHECK(std::strstr(smore_last_error(), "graph") != nullptr);
    // probe argument checks
    uint32_t sink[4];
    CHECK(smore_gather_probe(nullptr, 64, 1, sink, 4, nullptr) == SMORE_E_INVALID_ARG);
    CHECK(smore_gather_probe(dummy, 32, 1, sink, 4, nullptr) == SMORE_E_INVALID_ARG);
    CHECK(smore_gather_probe(dummy, 64, 0, sink, 4, nullptr) == SMORE_E_INVALID_ARG);
    CHECK(smore_graph_info(nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr) ==
          SMORE_E_INVALID_ARG);
    CHECK(smore_graph_copy(nullptr, 0, dummy, 1) == SMORE_E_INVALID_ARG);
    smore_free_graph(nullptr);
}

int main()
{
    undrawn_rows();
    presets_and_planner();
    validation();
    if (n_fail) {
        std::fprintf(stderr, "%d checks failed\n", n_fail);
        return 1;
    }
    std::printf("host checks ok\n");
    return 0;
}
