"""Host code under the address sanitizer (CPU only).

* The CPU oracle is compiled with the address and undefined-behaviour
  sanitizers together with a driver (tests/helpers/oracle_asan_main.c) that
  calls every entry point on a small random graph for all fourteen shapes:
  sampling with and without negatives, an exhausted draw budget, max_fanout,
  shared-candidate minibatches with an empty and a non-empty set,
  verification with no candidates and with out-of-range ones, answer sets,
  the bidirectional check and its line count on every node cut, and the
  line count of a query whose cached set crosses the staging budget.  Each printed array must
  equal what the ordinary oracle build returns through its wrapper.
* The sampling library's host side (the C ABI in capi.cpp) is compiled with
  the address sanitizer on the host pass only and linked with the library's
  device objects; a driver (tests/helpers/capi_asan_main.cpp) runs the
  presets, the planner, workspace sizing, argument validation of every entry
  point, and the per-query rows of queries that draw no candidates
  (write_undrawn_row) in all three call modes, with the per-query arrays
  NULL where a call has none (the empty shared set)."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import kgsynth
import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HELPERS = os.path.join(ROOT, "tests", "helpers")
PKG = os.path.join(ROOT, "paper_2110_14890_amd")
CSRC = os.path.join(PKG, "csrc")
ENV = dict(os.environ, ASAN_OPTIONS="abort_on_error=0:halt_on_error=1:detect_leaks=1",
           UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="2")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd[:3])} ... failed ({r.returncode}):\n{r.stdout[-2000:]}\n{r.stderr[-4000:]}"
    return r


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_asan")
    _run(["gcc", "-std=c11", "-O1", "-g", "-fopenmp", "-fsanitize=address,undefined",
          "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
          "-I", os.path.join(ROOT, "oracle"), os.path.join(ROOT, "oracle", "oracle.c"),
          os.path.join(HELPERS, "oracle_asan_main.c"), "-o", exe])
    rng = np.random.default_rng(77)
    V, R = 30, 3
    tr = kgsynth.random_tiny(rng, V, R, 160)
    text = f"{V} {R} 1 {len(tr)}\n" + "\n".join(" ".join(map(str, t)) for t in tr.tolist()) + "\n"
    r = _run([exe], input=text, env=ENV)
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr
    got = {}
    for line in r.stdout.splitlines():
        f = line.split()
        got[(f[0], f[1], int(f[2]))] = np.array([int(x) for x in f[3:]], dtype=np.int64)
    g = oracle.Graph(tr, V, R, add_inverse=True)
    as_i32 = lambda a: np.asarray(a).reshape(-1).astype(np.int64)
    u32 = lambda a: np.asarray(a).reshape(-1).view(np.int32).astype(np.int64)
    n_checked = 0
    for qt in oracle.TYPES:
        for k, (nn, nt, mf) in enumerate([(0, 0, 0), (5, 20, 0), (5, 5, 0), (3, 12, 2)]):
            ref = g.sample(qt, 24, nn, seed=11, query_offset=7, pos_tries=8, neg_tries=nt,
                           max_fanout=mf, threads=2)
            for name in ("anchors", "relations", "positive", "negatives", "n_valid",
                         "pos_attempts", "neg_draws"):
                assert np.array_equal(got[(name, qt, k)], as_i32(ref[name])), (qt, k, name)
                n_checked += 1
        for k, ns in enumerate((0, 7)):
            ref = g.sample_shared(qt, 24, ns, seed=5, query_offset=3, pos_tries=8, neg_tries=4 * ns,
                                  threads=2)
            assert np.array_equal(got[("shared", qt, k)], as_i32(ref["shared"])), (qt, k)
            assert got[("n_shared", qt, k)][0] == int(np.asarray(ref["n_shared"]).reshape(-1)[0])
            assert np.array_equal(got[("mask", qt, k)], u32(ref["mask"]) if ns else []), (qt, k)
            assert np.array_equal(got[("shared_n_valid", qt, k)], as_i32(ref["n_valid"])), (qt, k)
            n_checked += 4
        anc, rel = ref["anchors"], ref["relations"]
        for k, m in enumerate((0, 9)):
            cand = ((np.arange(24 * m, dtype=np.int64) * 7919) % (V + 6) - 3).astype(np.int32)
            ref_v = g.verify(qt, anc, rel, cand.reshape(24, m), threads=2)
            assert np.array_equal(got[("verify_n_valid", qt, k)], as_i32(ref_v["n_valid"])), (qt, k)
            if m:
                assert np.array_equal(got[("verify_mask", qt, k)], u32(ref_v["mask"])), (qt, k)
            n_checked += 2
        rows = np.nonzero(anc[:, 0] >= 0)[0]
        if len(rows):
            b = int(rows[0])
            ans = g.answer_set(qt, anc[b], rel[b])
            assert np.array_equal(got[("answers", qt, 0)], np.sort(as_i32(ans))), qt
            cuts = [key[2] for key in got if key[0] == "bidir" and key[1] == qt]
            assert cuts, qt
            member = np.isin(np.arange(V), as_i32(ans)).astype(np.int64)
            for cut in cuts:   # the bidirectional test is membership, on every node cut
                assert np.array_equal(got[("bidir", qt, cut)], member), (qt, cut)
                lb = got[("lines", qt, cut)]
                assert lb[0] == b
                want = g.verify_lines(qt, anc[b:b + 1], rel[b:b + 1], ref["positive"][b:b + 1],
                                      cut, 5, b, 40)
                assert np.array_equal(lb[1:], np.asarray(want).reshape(-1)), (qt, cut)
                n_checked += 2
    # a cached set just under and just over the staging budget
    for nf in (1024, 1025):
        ht = [[0, 0, 1 + i] for i in range(nf)] + [[3, 1, 1150], [1105, 1, 1151], [1110, 1, 1151]]
        h = oracle.Graph(np.array(ht, np.int32), 1200, 2)
        keys = [k for k in got if k[0] == "hublines" and k[2] // 16 == nf]
        assert keys, nf
        for k in keys:
            want = h.verify_lines("2p", np.array([[0, -1, -1]], np.int32),
                                  np.array([[0, 1, -1]], np.int32), np.array([1150], np.int32),
                                  k[2] % 16, 3, 0, 4000)
            assert np.array_equal(got[k], np.asarray(want).reshape(-1)), k
            n_checked += 1
    assert n_checked > 500


def _hipcc():
    h = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(h):
        pytest.skip("hipcc not available")
    return h


def test_capi_host_side_under_address_sanitizer(tmp_path):
    from paper_2110_14890_amd import build as libbuild

    hipcc = _hipcc()
    objs = [os.path.join(libbuild.BUILD, os.path.splitext(s)[0] + ".o")
            for s in libbuild.SOURCES if s.endswith(".hip")]
    if not all(os.path.exists(o) for o in objs):
        libbuild.build()
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    common = ["-O1", "-g", "-std=c++17", "-fPIC", f"--offload-arch={libbuild.ARCH}",
              "-fno-omit-frame-pointer", "-Xarch_host", "-fsanitize=address"]
    capi_o, drv_o, exe = (str(tmp_path / n) for n in ("capi.o", "drv.o", "capi_asan"))
    _run([hipcc, "-c", os.path.join(CSRC, "capi.cpp"), "-o", capi_o] + common + inc)
    _run([hipcc, "-c", os.path.join(HELPERS, "capi_asan_main.cpp"), "-o", drv_o] + common + inc)
    _run([hipcc, "-o", exe, drv_o, capi_o] + objs +
         [f"--offload-arch={libbuild.ARCH}", "-Xarch_host", "-fsanitize=address"])
    r = _run([exe], env=ENV)
    assert "host checks ok" in r.stdout
    assert "ERROR: AddressSanitizer" not in r.stderr, r.stderr
