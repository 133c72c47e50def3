"""Pins of the oracle's count of memory lines a bidirectional check reads
(oracle_verify_lines; the cost of forward caching and backward verification,
Sec. 3.2, in 64-byte lines of the device layout: node[V+1] int32,
grp[S+1] int32 pairs, nbr[E] int32 per direction).

* Hand graphs whose group and edge indices are written out here: the lines
  of every read follow from those indices and the byte offsets 4v, 8s and
  4e, so each expected line set is derived without the oracle's code.
* A cached set one entry over the per-query staging budget is searched
  where it is stored (its forward group), one entry under it is free; so
  is a membership test in it, and sets are staged greedily in node order.
* Invariants on random graphs for all fourteen shapes: every draw reads its
  own node entries (a lower bound from the draws alone), the parts bound
  the total, a graph whose lists never exceed eight entries puts nothing in
  the long-list part, and more draws never read fewer lines.
* The oracle's strict cut (oracle/cuts.py) equals the library planner's."""
import numpy as np
import pytest

import kgsynth
from oracle import cuts as C

TAG_NEG = 2


def draws(oracle_lib, seed, qid, n, V):
    return [oracle_lib.pick(oracle_lib.draw(seed, TAG_NEG, qid, 0, j), V) for j in range(n)]


def lines_of(byte_off, nbytes):
    return set(range(byte_off >> 6, ((byte_off + nbytes - 1) >> 6) + 1))


def strict_mask(oracle_lib, qt):
    op, ch, slot, root = oracle_lib.type_plan(qt)
    return C.mask(C.strict(op, ch, root))


def test_edge_tests_against_an_anchor(oracle_lib):
    # 1p over anchor 0: edges (0, 0, t) for t = 10 .. 17.  Reverse groups:
    # entity t -> group t - 10 (one group each); reverse edges: tail t ->
    # edge t - 10.  The cut is the anchor: nothing is cached forward; a
    # candidate reads its node entries, and one with an in-edge its group
    # (search probe and bounds) and its one-entry list.  Group 7 ends on the
    # next line (its end bound is entry 8, bytes 68..71).
    V = 200
    tr = np.array([[0, 0, t] for t in range(10, 18)], np.int32)
    g = oracle_lib.Graph(tr, V, 1)
    anchors, rels, pos = np.array([[0, -1, -1]], np.int32), np.array([[0, -1, -1]], np.int32), \
        np.array([10], np.int32)
    n, seed = 60, 5
    hit_seen = crossing_seen = False
    for qid in range(40):
        cs = draws(oracle_lib, seed, qid, n, V)
        node, grp, nbr = set(), set(), set()
        for c in cs:
            node |= lines_of(4 * c, 8)
            if 10 <= c <= 17:
                s = c - 10
                crossing_seen |= s == 7
                grp |= lines_of(8 * s, 4) | lines_of(8 * s + 4, 4) | lines_of(8 * (s + 1) + 4, 4)
                nbr |= lines_of(4 * s, 4)
                hit_seen = True
        got = g.verify_lines("1p", anchors, rels, pos, strict_mask(oracle_lib, "1p"), seed, qid, n)
        want = len(node) + len(grp) + len(nbr)
        assert got[0].tolist() == [want, 0, want], qid
    assert hit_seen and crossing_seen


def test_two_hop_long_list_goes_to_the_long_part(oracle_lib):
    # 2p: anchor 0 -(r0)-> 1..20, each of 1..20 -(r1)-> 100; the strict cut
    # caches F0 = {1..20} (forward group 0 of entity 0, forward edges 0..19).
    # Reverse groups: entities 1..20 -> groups 0..19 (relation 0), entity 100
    # -> group 20 (relation 1); reverse edges: tails 1..20 -> edges 0..19,
    # tail 100 -> edges 20..39 (heads 1..20).  R_r1(100) has 20 > 8 entries:
    # it is met with F0 (20 entries, not fewer than the list) by reading the
    # list in order, and its first entry (entity 1, edge 20) is in F0.
    V = 300
    tr = [[0, 0, y] for y in range(1, 21)] + [[y, 1, 100] for y in range(1, 21)]
    g = oracle_lib.Graph(np.array(tr, np.int32), V, 2)
    anchors, rels = np.array([[0, -1, -1]], np.int32), np.array([[0, 1, -1]], np.int32)
    pos = np.array([100], np.int32)
    fwd = lines_of(0, 8) | set()                    # forward node entries of 0
    fgrp = lines_of(0, 4) | lines_of(4, 4) | lines_of(12, 4)
    fnbr = lines_of(0, 80)
    n, seed = 400, 9
    for qid in (0, 1, 2, 3):
        cs = draws(oracle_lib, seed, qid, n, V)
        node, grp, nbr_long = set(), set(), set()
        for c in cs:
            node |= lines_of(4 * c, 8)
            if 1 <= c <= 20:     # in-edges, but none under r1: the search fails
                grp |= lines_of(8 * (c - 1), 4)
            elif c == 100:
                grp |= lines_of(8 * 20, 4) | lines_of(8 * 20 + 4, 4) | lines_of(8 * 21 + 4, 4)
                nbr_long |= lines_of(4 * 20, 4)
        got = g.verify_lines("2p", anchors, rels, pos, strict_mask(oracle_lib, "2p"), seed, qid, n)
        part0 = len(fwd) + len(fgrp) + len(fnbr) + len(node) + len(grp)
        assert got[0].tolist() == [part0, len(nbr_long), part0 + len(nbr_long)], qid
        assert (100 in cs) == (len(nbr_long) == 1)


# Probes of the lower-bound search of a key in F0 = {1..n_f} (entry i holds
# i + 1), worked out by hand: key 3 ends at entry 2 and reads it once more;
# keys 1105 and 1110 exceed every entry and end past the last one.
PROBES = {
    1025: {3: [512, 256, 128, 64, 32, 16, 8, 4, 2, 1, 2],
           1105: [512, 769, 897, 961, 993, 1009, 1017, 1021, 1023, 1024]},
}


@pytest.mark.parametrize("n_f", [1024, 1025])
def test_cached_set_over_the_staging_budget_is_searched_in_place(oracle_lib, n_f):
    # 2p: anchor 0 -(r0)-> 1..n_f, 3 -(r1)-> 1150, 1105 and 1110 -(r1)-> 1151.
    # The strict cut caches F0 = {1..n_f}: forward group 0 of entity 0,
    # forward edges 0..n_f-1.  Reverse groups: entities 1..n_f -> groups
    # 0..n_f-1 (relation 0), 1150 -> group n_f, 1151 -> group n_f+1 (both
    # relation 1); reverse edges: tails 1..n_f -> edges 0..n_f-1, 1150 -> edge
    # n_f (head 3), 1151 -> edges n_f+1, n_f+2 (heads 1105, 1110).  Both lists
    # are shorter than F0, so their entries are the keys searched in F0.
    # With 1,024 entries F0 is staged: the searches are free and the short
    # lists are part 0.  With 1,025 it is not: every backward read is part 1
    # and each probe of F0 reads its forward edge.
    V = 1200
    tr = [[0, 0, y] for y in range(1, n_f + 1)] + [[3, 1, 1150], [1105, 1, 1151], [1110, 1, 1151]]
    g = oracle_lib.Graph(np.array(tr, np.int32), V, 2)
    anchors, rels = np.array([[0, -1, -1]], np.int32), np.array([[0, 1, -1]], np.int32)
    pos = np.array([1150], np.int32)
    fnode = lines_of(0, 8)                          # forward node entries of 0
    fgrp = lines_of(0, 4) | lines_of(4, 4) | lines_of(12, 4)
    fnbr = lines_of(0, 4 * n_f)
    n, seed = 4000, 3
    seen = set()
    for qid in range(4):
        cs = draws(oracle_lib, seed, qid, n, V)
        node, grp, rnbr, fprobe = set(), set(), set(), set()
        for c in cs:
            node |= lines_of(4 * c, 8)
            if 1 <= c <= n_f:
                grp |= lines_of(8 * (c - 1), 4)
            elif c in (1150, 1151):
                s_ = n_f + (c - 1150)
                grp |= lines_of(8 * s_, 4) | lines_of(8 * s_ + 4, 4) | lines_of(8 * (s_ + 1) + 4, 4)
                edges = [n_f] if c == 1150 else [n_f + 1, n_f + 2]
                for e_ in edges:
                    rnbr |= lines_of(4 * e_, 4)
                if n_f in PROBES:
                    for i in PROBES[n_f][3 if c == 1150 else 1105]:
                        fprobe |= lines_of(4 * i, 4)
                seen.add(c)
        got = g.verify_lines("2p", anchors, rels, pos, strict_mask(oracle_lib, "2p"), seed, qid, n)
        base = len(fnode) + len(fgrp) + len(fnbr) + len(node) + len(grp)
        if n_f in PROBES:
            assert fprobe <= fnbr
            assert got[0].tolist() == [base, len(rnbr) + len(fprobe), base + len(rnbr)], qid
        else:
            assert got[0].tolist() == [base + len(rnbr), 0, base + len(rnbr)], qid
    assert seen == {1150, 1151}


def test_membership_in_a_set_over_the_budget_and_greedy_staging(oracle_lib):
    # ip: F0 = A_r0(0) = {1..1025} (forward edges 0..1024) is over the
    # budget; F1 = A_r1(2000) = {3, 5} (forward edges 1027, 1028: heads 3 and
    # 4 hold edges 1025, 1026 under r2) still fits what F0 left, so it is
    # staged (greedy in node order).  The only in-edges under r2 end at
    # 3000, from 3 and 4 (reverse edges 1027, 1028: tails 1..1025 hold edges
    # 0..1026, tails 3 and 5 two each).  Verifying 3000 expands its list in
    # the long part: entry 3 (edge 1027, reverse line 64) is tested in F0 by
    # bisection in its forward group - probes 512, 256, ..., 2, 1 and a last
    # read of entry 2, lines 32, 16, 8, 4, 2, 1, 0 - and in F1 for free, and
    # it is in both, so 3 decides.  The forward lines are part 0's as well
    # (forward caching reads F0 whole), so the total grows by one line.
    V = 3100
    tr = ([[0, 0, y] for y in range(1, 1026)] + [[2000, 1, 3], [2000, 1, 5]]
          + [[3, 2, 3000], [4, 2, 3000]])
    g = oracle_lib.Graph(np.array(tr, np.int32), V, 3)
    anchors = np.array([[0, 2000, -1]], np.int32)
    rels = np.array([[0, 1, 2]], np.int32)
    assert sorted(np.asarray(g.answer_set("ip", anchors[0], rels[0])).tolist()) == [3000]
    pos = np.array([3000], np.int32)
    n, seed = 2000, 4
    seen = {True: 0, False: 0}
    for qid in range(12):
        drawn = 3000 in draws(oracle_lib, seed, qid, n, V)
        got = g.verify_lines("ip", anchors, rels, pos, strict_mask(oracle_lib, "ip"), seed, qid, n)[0]
        if drawn:
            assert got[1] == 8 and got[2] == got[0] + 1, (qid, got)
        else:
            assert got[1] == 0 and got[2] == got[0], (qid, got)
        seen[drawn] += 1
    assert seen[True] and seen[False]


@pytest.mark.parametrize("qt", ["1p", "2p", "3p", "2i", "3i", "ip", "pi", "2u", "up",
                                "2in", "3in", "inp", "pin", "pni"])
def test_invariants_on_random_graphs(oracle_lib, qt):
    rng = np.random.default_rng(8)
    V = 1500
    tr = kgsynth.random_tiny(rng, V, 4, 9000)
    g = oracle_lib.Graph(tr, V, 4, add_inverse=True)
    q = g.sample(qt, 48, 0, seed=2)
    ok = q["positive"] >= 0
    assert ok.sum() > 20
    m = strict_mask(oracle_lib, qt)
    L40 = g.verify_lines(qt, q["anchors"], q["relations"], q["positive"], m, 2, 0, 40)
    L80 = g.verify_lines(qt, q["anchors"], q["relations"], q["positive"], m, 2, 0, 80)
    assert (L40[~ok] == 0).all()
    for b in np.nonzero(ok)[0]:
        p0, p1, tot = L40[b]
        assert max(p0, p1) <= tot <= p0 + p1
        lower = set()
        for c in draws(oracle_lib, 2, int(b), 40, V):
            lower |= lines_of(4 * c, 8)
        assert p0 >= len(lower)
        assert (L80[b] >= L40[b]).all()
    # lists of this graph: reverse groups up to how many entries?
    e, r, o = g.dump(reverse=True)
    _, counts = np.unique(e.astype(np.int64) * 64 + r, return_counts=True)
    if counts.max() <= 8:
        assert (L40[:, 1] == 0).all()


def test_strict_cut_equals_the_library_planner(oracle_lib):
    sm = pytest.importorskip("paper_2110_14890_amd")
    import os
    if not os.path.exists(sm.LIB_PATH):
        pytest.skip("library not built")
    for qt in oracle_lib.TYPES:
        op, ch, slot, root = oracle_lib.type_plan(qt)
        assert sorted(C.strict(op, ch, root)) == sorted(sm.plan(qt, 0)), qt
