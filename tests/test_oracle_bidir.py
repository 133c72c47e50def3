"""Pins of the bidirectional checker and the node-cut machinery.

- For every node cut of every shape (Def. "Node cut", enumerated by brute
  force) and every candidate entity, forward caching + backward verification
  (Sec. 3.2) decides membership exactly as the exhaustive answer set does.
- Closed forms on layered trees (Sec. 3.2 cost discussion and the
  optimal-scheduling equation): a k-hop chain over an out-tree of fan-out C
  has C^k answers and caching up to the i-th node materialises C^i
  entities; backward verification over an in-tree of fan-in C visits
  C + C^2 + ... + C^(k-i) entities when the two sides never meet.
- The worked example of Sec. 3.2 and of the appendix on reverse sampling,
  hand-encoded from the names in the text (tests/golden/coauthor_turing.json).
"""
import json
import os

import numpy as np
import pytest

import kgsynth
from oracle import cuts as C

TYPES = ("1p", "2p", "3p", "2i", "3i", "ip", "pi", "2u", "up", "2in", "3in", "inp", "pin", "pni")


@pytest.mark.parametrize("qtype", TYPES)
def test_bidirectional_equals_membership_for_every_cut(oracle_lib, qtype):
    op, ch, sl, root = oracle_lib.type_plan(qtype)
    cuts = C.all_cuts(op, ch, root)
    assert len(cuts) >= 2
    for seed in range(3):
        rng = np.random.default_rng(seed)
        V, R = 12, 3
        tr = kgsynth.random_tiny(rng, V, R, 60)
        g = oracle_lib.Graph(tr, V, R, add_inverse=True)
        out = g.sample(qtype, 6, 1, seed=seed, neg_tries=1)
        for b in range(6):
            if out["n_valid"][b] < 0:
                continue
            a, r = out["anchors"][b], out["relations"][b]
            ans = set(g.answer_set(qtype, a, r).tolist())
            for cut in cuts:
                m = C.mask(cut)
                for c in range(V):
                    got, _, _ = g.bidir_check(qtype, a, r, m, c)
                    assert got == (c in ans), (qtype, sorted(cut), c)


def test_non_cut_masks_are_refused(oracle_lib):
    tr = np.array([[0, 0, 1], [1, 1, 2]], np.int32)
    g = oracle_lib.Graph(tr, 3, 2)
    a = np.array([0, -1, -1], np.int32)
    r = np.array([0, 1, -1], np.int32)
    # 2p plan: 0 anchor, 1 V1, 2 root
    assert g.bidir_check("2p", a, r, 0b000, 2)[0] == -1      # empty
    assert g.bidir_check("2p", a, r, 0b011, 2)[0] == -1      # two nodes on one path
    assert g.bidir_check("2p", a, r, 0b010, 2)[0] == 1


def out_tree(k, fan):
    """Node 0 at layer 0; each node of layer l < k has `fan` children under relation l."""
    tr, layer, nxt = [], [0], 1
    for lvl in range(k):
        new = []
        for v in layer:
            for _ in range(fan):
                tr.append((v, lvl, nxt))
                new.append(nxt)
                nxt += 1
        layer = new
    return np.array(tr, np.int32), nxt


def in_tree(k, fan, offset):
    """Entity `offset` with `fan` in-neighbours under relation k-1, each with `fan`
    in-neighbours under relation k-2, and so on down k levels."""
    tr, layer, nxt = [], [offset], offset + 1
    for lvl in range(k - 1, -1, -1):
        new = []
        for v in layer:
            for _ in range(fan):
                tr.append((nxt, lvl, v))
                new.append(nxt)
                nxt += 1
        layer = new
    return tr, nxt


@pytest.mark.parametrize("k,qtype", [(1, "1p"), (2, "2p"), (3, "3p")])
@pytest.mark.parametrize("fan", [2, 3, 5])
def test_layered_closed_forms(oracle_lib, k, qtype, fan):
    tr1, n1 = out_tree(k, fan)
    tr2, n2 = in_tree(k, fan, n1)
    tr = np.concatenate([tr1, np.array(tr2, np.int32).reshape(-1, 3)])
    g = oracle_lib.Graph(tr, n2, 3)
    a = np.array([0, -1, -1], np.int32)
    r = np.array([0, 1, 2], np.int32)[:k].tolist() + [-1] * (3 - k)
    r = np.array(r, np.int32)
    assert len(g.answer_set(qtype, a, r)) == fan ** k          # |A_q| = C^k
    for i in range(k + 1):                                      # cut at plan node i (V_i)
        m = 1 << i
        # forward: C^i entities cached; a leaf of the out-tree is an answer
        got, fwd, _ = g.bidir_check(qtype, a, r, m, n1 - 1)
        assert got == 1 and fwd == fan ** i
        # backward from the in-tree root, which the anchor never reaches
        got, fwd, visited = g.bidir_check(qtype, a, r, m, n1)
        assert got == 0 and visited == sum(fan ** l for l in range(1, k - i + 1))


def test_worked_example(oracle_lib):
    path = os.path.join(os.path.dirname(__file__), "golden", "coauthor_turing.json")
    ex = json.load(open(path))
    ent = {n: i for i, n in enumerate(ex["entities"])}
    rel = {n: i for i, n in enumerate(ex["relations"])}
    tr = np.array([[ent[h], rel[r], ent[t]] for h, r, t in ex["triples"]], np.int32)
    g = oracle_lib.Graph(tr, len(ent), len(rel))
    q = ex["query"]
    a = np.array([ent[x] for x in q["anchors"]] + [-1], np.int32)
    r = np.array([rel[x] for x in q["relations"]], np.int32)
    ans = g.answer_set(q["type"], a, r)
    assert [ex["entities"][x] for x in ans] == ex["answers"]
    # a cut at the intersection output caches exactly {Bengio}
    node = ex["intersection_node"]
    op, ch, sl, root = oracle_lib.type_plan("ip")
    assert op[node] == 2 and C.is_cut(op, ch, root, {node})
    got, fwd, _ = g.bidir_check("ip", a, r, 1 << node, ent["Neal"])
    assert got == 1 and fwd == len(ex["cached_at_intersection"])
    # reverse sampling: whenever the root is Neal, the walk passes Bengio and
    # grounds the two branches to (Turing Award, Win) and (Canada, Citizen)
    out = g.sample("ip", 400, 1, seed=3, pos_tries=64, neg_tries=4)
    hits = out["positive"] == ent["Neal"]
    assert hits.any()
    for b in np.nonzero(hits)[0]:
        pairs = {(out["anchors"][b][k], out["relations"][b][k]) for k in range(2)}
        assert pairs == {(ent["TuringAward"], rel["Win"]), (ent["Canada"], rel["Citizen"])}
        assert out["relations"][b][2] == rel["CoAuthor"]
