"""Pin of the draw order of reverse sampling (the RNG reading: attempt t of
query q uses draw j = 0 for the root, then, in grounding order, two draws
per projection step and one for the sibling entity of a complemented
operand).

Each query's positive is re-derived here in plain Python from the raw
triples: sorted in-relations and in-neighbours by value, forward lists
sorted by value, the separately pinned draw and pick functions, and the
acceptance rules of the walk (dead ends, equal single-projection siblings,
the complemented set).  The oracle's rows must match one for one, so a
changed draw index or grounding order anywhere fails here even where the
sampling law stays the same.
"""
from collections import defaultdict

import numpy as np
import pytest

import kgsynth
from oracle import brute

TAG_POS = 1

# grounding programs in the order the walk takes them: ("proj", src, slot,
# dst) draws two, ("sib", x_reg, slot, dst) draws one (uniform over the
# forward list of the step x -(slot)-> e); "neg" is (the register that must
# stay outside the complemented set, that set from anchors a and relations
# r); "pairs" are single-projection sibling (anchor register, relation slot)
# pairs that must differ
def _tails(E, h, r):
    return {t for (x, q, t) in E if x == h and q == r}


def _two_hop(E, a, r0, r1):
    return {t for y in _tails(E, a, r0) for t in _tails(E, y, r1)}


PROGRAMS = {
    "1p": ([("proj", "root", 0, "a0")], {"a0": 0}, None, []),
    "2p": ([("proj", "root", 1, "v1"), ("proj", "v1", 0, "a0")], {"a0": 0}, None, []),
    "3p": ([("proj", "root", 2, "v2"), ("proj", "v2", 1, "v1"), ("proj", "v1", 0, "a0")],
           {"a0": 0}, None, []),
    "2i": ([("proj", "root", 0, "a0"), ("proj", "root", 1, "a1")], {"a0": 0, "a1": 1}, None,
           [(("a0", 0), ("a1", 1))]),
    "ip": ([("proj", "root", 2, "x"), ("proj", "x", 0, "a0"), ("proj", "x", 1, "a1")],
           {"a0": 0, "a1": 1}, None, [(("a0", 0), ("a1", 1))]),
    "pi": ([("proj", "root", 1, "v1"), ("proj", "v1", 0, "a0"), ("proj", "root", 2, "a1")],
           {"a0": 0, "a1": 1}, None, []),
    "up": ([("proj", "root", 2, "x"), ("proj", "x", 0, "a0"), ("proj", "x", 1, "a1")],
           {"a0": 0, "a1": 1}, None, [(("a0", 0), ("a1", 1))]),
    "2in": ([("proj", "root", 0, "a0"), ("sib", "a0", 0, "w"), ("proj", "w", 1, "a1")],
            {"a0": 0, "a1": 1}, ("root", lambda E, a, r: _tails(E, a[1], r[1])), []),
    "3in": ([("proj", "root", 0, "a0"), ("proj", "root", 1, "a1"), ("sib", "a0", 0, "w"),
             ("proj", "w", 2, "a2")], {"a0": 0, "a1": 1, "a2": 2},
            ("root", lambda E, a, r: _tails(E, a[2], r[2])), [(("a0", 0), ("a1", 1))]),
    "inp": ([("proj", "root", 2, "x"), ("proj", "x", 0, "a0"), ("sib", "a0", 0, "w"),
             ("proj", "w", 1, "a1")], {"a0": 0, "a1": 1},
            ("x", lambda E, a, r: _tails(E, a[1], r[1])), []),
    "pin": ([("proj", "root", 1, "v1"), ("proj", "v1", 0, "a0"), ("sib", "v1", 1, "w"),
             ("proj", "w", 2, "a1")], {"a0": 0, "a1": 1},
            ("root", lambda E, a, r: _tails(E, a[1], r[2])), []),
    "pni": ([("proj", "root", 2, "a1"), ("sib", "a1", 2, "w"), ("proj", "w", 1, "y"),
             ("proj", "y", 0, "a0")], {"a0": 0, "a1": 1},
            ("root", lambda E, a, r: _two_hop(E, a[0], r[0], r[1])), []),
}


def rederive(oracle_lib, E, V, shape, seed, qid, pos_tries):
    steps, anchors, target, pairs = PROGRAMS[shape]
    inn = defaultdict(lambda: defaultdict(list))
    out = defaultdict(lambda: defaultdict(list))
    for h, r, t in sorted(E):
        inn[t][r].append(h)
        out[h][r].append(t)
    roots = sorted(inn)
    for t in range(pos_tries):
        if not roots:
            break
        reg = {"root": roots[oracle_lib.pick(oracle_lib.draw(seed, TAG_POS, qid, t, 0), len(roots))]}
        rel, j, ok = {}, 1, True
        for kind, src, slot, dst in steps:
            if kind == "sib":
                lst = sorted(set(out[reg[src]][rel[slot]]))
                reg[dst] = lst[oracle_lib.pick(oracle_lib.draw(seed, TAG_POS, qid, t, j), len(lst))]
                j += 1
                continue
            u0 = oracle_lib.draw(seed, TAG_POS, qid, t, j)
            u1 = oracle_lib.draw(seed, TAG_POS, qid, t, j + 1)
            j += 2
            rs = sorted(inn.get(reg[src], {}))
            if not rs:
                ok = False
                break
            r = rs[oracle_lib.pick(u0, len(rs))]
            xs = sorted(set(inn[reg[src]][r]))
            reg[dst] = xs[oracle_lib.pick(u1, len(xs))]
            rel[slot] = r
        if not ok:
            continue
        if any(reg[a] == reg[b] and rel[sa] == rel[sb] for (a, sa), (b, sb) in pairs):
            continue
        a = [-1, -1, -1]
        for n, sl in anchors.items():
            a[sl] = reg[n]
        if target is not None and reg[target[0]] in target[1](E, a, rel):
            continue
        return reg["root"], a, [rel.get(k, -1) for k in range(3)], t + 1
    return -1, [-1, -1, -1], [-1, -1, -1], pos_tries


@pytest.mark.parametrize("shape", list(PROGRAMS))
def test_positive_rows_follow_the_draw_order(oracle_lib, shape):
    rng = np.random.default_rng(404)
    V, R = 12, 3
    tr = kgsynth.random_tiny(rng, V, R, 60)
    E = sorted({tuple(x) for x in tr.tolist()})
    g = oracle_lib.Graph(tr, V, R)
    out = g.sample(shape, 40, 0, seed=77, query_offset=9, pos_tries=8)
    found = 0
    for b in range(40):
        root, a, r, att = rederive(oracle_lib, E, V, shape, 77, 9 + b, 8)
        assert out["positive"][b] == root, (shape, b)
        assert list(out["anchors"][b]) == a and list(out["relations"][b]) == r, (shape, b)
        assert out["pos_attempts"][b] == att, (shape, b)
        if root >= 0:   # and the positive answers the query
            assert root in brute.answers(E, V, shape, a, r), (shape, b)
        found += root >= 0
    assert found >= 10
