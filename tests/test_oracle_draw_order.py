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


def rederive(oracle_lib, E, V, shape, seed, qid, pos_tries, max_fanout=0, skip_fanout_step=-1):
    """Positive of query qid.  max_fanout > 0: an attempt is rejected when a
    projection step grounded as (x, r) -> e has |A_r(x)| > max_fanout (the
    maximum expansion C per relation, Sec. 5.2).  skip_fanout_step leaves
    that check out at one projection step (index among the projection
    steps), to show the fixtures tell the steps apart."""
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
        rel, j, ok, k_proj = {}, 1, True, -1
        for kind, src, slot, dst in steps:
            if kind == "sib":
                lst = sorted(set(out[reg[src]][rel[slot]]))
                reg[dst] = lst[oracle_lib.pick(oracle_lib.draw(seed, TAG_POS, qid, t, j), len(lst))]
                j += 1
                continue
            u0 = oracle_lib.draw(seed, TAG_POS, qid, t, j)
            u1 = oracle_lib.draw(seed, TAG_POS, qid, t, j + 1)
            j += 2
            k_proj += 1
            rs = sorted(inn.get(reg[src], {}))
            if not rs:
                ok = False
                break
            r = rs[oracle_lib.pick(u0, len(rs))]
            xs = sorted(set(inn[reg[src]][r]))
            reg[dst] = xs[oracle_lib.pick(u1, len(xs))]
            rel[slot] = r
            if max_fanout > 0 and k_proj != skip_fanout_step and len(set(out[reg[dst]][r])) > max_fanout:
                ok = False
                break
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


N_PROJ = {shape: sum(1 for st in PROGRAMS[shape][0] if st[0] == "proj") for shape in PROGRAMS}


@pytest.mark.parametrize("shape", list(PROGRAMS))
def test_max_fanout_checked_at_every_projection_step(oracle_lib, shape):
    """The maximum expansion C (Sec. 5.2, max_fanout) rejects an attempt
    when any grounded projection step (x, r) -> e has |A_r(x)| > C, at every
    step of the walk, not only the one into the root.  Every row of the
    oracle equals the plain-Python re-derivation for C = 1, 2, 3, and for
    each projection step the derivation that skips the check at that step
    alone disagrees with the oracle on some row, so a check dropped from any
    step fails here."""
    rng = np.random.default_rng(505)
    V, R = 14, 2
    tr = kgsynth.random_tiny(rng, V, R, 90)
    E = sorted({tuple(x) for x in tr.tolist()})
    g = oracle_lib.Graph(tr, V, R)
    nq, seed, off, tries = 60, 31, 5, 6
    told_apart = [False] * N_PROJ[shape]
    accepted = 0
    for C in (1, 2, 3):
        out = g.sample(shape, nq, 0, seed=seed, query_offset=off, pos_tries=tries, max_fanout=C)
        for b in range(nq):
            root, a, r, att = rederive(oracle_lib, E, V, shape, seed, off + b, tries, max_fanout=C)
            assert out["positive"][b] == root, (shape, C, b)
            assert list(out["anchors"][b]) == a and list(out["relations"][b]) == r, (shape, C, b)
            assert out["pos_attempts"][b] == att, (shape, C, b)
            accepted += root >= 0
            for k in range(N_PROJ[shape]):
                if told_apart[k]:
                    continue
                alt = rederive(oracle_lib, E, V, shape, seed, off + b, tries, max_fanout=C,
                               skip_fanout_step=k)
                told_apart[k] = alt != (root, a, r, att)
    assert accepted > 0, shape
    assert all(told_apart), (shape, told_apart)


def test_max_fanout_on_the_second_and_third_hop_only(oracle_lib):
    """Hand graphs where only a deeper hop is wide: the oracle must reject
    walks whose second (2p) or third (3p) step expands beyond C although the
    step into the root is narrow."""
    # 2p: root 9 <-(r1) 5 <-(r0) 0; anchor 0 has 4 out-edges under r0, so the
    # second step (x = 0, r0) is wide while the first (x = 5, r1) has one
    tr = np.array([[0, 0, 5], [0, 0, 6], [0, 0, 7], [0, 0, 8], [5, 1, 9]], np.int32)
    g = oracle_lib.Graph(tr, 10, 2)
    # qids whose root is 9 (the only root that reaches an anchor in two hops)
    out = g.sample("2p", 64, 0, seed=3, pos_tries=64, max_fanout=0)
    assert (out["positive"] == 9).any()
    assert (out["anchors"][out["n_valid"] >= 0, 0] == 0).all()
    out = g.sample("2p", 64, 0, seed=3, pos_tries=64, max_fanout=3)
    assert (out["n_valid"] == -1).all()
    out = g.sample("2p", 64, 0, seed=3, pos_tries=64, max_fanout=4)
    assert (out["n_valid"] >= 0).any()
    # 3p: root 12 <-(r2) 11 <-(r1) 10 <-(r0) 0; only the third step (anchor 0
    # under r0, 3 tails) is wide
    tr = np.array([[0, 0, 10], [0, 0, 1], [0, 0, 2], [10, 1, 11], [11, 2, 12]], np.int32)
    g = oracle_lib.Graph(tr, 13, 3)
    out = g.sample("3p", 64, 0, seed=4, pos_tries=64, max_fanout=0)
    assert (out["n_valid"] >= 0).all() and (out["anchors"][:, 0] == 0).all()
    for C in (1, 2):
        out = g.sample("3p", 64, 0, seed=4, pos_tries=64, max_fanout=C)
        assert (out["n_valid"] == -1).all(), C
    out = g.sample("3p", 64, 0, seed=4, pos_tries=64, max_fanout=3)
    assert (out["n_valid"] >= 0).all()
