"""Pins of the oracle's five shapes with negation (2in 3in inp pin pni, the
BetaE structures of the experiments, Sec. 5.1; complement is a plan
operator, appendix on the computation plan).

- Answer sets equal those of the first-order formula with a negated
  operand, found by enumerating every variable assignment (oracle/brute.py),
  on random tiny KGs and in every set-building mode; the intersection with a
  complemented operand is the set difference of the appendix on the optimal
  cut.
- Reverse sampling with a negated operand follows the reading stated in the
  oracle's header: positive operands first, then a sibling entity w drawn
  uniformly from the first positive operand's step A_r(x), the negated
  operand grounded from w, and rejection when the intersection's entity
  falls in the negated set.  The law of every output row under that reading
  is enumerated here from the raw triples in plain Python and the oracle's
  rows are tested against it (chi-square), with the attempts geometric in
  the acceptance probability.
- Every sampled positive is an answer and every negative a non-answer; the
  negated set always shares w with the positive operand it was drawn from.
"""
from collections import Counter, defaultdict
from fractions import Fraction

import numpy as np
import pytest
from scipy import stats

import kgsynth
import oracle
from oracle import brute

NEG_TYPES = ("2in", "3in", "inp", "pin", "pni")

TRIPLES = np.array([
    (0, 0, 1), (2, 0, 1), (3, 0, 1), (4, 1, 1),
    (1, 0, 2), (5, 1, 2), (0, 0, 2),
    (1, 2, 3), (2, 2, 3), (6, 0, 3), (7, 1, 3), (0, 1, 3), (0, 0, 3),
    (3, 0, 4), (3, 1, 4), (4, 1, 3),
    (4, 2, 5), (4, 2, 2),
    (2, 1, 6), (6, 1, 6), (1, 1, 6),
    (5, 0, 7), (6, 1, 5),
], dtype=np.int32)
V, R = 8, 3

# positive steps (source register, relation slot, target register); the
# sibling (register x, relation slot) whose A_r(x) holds w; the negated
# steps from w; the register that must stay outside the negated set; the
# negated set from (registers, relations); anchor registers by slot;
# single-projection sibling pairs that must differ.
def _tails(E, h, r):
    return {t for (a, b, t) in E if a == h and b == r}


def _two_hop(E, a, r0, r1):
    return {t for y in _tails(E, a, r0) for t in _tails(E, y, r1)}


SHAPES = {
    "2in": ([("root", 0, "a0")], ("a0", 0), [("w", 1, "a1")], "root",
            lambda E, g, r: _tails(E, g["a1"], r[1]), ["a0", "a1"], []),
    "3in": ([("root", 0, "a0"), ("root", 1, "a1")], ("a0", 0), [("w", 2, "a2")], "root",
            lambda E, g, r: _tails(E, g["a2"], r[2]), ["a0", "a1", "a2"],
            [((0, "a0"), (1, "a1"))]),
    "inp": ([("root", 2, "x"), ("x", 0, "a0")], ("a0", 0), [("w", 1, "a1")], "x",
            lambda E, g, r: _tails(E, g["a1"], r[1]), ["a0", "a1"], []),
    "pin": ([("root", 1, "v1"), ("v1", 0, "a0")], ("v1", 1), [("w", 2, "a1")], "root",
            lambda E, g, r: _tails(E, g["a1"], r[2]), ["a0", "a1"], []),
    "pni": ([("root", 2, "a1")], ("a1", 2), [("w", 1, "y"), ("y", 0, "a0")], "root",
            lambda E, g, r: _two_hop(E, g["a0"], r[0], r[1]), ["a0", "a1"], []),
}


def exact_law(shape, tr):
    pos, (sx, ss), neg, target, negset, anchors, siblings = SHAPES[shape]
    E = {tuple(x) for x in tr.tolist()}
    inn = defaultdict(lambda: defaultdict(set))
    for h, r, t in E:
        inn[t][r].add(h)
    roots = sorted(inn)
    law = defaultdict(Fraction)

    def choices(e):
        rs = inn.get(e, {})
        return [(r, x, Fraction(1, len(rs) * len(xs))) for r, xs in rs.items() for x in sorted(xs)]

    def run(steps, k, reg, rel, p, done):
        if k == len(steps):
            done(reg, rel, p)
            return
        src, slot, dst = steps[k]
        for r, x, q in choices(reg[src]):
            run(steps, k + 1, {**reg, dst: x}, {**rel, slot: r}, p * q, done)

    def finish(reg, rel, p):
        if reg[target] in negset(E, reg, rel):
            return                                      # intersection entity negated: rejected
        for (s0, n0), (s1, n1) in siblings:
            if reg[n0] == reg[n1] and rel[s0] == rel[s1]:
                return
        key = (tuple(reg[a] for a in anchors), tuple(rel[s] for s in sorted(rel)), reg["root"])
        law[key] += p

    def after_positive(reg, rel, p):
        ws = sorted(_tails(E, reg[sx], rel[ss]))
        for w in ws:
            run(neg, 0, {**reg, "w": w}, rel, p * Fraction(1, len(ws)), finish)

    for e in roots:
        run(pos, 0, {"root": e}, {}, Fraction(1, len(roots)), after_positive)
    acc = sum(law.values())
    return {k: v / acc for k, v in law.items()}, acc


def chi2_p(law, rows, n):
    keys = sorted(law)
    obs = np.array([rows.get(k, 0) for k in keys], float)
    exp = np.array([float(law[k]) * n for k in keys])
    small = exp < 5
    if small.any():
        obs = np.append(obs[~small], obs[small].sum())
        exp = np.append(exp[~small], exp[small].sum())
    return stats.chisquare(obs, exp).pvalue


N = 200_000


@pytest.mark.parametrize("shape", NEG_TYPES)
def test_negation_rows_follow_the_sibling_grounding_law(oracle_lib, shape):
    law, acc = exact_law(shape, TRIPLES)
    pa = float(acc)
    assert 0.02 < pa < 1.0 and len(law) >= 5
    g = oracle_lib.Graph(TRIPLES, V, R)
    out = g.sample(shape, N, 0, seed=20211028, pos_tries=64)
    _, _, _, _, _, anchors, _ = SHAPES[shape]
    n_rel = 2 if shape == "2in" else 3
    rows = Counter()
    for a, r, p, ok in zip(out["anchors"].tolist(), out["relations"].tolist(),
                           out["positive"].tolist(), out["n_valid"].tolist()):
        if ok == 0:
            rows[(tuple(a[:len(anchors)]), tuple(r[:n_rel]), p)] += 1
    fails = int((out["n_valid"] == -1).sum())
    assert stats.binomtest(fails, N, (1 - pa) ** 64).pvalue > 1e-6
    assert set(rows) <= set(law), set(rows) - set(law)
    assert chi2_p(law, rows, N - fails) > 1e-6
    att = out["pos_attempts"][out["n_valid"] >= 0]
    obs = [int((att == c).sum()) for c in (1, 2)] + [int((att > 2).sum())]
    exp = [N * pa, N * pa * (1 - pa)]
    exp.append(len(att) - sum(exp))
    assert stats.chisquare(obs, exp).pvalue > 1e-6


@pytest.mark.parametrize("shape", NEG_TYPES)
def test_positive_answers_the_negated_query(oracle_lib, shape):
    # grounding the negated operand from the intersection's own entity (the
    # plausible other reading) would put the root in the negated set, so
    # the root would never be an answer
    g = oracle_lib.Graph(TRIPLES, V, R)
    out = g.sample(shape, 2000, 0, seed=5, pos_tries=64)
    E = {tuple(x) for x in TRIPLES.tolist()}
    ok = out["n_valid"] >= 0
    assert ok.sum() > 100
    for b in np.nonzero(ok)[0][:200]:
        a, r, v = out["anchors"][b], out["relations"][b], out["positive"][b]
        assert v in brute.answers(E, V, shape, a, r)


@pytest.mark.parametrize("shape", NEG_TYPES)
def test_positive_negated_set_overlaps_its_sibling(oracle_lib, shape):
    for seed in range(4):
        rng = np.random.default_rng(300 + seed)
        Vt, Rt = 12, 3
        tr = kgsynth.random_tiny(rng, Vt, Rt, 70)
        inv = seed % 2 == 1
        g = oracle_lib.Graph(tr, Vt, Rt, add_inverse=inv)
        E = set(brute.with_inverse(tr, Rt)) if inv else {tuple(x) for x in tr.tolist()}
        out = g.sample(shape, 60, 4, seed=seed, pos_tries=32, neg_tries=12)
        ok = out["n_valid"] >= 0
        assert ok.sum() > 10
        for b in np.nonzero(ok)[0]:
            a, r = out["anchors"][b].tolist(), out["relations"][b].tolist()
            ans = set(brute.answers(E, Vt, shape, a, r))
            assert out["positive"][b] in ans
            nv = out["n_valid"][b]
            assert not (set(out["negatives"][b][:nv].tolist()) & ans)
            # the sibling entity w lies in both the positive operand's step
            # set and the negated set, so the two meet
            if shape == "2in":
                meet = _tails(E, a[0], r[0]) & _tails(E, a[1], r[1])
            elif shape == "3in":
                meet = _tails(E, a[0], r[0]) & _tails(E, a[2], r[2])
            elif shape == "inp":
                meet = _tails(E, a[0], r[0]) & _tails(E, a[1], r[1])
            elif shape == "pin":
                meet = _two_hop(E, a[0], r[0], r[1]) & _tails(E, a[1], r[2])
            else:
                meet = _tails(E, a[1], r[2]) & _two_hop(E, a[0], r[0], r[1])
            assert meet, (shape, seed, b)


def test_negated_branch_without_meeting_never_subtracts(oracle_lib):
    # 2in with a negated operand disjoint from the positive one answers
    # like 1p; an equal operand leaves nothing
    tr = np.array([[0, 0, 1], [0, 0, 2], [3, 1, 4], [3, 0, 1]], np.int32)
    g = oracle_lib.Graph(tr, 5, 2)
    a = np.array([0, 3, -1], np.int32)
    assert list(g.answer_set("2in", a, np.array([0, 1, -1], np.int32))) == [1, 2]
    assert list(g.answer_set("2in", a, np.array([0, 0, -1], np.int32))) == [2]
    assert list(g.answer_set("2in", np.array([0, 0, -1], np.int32),
                             np.array([0, 0, -1], np.int32))) == []
    # a graph where every sibling w equals the root: 2in can never be grounded
    tr = np.array([[0, 0, 1], [2, 0, 3]], np.int32)
    g = oracle_lib.Graph(tr, 4, 1)
    out = g.sample("2in", 20, 1, pos_tries=8, neg_tries=1)
    assert (out["n_valid"] == -1).all() and (out["pos_attempts"] == 8).all()
