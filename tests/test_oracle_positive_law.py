"""Pins of the law of the oracle's positive sampler (Sec. 3.1 and the
appendix on reverse directional sampling).

The sampler grounds the root uniformly among entities with an in-edge, then,
for every projection edge of the query, picks one of the current entity's
distinct in-relations uniformly and one in-neighbour under it uniformly;
intersection and union branches are grounded from the same entity; an
attempt that reaches an entity without in-edges, or gives two
single-projection siblings the same (anchor, relation), is discarded and a
fresh attempt is made.  The probability of every possible output row
(anchors, relations, positive) therefore follows from the graph alone: the
product of those uniform choices, summed over the hidden intermediate
entities, conditioned on acceptance.  Here that law is enumerated from the
raw triples in plain Python (no oracle code) and the oracle's rows are
tested against it with a chi-square goodness-of-fit test; the number of
attempts per query must be geometric with the acceptance probability.  The
same test rejects the plausible wrong law "uniform over in-edges", so it has
the power to see a sampler that skips the relation step.
"""
from collections import Counter, defaultdict
from fractions import Fraction

import numpy as np
import pytest
from scipy import stats

import oracle

# A small KG whose entities have in-relations of unequal sizes (so the
# two-step choice differs from a uniform in-edge), some entities without
# in-edges (dead ends) and equal sibling pairs made possible by a single
# in-edge.
TRIPLES = np.array([
    (0, 0, 1), (2, 0, 1), (3, 0, 1), (4, 1, 1),
    (1, 0, 2), (5, 1, 2),
    (1, 2, 3), (2, 2, 3), (6, 0, 3), (7, 1, 3), (0, 1, 3),
    (3, 0, 4), (3, 1, 4),
    (4, 2, 5),
    (2, 1, 6), (6, 1, 6), (1, 1, 6),
    (5, 0, 7),
], dtype=np.int32)
V, R = 8, 3

SHAPES = {
    # projection steps (source, relation slot, target), the registers are
    # "root" and intermediate names; anchors by slot; sibling groups whose
    # (anchor, relation) pairs must differ
    "1p": ([("root", 0, "a0")], ["a0"], []),
    "2p": ([("root", 1, "v1"), ("v1", 0, "a0")], ["a0"], []),
    "3p": ([("root", 2, "v2"), ("v2", 1, "v1"), ("v1", 0, "a0")], ["a0"], []),
    "2i": ([("root", 0, "a0"), ("root", 1, "a1")], ["a0", "a1"], [((0, "a0"), (1, "a1"))]),
    "3i": ([("root", 0, "a0"), ("root", 1, "a1"), ("root", 2, "a2")], ["a0", "a1", "a2"],
           [((0, "a0"), (1, "a1")), ((0, "a0"), (2, "a2")), ((1, "a1"), (2, "a2"))]),
    "ip": ([("root", 2, "x"), ("x", 0, "a0"), ("x", 1, "a1")], ["a0", "a1"],
           [((0, "a0"), (1, "a1"))]),
    "pi": ([("root", 1, "v1"), ("v1", 0, "a0"), ("root", 2, "a1")], ["a0", "a1"], []),
    "2u": ([("root", 0, "a0"), ("root", 1, "a1")], ["a0", "a1"], [((0, "a0"), (1, "a1"))]),
    "up": ([("root", 2, "x"), ("x", 0, "a0"), ("x", 1, "a1")], ["a0", "a1"],
           [((0, "a0"), (1, "a1"))]),
}


def in_lists():
    """in-relations of each entity with their in-neighbour lists (set semantics)."""
    by = defaultdict(lambda: defaultdict(set))
    for h, r, t in TRIPLES.tolist():
        by[t][r].add(h)
    return {e: {r: sorted(s) for r, s in rs.items()} for e, rs in by.items()}


def exact_law(shape, edge_law=False):
    """P(anchors, relations, positive | accepted), and the acceptance
    probability of one attempt, by enumerating every walk."""
    steps, anchors, siblings = SHAPES[shape]
    inn = in_lists()
    roots = sorted(inn)
    law = defaultdict(Fraction)

    def choices(e):
        # (relation, neighbour, probability) of one projection step from e
        rs = inn.get(e, {})
        if edge_law:
            n = sum(len(v) for v in rs.values())
            return [(r, x, Fraction(1, n)) for r, xs in rs.items() for x in xs]
        return [(r, x, Fraction(1, len(rs) * len(xs))) for r, xs in rs.items() for x in xs]

    def walk(k, reg, rel, p):
        if k == len(steps):
            for (s0, n0), (s1, n1) in siblings:
                if reg[n0] == reg[n1] and rel[s0] == rel[s1]:
                    return                                  # degenerate siblings: rejected
            key = (tuple(reg[a] for a in anchors), tuple(rel[s] for s in sorted(rel)), reg["root"])
            law[key] += p
            return
        src, slot, dst = steps[k]
        for r, x, q in choices(reg[src]):                   # no choice = dead end: rejected
            walk(k + 1, {**reg, dst: x}, {**rel, slot: r}, p * q)

    for e in roots:
        walk(0, {"root": e}, {}, Fraction(1, len(roots)))
    acc = sum(law.values())
    return {k: v / acc for k, v in law.items()}, acc


def oracle_rows(shape, batch):
    g = oracle.Graph(TRIPLES, V, R)
    out = g.sample(shape, batch, 0, seed=20211028, pos_tries=64)
    steps, anchors, _ = SHAPES[shape]
    n_rel = len({s for _, s, _ in steps})
    rows = Counter()
    for a, r, p, ok in zip(out["anchors"].tolist(), out["relations"].tolist(),
                           out["positive"].tolist(), out["n_valid"].tolist()):
        if ok == 0:
            rows[(tuple(a[:len(anchors)]), tuple(r[:n_rel]), p)] += 1
    return rows, out


def chi2_p(law, rows, n):
    keys = sorted(law)
    obs = np.array([rows.get(k, 0) for k in keys], float)
    exp = np.array([float(law[k]) * n for k in keys])
    small = exp < 5
    if small.any():        # pool the sparse cells into one
        obs = np.append(obs[~small], obs[small].sum())
        exp = np.append(exp[~small], exp[small].sum())
    return stats.chisquare(obs, exp).pvalue


N = 200_000


@pytest.mark.parametrize("shape", list(SHAPES))
def test_positive_rows_follow_the_reverse_sampling_law(shape):
    law, acc = exact_law(shape)
    rows, out = oracle_rows(shape, N)
    pa = float(acc)
    # a query fails only after 64 rejected attempts
    fails = int((out["n_valid"] == -1).sum())
    assert stats.binomtest(fails, N, (1 - pa) ** 64).pvalue > 1e-6
    # every sampled row is a possible one, with the law's frequencies
    assert set(rows) <= set(law), set(rows) - set(law)
    assert chi2_p(law, rows, N - fails) > 1e-6
    # attempts are geometric with the acceptance probability of one attempt
    att = out["pos_attempts"]
    cells = [1, 2, 3]
    obs = [int((att == c).sum()) for c in cells] + [int((att > 3).sum())]
    exp = [N * pa * (1 - pa) ** (c - 1) for c in cells] + [N * (1 - pa) ** 3]
    if pa == 1.0:
        assert (att == 1).all()
    else:
        keep = [i for i, e in enumerate(exp) if e >= 5]
        o = np.array([obs[i] for i in keep], float)
        e = np.array([exp[i] for i in keep])
        o = np.append(o, N - o.sum())
        e = np.append(e, N - e.sum())
        if e[-1] < 5:
            o, e = o[:-2].tolist() + [o[-2] + o[-1]], e[:-2].tolist() + [e[-2] + e[-1]]
        assert stats.chisquare(o, e).pvalue > 1e-6


@pytest.mark.parametrize("shape", ["1p", "2p", "ip"])
def test_law_test_rejects_uniform_in_edges(shape):
    # the competing law differs on this graph, and the same data rejects it
    law, _ = exact_law(shape)
    wrong, _ = exact_law(shape, edge_law=True)
    assert max(abs(float(law.get(k, 0) - wrong.get(k, 0))) for k in set(law) | set(wrong)) > 0.01
    rows, _ = oracle_rows(shape, N)
    assert chi2_p(wrong, rows, N) < 1e-12
