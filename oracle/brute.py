"""Brute-force answers of the fourteen query shapes (test infrastructure only).

Each shape is written as the first-order formula of the paper's definition
of logical queries (Sec. 2, Def. "Logical queries"): a target variable V_?,
existentially quantified variables, and a disjunction of conjunctions of
atoms r(x, y) meaning (x, r, y) is a triple of the KG.  The answer set is
every V_? for which SOME assignment of the bound variables satisfies the
formula, found here by enumerating all assignments over V.  This is
deliberately a different formulation from the computation-plan traversal
the oracle performs, so each pins the other.  Only for tiny graphs.

The five shapes with negation (2in 3in inp pin pni, the BetaE structures
the experiments use, Sec. 5.1) negate one operand of the conjunction; a
negated operand with a bound variable of its own (pni) reads "no
assignment of that variable satisfies it", so it is checked over all of V.
"""
from itertools import product


def _formula(qtype, a, r):
    """(number of bound variables, predicate(E, vq, xs) -> bool)."""
    a0, a1, a2 = a
    r0, r1, r2 = r
    if qtype == "1p":
        return 0, lambda E, v, x: (a0, r0, v) in E
    if qtype == "2p":
        return 1, lambda E, v, x: (a0, r0, x[0]) in E and (x[0], r1, v) in E
    if qtype == "3p":
        return 2, lambda E, v, x: ((a0, r0, x[0]) in E and (x[0], r1, x[1]) in E
                                   and (x[1], r2, v) in E)
    if qtype == "2i":
        return 0, lambda E, v, x: (a0, r0, v) in E and (a1, r1, v) in E
    if qtype == "3i":
        return 0, lambda E, v, x: (a0, r0, v) in E and (a1, r1, v) in E and (a2, r2, v) in E
    if qtype == "ip":
        return 1, lambda E, v, x: ((a0, r0, x[0]) in E and (a1, r1, x[0]) in E
                                   and (x[0], r2, v) in E)
    if qtype == "pi":
        return 1, lambda E, v, x: ((a0, r0, x[0]) in E and (x[0], r1, v) in E
                                   and (a1, r2, v) in E)
    if qtype == "2u":
        return 0, lambda E, v, x: (a0, r0, v) in E or (a1, r1, v) in E
    if qtype == "up":
        # disjunctive normal form: two conjunctions sharing the bound variable
        return 1, lambda E, v, x: (((a0, r0, x[0]) in E and (x[0], r2, v) in E)
                                   or ((a1, r1, x[0]) in E and (x[0], r2, v) in E))
    if qtype == "2in":
        return 0, lambda E, v, x: (a0, r0, v) in E and (a1, r1, v) not in E
    if qtype == "3in":
        return 0, lambda E, v, x: ((a0, r0, v) in E and (a1, r1, v) in E
                                   and (a2, r2, v) not in E)
    if qtype == "inp":
        return 1, lambda E, v, x: ((a0, r0, x[0]) in E and (a1, r1, x[0]) not in E
                                   and (x[0], r2, v) in E)
    if qtype == "pin":
        return 1, lambda E, v, x: ((a0, r0, x[0]) in E and (x[0], r1, v) in E
                                   and (a1, r2, v) not in E)
    if qtype == "pni":
        # the negated operand (a0 -r0-> y -r1-> v) has its own bound y
        return 0, lambda E, v, x: ((a1, r2, v) in E
                                   and not any((a0, r0, y) in E and (y, r1, v) in E
                                               for y in range(E.n_entities)))
    raise ValueError(qtype)


class _Triples(set):
    n_entities = 0


def answers(triples, n_entities, qtype, anchors, relations):
    """Sorted list of V_? satisfying the formula, by exhaustive assignment."""
    E = _Triples((int(h), int(r), int(t)) for h, r, t in triples)
    E.n_entities = n_entities
    k, pred = _formula(qtype, [int(x) for x in anchors], [int(x) for x in relations])
    out = []
    for v in range(n_entities):
        for xs in product(range(n_entities), repeat=k):
            if pred(E, v, xs):
                out.append(v)
                break
    return out


def with_inverse(triples, n_relations):
    """The triple set plus (t, r + R, h) for every (h, r, t)."""
    out = [(int(h), int(r), int(t)) for h, r, t in triples]
    out += [(int(t), int(r) + n_relations, int(h)) for h, r, t in triples]
    return out
