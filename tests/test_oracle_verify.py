"""Pins of the oracle's membership verification (the test behind rejection
sampling, Sec. 3.2) and of its use for evaluation on nested graphs
(appendix on the task setup: G_train within G_valid within G_test).

- Mask bits against brute-force answer sets of the first-order formulas
  (Sec. 2, Def. of logical queries) for random candidates, including ids
  outside [0, V), which are never negatives.
- Monotonicity on nested graphs for the shapes without negation: adding
  edges can only add answers there, so a candidate that is a non-answer on
  the larger graph is one on the smaller.
- A query's own positive is an answer of the graph it was sampled on.
"""
import numpy as np
import pytest

import kgsynth
from oracle import brute

TYPES = ("1p", "2p", "3p", "2i", "3i", "ip", "pi", "2u", "up", "2in", "3in", "inp", "pin", "pni")


def bits(mask, n):
    return np.array([[(int(row[k // 32]) >> (k % 32)) & 1 for k in range(n)] for row in mask])


@pytest.mark.parametrize("qtype", TYPES)
def test_verify_against_brute_force(oracle_lib, qtype):
    rng = np.random.default_rng(90)
    V, R = 10, 3
    tr = kgsynth.random_tiny(rng, V, R, 40)
    g = oracle_lib.Graph(tr, V, R)
    E = [tuple(x) for x in tr.tolist()]
    q = g.sample(qtype, 25, 0, seed=2, pos_tries=32, neg_tries=0)
    n = 40
    cand = rng.integers(-2, V + 2, size=(25, n)).astype(np.int32)
    out = g.verify(qtype, q["anchors"], q["relations"], cand)
    b = bits(out["mask"], n)
    for i in range(25):
        if q["n_valid"][i] < 0:
            # a query without a positive has -1 slots: refused, row zero
            assert out["n_valid"][i] == -1 and not b[i].any()
            continue
        ans = set(brute.answers(E, V, qtype, q["anchors"][i], q["relations"][i]))
        want = [int(0 <= c < V and c not in ans) for c in cand[i]]
        assert list(b[i]) == want
        assert out["n_valid"][i] == sum(want)


# Adding edges can also grow a negated operand's set, so a shape with
# negation may lose answers on the larger graph: monotone only without it.
@pytest.mark.parametrize("qtype", TYPES[:9])
def test_verify_is_monotone_on_nested_graphs(oracle_lib, qtype):
    rng = np.random.default_rng(91)
    V, R = 300, 4
    tr = kgsynth.random_tiny(rng, V, R, 3000)
    perm = rng.permutation(len(tr))
    train, valid = tr[perm[:2400]], tr[perm[:2700]]
    gt, gv, gx = (oracle_lib.Graph(t, V, R) for t in (train, valid, tr))
    q = gx.sample(qtype, 60, 0, seed=5, neg_tries=0)
    cand = np.concatenate([q["positive"][:, None],
                           rng.integers(0, V, size=(60, 63)).astype(np.int32)], axis=1)
    bt, bv, bx = (bits(g.verify(qtype, q["anchors"], q["relations"], cand)["mask"], 64)
                  for g in (gt, gv, gx))
    ok = q["n_valid"] >= 0
    assert ok.sum() > 30
    # non-answer on G_test => non-answer on G_valid => non-answer on G_train
    assert (bx[ok] <= bv[ok]).all() and (bv[ok] <= bt[ok]).all()
    # the positive (column 0) answers the graph it was sampled on
    assert (bx[ok, 0] == 0).all()
