"""Pins of the oracle's answer sets, positives and negatives.

- A_q by exhaustive plan traversal equals the answers of the first-order
  formula of the query definition found by enumerating every variable
  assignment (Sec. 2, Def. "Logical queries"), on random tiny KGs, in every
  set-building mode of the oracle.
- Textbook special cases on mid-size graphs: 1p is one dictionary lookup
  (Sec. 3, first paragraph), 2i a set intersection, 2u a set union, 2p a
  union of lookups (Python sets over numpy-deduplicated triples).
- Invariants of the sample (Sec. 2 contrastive setup; Sec. 3.1 and 3.2):
  the positive is an answer, every negative is a non-answer, negatives are
  distinct, n_valid and neg_draws agree with the acceptance sequence
  re-derived from the draws and the brute-force answer set.
"""
import numpy as np
import pytest

from oracle import brute
import kgsynth

TYPES = ("1p", "2p", "3p", "2i", "3i", "ip", "pi", "2u", "up", "2in", "3in", "inp", "pin", "pni")


def tiny_graph(seed, V=9, R=3, n=30, inverse=False):
    rng = np.random.default_rng(seed)
    return kgsynth.random_tiny(rng, V, R, n), V, R


@pytest.mark.parametrize("qtype", TYPES)
@pytest.mark.parametrize("mode", [0, 1, 2])
def test_answer_set_equals_first_order_brute_force(oracle_lib, qtype, mode):
    oracle_lib.set_proj_mode(mode)
    try:
        for seed in range(6):
            tr, V, R = tiny_graph(seed, V=8 if qtype in ("3p",) else 9)
            inv = seed % 2 == 1
            g = oracle_lib.Graph(tr, V, R, add_inverse=inv)
            E = brute.with_inverse(tr, R) if inv else tr
            rng = np.random.default_rng(100 + seed)
            for _ in range(8):
                a = rng.integers(0, V, 3).astype(np.int32)
                r = rng.integers(0, g.R, 3).astype(np.int32)
                got = list(g.answer_set(qtype, a, r))
                want = brute.answers(E, V, qtype, a, r)
                assert got == want, (seed, a, r)
    finally:
        oracle_lib.set_proj_mode(0)


def _lookup(E):
    d = {}
    for h, r, t in E:
        d.setdefault((h, r), set()).add(t)
    return d


def test_special_cases_by_set_operations(oracle_lib):
    tr = kgsynth.generate("fb15k237")
    cfg = kgsynth.CONFIGS["fb15k237"]
    g = oracle_lib.Graph(tr, cfg.n_entities, cfg.n_relations)
    E = [tuple(x) for x in np.unique(tr, axis=0).tolist()]
    d = _lookup(E)
    rng = np.random.default_rng(3)
    heads = np.unique(tr[:, 0])
    for _ in range(40):
        a = rng.choice(heads, 3).astype(np.int32)
        r = np.array([tr[tr[:, 0] == x][rng.integers(0, (tr[:, 0] == x).sum()), 1] for x in a],
                     dtype=np.int32)
        s0 = d.get((a[0], r[0]), set())
        s1 = d.get((a[1], r[1]), set())
        assert list(g.answer_set("1p", a, r)) == sorted(s0)
        assert list(g.answer_set("2i", a, r)) == sorted(s0 & s1)
        assert list(g.answer_set("2u", a, r)) == sorted(s0 | s1)
        two = set()
        for y in s0:
            two |= d.get((y, r[1]), set())
        assert list(g.answer_set("2p", a, r)) == sorted(two)


@pytest.mark.parametrize("qtype", TYPES)
def test_sample_invariants_against_brute_force(oracle_lib, qtype):
    for seed in range(4):
        tr, V, R = tiny_graph(50 + seed, V=10, R=3, n=40)
        inv = seed % 2 == 0
        g = oracle_lib.Graph(tr, V, R, add_inverse=inv)
        E = brute.with_inverse(tr, R) if inv else [tuple(x) for x in tr.tolist()]
        Eset = set(map(tuple, E))
        n_neg, neg_tries = 3, 7
        out = g.sample(qtype, 40, n_neg, seed=seed, query_offset=11, pos_tries=16,
                       neg_tries=neg_tries)
        for b in range(40):
            nv = out["n_valid"][b]
            if nv < 0:
                assert out["positive"][b] == -1 and out["pos_attempts"][b] == 16
                assert (out["negatives"][b] == -1).all() and out["neg_draws"][b] == -1
                continue
            a, r = out["anchors"][b], out["relations"][b]
            ans = set(brute.answers(E, V, qtype, a, r))
            assert out["positive"][b] in ans
            # anchors/relations used by the shape are set, unused are -1
            used = {"1p": 1, "2p": 1, "3p": 1, "2i": 2, "3i": 3, "ip": 2, "pi": 2, "2u": 2,
                    "up": 2, "2in": 2, "3in": 3, "inp": 2, "pin": 2, "pni": 2}[qtype]
            nrel = {"1p": 1, "2p": 2, "3p": 3, "2i": 2, "2u": 2, "2in": 2}.get(qtype, 3)
            assert (a[:used] >= 0).all() and (a[used:] == -1).all()
            assert (r[:nrel] >= 0).all() and (r[nrel:] == -1).all()
            # edges touching the anchors exist (witness of the grounding)
            for k in range(used):
                assert any(h == a[k] for h, _, _ in Eset)
            # re-derive the acceptance sequence from the draws
            seen, acc, draws = set(), [], neg_tries
            for j in range(neg_tries):
                c = oracle_lib.pick(oracle_lib.draw(seed, 2, 11 + b, 0, j), V)
                first = c not in seen
                seen.add(c)
                if first and c not in ans:
                    acc.append(c)
                    if len(acc) == n_neg:
                        draws = j + 1
                        break
            assert nv == len(acc)
            assert list(out["negatives"][b][:nv]) == acc
            assert (out["negatives"][b][nv:] == -1).all()
            assert out["neg_draws"][b] == draws
            assert len(set(acc)) == len(acc) and not (set(acc) & ans)


def test_no_positive_when_graph_has_no_path(oracle_lib):
    # every entity has in-edges only from entities without in-edges: a 2p
    # walk always reaches an entity with no in-edge and is rejected
    tr = np.array([[0, 0, 2], [1, 0, 3]], np.int32)
    g = oracle_lib.Graph(tr, 4, 1)
    out = g.sample("2p", 5, 2, pos_tries=4, neg_tries=2)
    assert (out["n_valid"] == -1).all() and (out["pos_attempts"] == 4).all()
    assert (out["positive"] == -1).all() and (out["anchors"] == -1).all()
    out = g.sample("1p", 5, 2, pos_tries=4, neg_tries=2)
    assert (out["pos_attempts"] == 1).all() and (out["positive"] >= 2).all()


def test_degenerate_intersection_rejected(oracle_lib):
    # a single in-edge: both 2i branches would be grounded to the same
    # (anchor, relation), so every attempt is rejected
    tr = np.array([[0, 0, 1]], np.int32)
    g = oracle_lib.Graph(tr, 2, 1)
    for q in ("2i", "2u", "3i", "ip", "up"):
        out = g.sample(q, 3, 1, pos_tries=5, neg_tries=1)
        assert (out["n_valid"] == -1).all(), q
    out = g.sample("pi", 3, 1, pos_tries=5, neg_tries=1)   # pi needs a 2-hop branch
    assert (out["n_valid"] == -1).all()


def test_max_fanout_rejects_wide_steps(oracle_lib):
    # entity 0 has 5 out-edges under relation 0; with max_fanout 4 no 1p
    # query anchored at 0 can be grounded
    tr = np.array([[0, 0, t] for t in range(1, 6)] + [[6, 0, 1]], np.int32)
    g = oracle_lib.Graph(tr, 7, 1)
    out = g.sample("1p", 200, 1, pos_tries=64, neg_tries=1, max_fanout=4)
    ok = out["n_valid"] >= 0
    assert ok.any() and (out["anchors"][ok, 0] == 6).all()
    out = g.sample("1p", 200, 1, pos_tries=64, neg_tries=1, max_fanout=0)
    assert (out["anchors"][:, 0] == 0).any()


def test_n_neg_zero_and_budget_exhaustion(oracle_lib):
    tr = np.array([[0, 0, 1], [0, 0, 2], [0, 0, 3]], np.int32)
    g = oracle_lib.Graph(tr, 4, 1)
    out = g.sample("1p", 6, 0, neg_tries=0)
    assert (out["n_valid"] == 0).all() and (out["neg_draws"] == 0).all()
    # A_q = {1, 2, 3} out of V = 4: at most one negative (entity 0) exists
    out = g.sample("1p", 6, 3, neg_tries=12)
    assert (out["n_valid"] <= 1).all() and (out["neg_draws"] == 12).all()
    assert set(out["negatives"][out["n_valid"] == 1, 0].tolist()) <= {0}
