"""Pins of the oracle's shared-negative minibatches (Sec. 4.3, sharing
negative samples: one candidate set N for the minibatch and a mask whose
entry (i, k) says whether N[k] is a negative of query i).

- The mask is checked against answer sets found by brute force over all
  variable assignments of the query's first-order formula (Sec. 2, Def. of
  logical queries), on random tiny KGs, with and without inverse edges.
- N is the first n distinct draws of the minibatch's candidate stream, in
  draw order (re-derived from the counter-based draws, whose generator is
  pinned separately); its size is smaller only when the draw budget runs out.
- The positives are those of the per-query sampler for the same arguments.
"""
import numpy as np
import pytest

import kgsynth
from oracle import brute

TYPES = ("1p", "2p", "3p", "2i", "3i", "ip", "pi", "2u", "up", "2in", "3in", "inp", "pin", "pni")


@pytest.mark.parametrize("qtype", TYPES)
def test_shared_mask_against_brute_force(oracle_lib, qtype):
    for seed in range(3):
        rng = np.random.default_rng(70 + seed)
        V, R = 10, 3
        tr = kgsynth.random_tiny(rng, V, R, 40)
        inv = seed % 2 == 0
        g = oracle_lib.Graph(tr, V, R, add_inverse=inv)
        E = brute.with_inverse(tr, R) if inv else [tuple(x) for x in tr.tolist()]
        n, tries = 7, 9
        out = g.sample_shared(qtype, 30, n, seed=seed, query_offset=5, pos_tries=16,
                              neg_tries=tries)
        # N: first distinct draws of the shared stream (tag 3, id = query_offset)
        want = []
        for j in range(tries):
            c = oracle_lib.pick(oracle_lib.draw(seed, 3, 5, 0, j), V)
            if c not in want:
                want.append(c)
            if len(want) == n:
                break
        ns = int(out["n_shared"][0])
        assert ns == len(want) and list(out["shared"][:ns]) == want
        assert (out["shared"][ns:] == -1).all()
        per_query = g.sample(qtype, 30, 0, seed=seed, query_offset=5, pos_tries=16, neg_tries=0)
        for k in ("anchors", "relations", "positive", "pos_attempts"):
            assert np.array_equal(out[k], per_query[k]), k
        for b in range(30):
            row = out["mask"][b]
            bits = [(int(row[k // 32]) >> (k % 32)) & 1 for k in range(n)]
            if out["n_valid"][b] < 0:
                assert out["positive"][b] == -1 and not any(bits)
                continue
            ans = set(brute.answers(E, V, qtype, out["anchors"][b], out["relations"][b]))
            assert bits[:ns] == [int(c not in ans) for c in want]
            assert not any(bits[ns:])
            assert out["n_valid"][b] == sum(bits)


def test_shared_set_is_a_set_of_entities(oracle_lib):
    rng = np.random.default_rng(5)
    tr = kgsynth.random_tiny(rng, 500, 4, 3000)
    g = oracle_lib.Graph(tr, 500, 4)
    for off in (0, 77, 2**32 - 40):
        out = g.sample_shared("2p", 40, 300, seed=9, query_offset=off, neg_tries=1200)
        ns = int(out["n_shared"][0])
        s = out["shared"][:ns]
        assert ns == 300 and len(set(s.tolist())) == ns and (s >= 0).all() and (s < 500).all()
        # a different minibatch id draws a different set
        other = g.sample_shared("2p", 40, 300, seed=9, query_offset=(off + 1) % 2**31,
                                neg_tries=1200)
        assert not np.array_equal(other["shared"], out["shared"])
    # a budget that cannot reach n distinct values leaves the rest -1
    out = g.sample_shared("2p", 4, 400, seed=1, neg_tries=400)
    ns = int(out["n_shared"][0])
    assert 0 < ns < 400 and (out["shared"][ns:] == -1).all()
