"""The synthetic-KG generator that stands in for the paper's datasets.

It feeds both the oracle and the library, so its stated recipe is checked
here: sizes and id ranges, distinct triples, determinism by seed, the
per-entity degree cap, and the skew of the rank-Zipf endpoint and relation
laws (uniform laws stay flat).
"""
import numpy as np
import pytest

import kgsynth


def test_fb15k237_shape_and_determinism():
    cfg = kgsynth.CONFIGS["fb15k237"]
    tr = kgsynth.generate(cfg)
    assert tr.shape == (cfg.n_triples, 3) and tr.dtype == np.int32
    assert tr[:, [0, 2]].min() >= 0 and tr[:, [0, 2]].max() < cfg.n_entities
    assert tr[:, 1].min() >= 0 and tr[:, 1].max() < cfg.n_relations
    assert len(np.unique(tr, axis=0)) == len(tr)          # the KG is a set of triples
    assert np.array_equal(tr, kgsynth.generate(cfg))       # same seed, same graph
    other = kgsynth.generate_raw(cfg.n_entities, cfg.n_relations, 10_000, head_zipf=True,
                                 head_s=1.1, rel_zipf=True, rel_s=1.0, graph_seed=1)
    assert not np.array_equal(other, tr[:10_000])


def test_zipf_heads_are_skewed_and_uniform_tails_are_flat():
    cfg = kgsynth.CONFIGS["fb15k237"]          # head Zipf(1.1), tail uniform, relation Zipf(1.0)
    tr = kgsynth.generate(cfg)
    heads = np.sort(np.bincount(tr[:, 0], minlength=cfg.n_entities))[::-1]
    tails = np.bincount(tr[:, 2], minlength=cfg.n_entities)
    rels = np.sort(np.bincount(tr[:, 1], minlength=cfg.n_relations))[::-1]
    mean = len(tr) / cfg.n_entities
    # rank-Zipf: the top head carries a large share, the median far below the mean
    assert heads[0] > 50 * mean and heads[len(heads) // 2] < mean
    # log-log slope of the head counts over ranks 10..1000 near -s (dedupe flattens the top)
    k = np.arange(10, 1000)
    slope = np.polyfit(np.log(k + 1), np.log(heads[k] + 1), 1)[0]
    assert -1.4 < slope < -0.7
    # uniform tails: every count within a few standard deviations of the mean
    assert abs(tails.mean() - mean) < 1e-9 and tails.std() < 3 * np.sqrt(mean)
    assert rels[0] > 10 * rels[len(rels) // 2]


@pytest.mark.parametrize("cap", [40, 200])
def test_degree_cap(cap):
    tr = kgsynth.generate_raw(20_000, 30, 60_000, head_zipf=True, head_s=1.3, tail_zipf=True,
                              tail_s=1.3, rel_zipf=True, rel_s=1.0, shared_perm=True, deg_cap=cap,
                              graph_seed=3, overdraw=3.0)
    assert len(np.unique(tr, axis=0)) == len(tr) == 60_000
    deg = np.bincount(tr[:, 0], minlength=20_000) + np.bincount(tr[:, 2], minlength=20_000)
    out_deg = np.bincount(tr[:, 0], minlength=20_000)
    in_deg = np.bincount(tr[:, 2], minlength=20_000)
    assert max(out_deg.max(), in_deg.max()) <= cap, (out_deg.max(), in_deg.max())
    assert deg.max() > cap // 2                           # the cap binds on the hubs


def test_shared_permutation_correlates_in_and_out_degree():
    kw = dict(head_zipf=True, head_s=1.2, tail_zipf=True, tail_s=1.2, rel_zipf=True, rel_s=1.0,
              graph_seed=5)
    shared = kgsynth.generate_raw(50_000, 20, 200_000, shared_perm=True, **kw)
    apart = kgsynth.generate_raw(50_000, 20, 200_000, shared_perm=False, **kw)

    def corr(tr):
        o = np.bincount(tr[:, 0], minlength=50_000).astype(float)
        i = np.bincount(tr[:, 2], minlength=50_000).astype(float)
        return np.corrcoef(np.log1p(o), np.log1p(i))[0, 1]

    assert corr(shared) > 0.5 and abs(corr(apart)) < 0.1
