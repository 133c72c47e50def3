"""Parity of shared-negative minibatches (smore_sample_shared; Sec. 4.3,
sharing negative samples) with the CPU oracle, bit for bit: the positives,
the shared candidate set and its size, every word of the mask and the
per-query counts.  Shapes, ragged sizes (set sizes that are not multiples
of 32 and sets larger than one candidate window), exhausted draw budgets,
queries without a positive and an empty set."""
import numpy as np
import pytest

import kgsynth
import paper_2110_14890_amd as sm
from gpu_common import config_graph, graph_pair, progress, require_gpu

pytestmark = pytest.mark.gpu


def gpu_shared(g, qt, batch, n, **kw):
    import torch
    out = sm.sample_shared(g, qt, batch, n, **kw)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items()}
    res["mask"] = res["mask"].view(np.uint32)
    return res


def assert_shared_same(got, ref, what):
    for k in sm.SHARED_FIELDS:
        a, b = got[k], ref[k]
        if not np.array_equal(a, b):
            bad = np.nonzero((a != b).reshape(len(a), -1).any(axis=1))[0] if a.ndim else [0]
            raise AssertionError(f"{what} field {k}: {len(bad)} rows differ, first {bad[0]}")


@pytest.mark.parametrize("qt", sm.TYPES)
def test_shared_parity_all_shapes(qt):
    require_gpu()
    rng = np.random.default_rng(21)
    tr = kgsynth.random_tiny(rng, 3000, 6, 60000)
    g, og = graph_pair(tr, 3000, 6, True)
    for seed, off, n, nt in [(0, 0, 37, 150), (2**64 - 1, 12345, 600, 1300), (7, 2**32 - 300, 5, 5)]:
        progress(f"shared {qt} seed {seed} n {n}")
        got = gpu_shared(g, qt, 300, n, seed=seed, query_offset=off, neg_tries=nt)
        ref = og.sample_shared(qt, 300, n, seed=seed, query_offset=off, neg_tries=nt)
        assert_shared_same(got, ref, f"{qt} seed {seed} n {n}")
        assert (got["n_valid"] >= 0).mean() > 0.5


@pytest.mark.parametrize("qt", sm.TYPES)
def test_shared_parity_fb15k237(qt):
    require_gpu()
    cfg, tr = config_graph("fb15k237")
    g, og = graph_pair(tr, cfg.n_entities, cfg.n_relations)
    got = gpu_shared(g, qt, cfg.batch, cfg.n_neg, seed=4)
    ref = og.sample_shared(qt, cfg.batch, cfg.n_neg, seed=4)
    assert_shared_same(got, ref, f"fb15k237 {qt}")


def test_shared_budget_and_pathless_graphs():
    require_gpu()
    rng = np.random.default_rng(3)
    tr = kgsynth.random_tiny(rng, 40, 2, 500)
    g, og = graph_pair(tr, 40, 2, False)
    for qt in ("1p", "2p", "3p", "2i", "pi", "up"):
        for n, nt in [(30, 30), (33, 4096), (1, 1)]:
            progress(f"shared budget {qt} n {n} tries {nt}")
            got = gpu_shared(g, qt, 97, n, seed=3, neg_tries=nt)
            ref = og.sample_shared(qt, 97, n, seed=3, neg_tries=nt)
            assert_shared_same(got, ref, f"{qt} n {n} tries {nt}")
    # no entity reachable twice: 2p/3p find no positive, rows stay zero
    tr = np.array([[0, 0, 1], [2, 0, 3], [4, 1, 5]], np.int32)
    g, og = graph_pair(tr, 6, 2)
    for qt in ("1p", "2p", "3p"):
        progress(f"shared pathless {qt}")
        got = gpu_shared(g, qt, 9, 4, pos_tries=5, neg_tries=6)
        ref = og.sample_shared(qt, 9, 4, pos_tries=5, neg_tries=6)
        assert_shared_same(got, ref, f"pathless {qt}")


def test_shared_empty_set():
    """An empty shared set (n_neg = 0): the set pointer, the mask and the
    workspace are NULL.  Such a call once wrote per-query draw counts through
    the NULL pointer (per-query mode was inferred from a NULL set); it now
    draws the empty set and launches no per-query negatives kernel, and the
    host-side rows of such calls run under the address sanitizer on the CPU
    (tests/test_host_sanitized.py)."""
    require_gpu()
    rng = np.random.default_rng(3)
    tr = kgsynth.random_tiny(rng, 40, 2, 500)
    g, og = graph_pair(tr, 40, 2, False)
    for qt in ("1p", "2p", "3p", "2i", "pi", "up"):
        progress(f"shared empty set {qt}")
        got = gpu_shared(g, qt, 97, 0, seed=3, neg_tries=0)
        ref = og.sample_shared(qt, 97, 0, seed=3, neg_tries=0)
        assert_shared_same(got, ref, f"{qt} empty set")


def test_shared_minibatch_is_deterministic_and_matches_smore_sample_positives():
    require_gpu()
    cfg, tr = config_graph("fb15k237")
    g, _ = graph_pair(tr, cfg.n_entities, cfg.n_relations)
    a = gpu_shared(g, "ip", 512, 256, seed=8, query_offset=99)
    b = gpu_shared(g, "ip", 512, 256, seed=8, query_offset=99)
    for k in sm.SHARED_FIELDS:
        assert np.array_equal(a[k], b[k]), k
    import torch
    per = sm.sample(g, "ip", 512, 4, seed=8, query_offset=99)
    torch.cuda.synchronize()
    for k in ("anchors", "relations", "positive", "pos_attempts"):
        assert np.array_equal(a[k], per[k].cpu().numpy()), k
